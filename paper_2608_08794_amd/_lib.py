"""ctypes binding of include/apack.h (argument marshalling only)."""

import ctypes
import os
import threading

HERE = os.path.dirname(os.path.abspath(__file__))

APACK_BF16, APACK_F32 = 0, 1
APACK_OTHER, APACK_AUDIO, APACK_VISUAL = 0, 1, 2

_STATUS = {
    0: "APACK_OK", 1: "APACK_E_ARG", 2: "APACK_E_SHAPE", 3: "APACK_E_DTYPE",
    4: "APACK_E_WORKSPACE", 5: "APACK_E_ALIAS", 6: "APACK_E_HIP", 7: "APACK_E_UNSUPPORTED",
}


class ApackError(RuntimeError):
    def __init__(self, status, message):
        self.status = status
        super().__init__(f"{_STATUS.get(status, status)}: {message}")


class Span(ctypes.Structure):
    _fields_ = [("begin", ctypes.c_int64), ("len", ctypes.c_int64),
                ("modality", ctypes.c_int32), ("reserved", ctypes.c_int32)]


APACK_RANK_JOINT = 1
ALIGNMENTS = {"gated_cka": 0, "cka": 1, "av_cosine": 2, "spatial_cka": 3}


class Seq(ctypes.Structure):
    _fields_ = [("tok_off", ctypes.c_int64), ("n_tokens", ctypes.c_int64),
                ("spans", ctypes.POINTER(Span)), ("n_spans", ctypes.c_int32),
                ("flags", ctypes.c_int32), ("q_off", ctypes.c_int64),
                ("q_len", ctypes.c_int64), ("keep", ctypes.c_double * 2),
                ("keep_basis", ctypes.c_int64 * 2)]


class DynParams(ctypes.Structure):
    _fields_ = [("window", ctypes.c_int32), ("dafps_k", ctypes.c_int32),
                ("tau_gate", ctypes.c_double), ("beta", ctypes.c_double),
                ("gamma", ctypes.c_double), ("tau_sim", ctypes.c_double),
                ("sigma", ctypes.c_double), ("lambda_seg", ctypes.c_double),
                ("cover_thresh", ctypes.c_double), ("dafps_power", ctypes.c_double),
                ("r_pre", ctypes.c_double), ("alignment", ctypes.c_int32)]


class AVSeq(ctypes.Structure):
    _fields_ = [("n_frames", ctypes.c_int32), ("tokens_per_frame", ctypes.c_int32),
                ("n_audio", ctypes.c_int64), ("n_query", ctypes.c_int64),
                ("vis_off", ctypes.c_int64), ("aud_off", ctypes.c_int64),
                ("qry_off", ctypes.c_int64)]


_P = ctypes.c_void_p
_I32, _I64, _SZ = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
_SIGS = {
    "apack_version": (ctypes.c_char_p, []),
    "apack_last_error": (ctypes.c_char_p, []),
    "apack_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "apack_keep_count": (_I64, [ctypes.c_double, _I64]),
    "apack_visual_budget": (_I64, [ctypes.c_double, _I64, _I64]),
    "apack_dyn_params_default": (None, [ctypes.POINTER(DynParams)]),
    "apack_prune_layer_query": (ctypes.c_int, [_I32, ctypes.POINTER(Seq), _I32, _I32, _I32,
                                               ctypes.POINTER(_I64), ctypes.POINTER(_SZ)]),
    "apack_prune_layer": (ctypes.c_int, [_I32, ctypes.POINTER(Seq), ctypes.c_int, _I32, _I32, _I32,
                                         _P, _I64, _I64, _P, _I64, _I64, _P, _P, _I64,
                                         ctypes.POINTER(_I64), _P, _SZ, _P]),
    "apack_compact_kv": (ctypes.c_int, [_I64, _P, _I64, _I32, ctypes.POINTER(_P), ctypes.POINTER(_P),
                                        ctypes.POINTER(_P), ctypes.POINTER(_P), _I32, _I32, ctypes.c_int,
                                        _I64, _I64, _P, _P, _I32, _P, _P, _I32, _I64, _I64, _P]),
    "apack_compact_kv_inplace_workspace": (_SZ, [_I64]),
    "apack_compact_kv_inplace_static": (ctypes.c_int, [_I64, _P, _I64, _I32, ctypes.POINTER(_P),
                                                       ctypes.POINTER(_P), _I32, _I32, ctypes.c_int, _I64, _P,
                                                       _I32, _P, _I32, _I64, _P]),
    "apack_compact_kv_inplace_status": (ctypes.c_int, [_P, _SZ, ctypes.POINTER(_I32), _P]),
    "apack_set_inplace_wait_limit": (ctypes.c_uint32, [ctypes.c_uint32]),
    "apack_layer_flops": (ctypes.c_double, [_I64, _I64, _I64]),
    "apack_prefill_flops": (ctypes.c_int, [_I32, ctypes.POINTER(_I64), _I64, _I64, _I64,
                                           ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]),
    "apack_schedule_lengths": (ctypes.c_int, [_I32, _I64, _I32, ctypes.POINTER(_I32), ctypes.POINTER(_I64),
                                              ctypes.POINTER(_I64)]),
    "apack_compact_kv_inplace": (ctypes.c_int, [_I64, _P, _I64, _I32, ctypes.POINTER(_P), ctypes.POINTER(_P),
                                                _I32, _I32, ctypes.c_int, _I64, _P, _I32, _P, _I32, _I64,
                                                _P, _SZ, _P]),
    "apack_score_dynamics_query": (ctypes.c_int, [_I32, ctypes.POINTER(AVSeq), _I32,
                                                  ctypes.POINTER(DynParams), ctypes.POINTER(_I64),
                                                  ctypes.POINTER(_SZ)]),
    "apack_score_dynamics": (ctypes.c_int, [_I32, ctypes.POINTER(AVSeq), ctypes.c_int, _I32,
                                            _P, _I64, _P, _I64, _P, _I64, ctypes.POINTER(DynParams),
                                            _P, _P, _P, _P, _P, _P, _I64, ctypes.POINTER(_I64),
                                            _P, _SZ, _P]),
}

_lib = None
_lock = threading.Lock()


def library_path():
    return os.environ.get("APACK_LIBRARY", os.path.join(HERE, "libapack.so"))


def library():
    """The loaded libapack.so (loaded on first use)."""
    global _lib
    with _lock:
        if _lib is None:
            path = library_path()
            if not os.path.exists(path):
                raise ApackError(6, f"{path} is missing: build it with paper_2608_08794_amd.build.build()")
            lib = ctypes.CDLL(path)
            for name, (res, args) in _SIGS.items():
                fn = getattr(lib, name)
                fn.restype = res
                fn.argtypes = args
            _lib = lib
        return _lib


def _check(status):
    if status != 0:
        msg = library().apack_last_error().decode(errors="replace")
        raise ApackError(status, msg)


# ---------------------------------------------------------------------------
# torch plumbing (device memory and streams only)
# ---------------------------------------------------------------------------

def _torch():
    import torch
    return torch


def _stream(stream):
    if stream is not None:
        return ctypes.c_void_p(stream if isinstance(stream, int) else stream.cuda_stream)
    return ctypes.c_void_p(_torch().cuda.current_stream().cuda_stream)


def _alloc_on(stream):
    """Context for the tensors the binding allocates for a call enqueued on
    `stream` (outputs, workspace): torch allocates and fills them on that
    stream, so the caching allocator does not hand their memory out again
    before the call's kernels are done, and any fill runs before them."""
    torch = _torch()
    if stream is None:
        return torch.cuda.stream(None)
    return torch.cuda.stream(torch.cuda.ExternalStream(stream) if isinstance(stream, int) else stream)


def _dtype_code(t):
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return APACK_BF16
    if t.dtype == torch.float32:
        return APACK_F32
    raise ApackError(3, f"unsupported dtype {t.dtype}")


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def _heads_rows(t, name):
    """[heads, rows, d] tensor with contiguous rows; returns head stride."""
    if t.dim() != 3 or t.stride(2) != 1 or t.stride(1) != t.shape[2]:
        raise ApackError(2, f"{name} must be [heads, rows, d] with contiguous d-element rows")
    return t.stride(0)


def _workspace(nbytes, device):
    torch = _torch()
    ws = torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)
    if ws.data_ptr() % 256:
        raise ApackError(4, "workspace allocation is not 256-byte aligned")
    return ws


# ---------------------------------------------------------------------------
# Entry points
# ---------------------------------------------------------------------------

def apack_keep_count(keep, n):
    return int(library().apack_keep_count(float(keep), int(n)))


def apack_visual_budget(r_pre, n_audio, n_visual):
    return int(library().apack_visual_budget(float(r_pre), int(n_audio), int(n_visual)))


def _seq_array(seqs):
    arr = (Seq * max(1, len(seqs)))()
    keep_alive = []
    for i, s in enumerate(seqs):
        g = s.__getitem__ if isinstance(s, dict) else lambda k, s=s: getattr(s, k)
        spans = g("spans")
        sp = (Span * max(1, len(spans)))()
        for j, (b, n, m) in enumerate(spans):
            sp[j] = Span(int(b), int(n), int(m), 0)
        keep_alive.append(sp)
        keep = g("keep")
        try:
            basis = g("keep_basis")
        except (KeyError, AttributeError):
            basis = (0, 0)
        try:
            joint = bool(g("joint"))
        except (KeyError, AttributeError):
            joint = False
        arr[i] = Seq(int(g("tok_off")), int(g("n_tokens")), sp, len(spans), APACK_RANK_JOINT if joint else 0,
                     int(g("q_off")), int(g("q_len")),
                     (ctypes.c_double * 2)(float(keep[0]), float(keep[1])),
                     (ctypes.c_int64 * 2)(int(basis[0]), int(basis[1])))
    return arr, keep_alive


def apack_prune_layer_query(seqs, hq, hkv, d):
    """(n_kept per sequence, workspace bytes) of a prune step."""
    arr, _keep = _seq_array(seqs)
    n = len(seqs)
    n_kept = (ctypes.c_int64 * max(1, n))()
    ws = ctypes.c_size_t(0)
    _check(library().apack_prune_layer_query(n, arr, hq, hkv, d, n_kept, ctypes.byref(ws)))
    return [int(n_kept[i]) for i in range(n)], int(ws.value)


def apack_prune_layer(q, k, seqs, scores=None, kept_rows=None, workspace=None, stream=None):
    """Score, select and list kept rows for a packed batch (Eq. 5-6).

    q: [Hq, q_rows, D] and k: [Hkv, k_rows, D] CUDA tensors (bf16 or f32)
    with contiguous D-element rows; seqs: descriptors with tok_off,
    n_tokens, spans [(begin, len, modality)], q_off, q_len, keep (audio,
    visual) and optionally keep_basis.  Returns (scores [k_rows] f32,
    kept_rows int32, n_kept list).
    """
    torch = _torch()
    hq, q_rows, d = q.shape
    hkv, k_rows, _ = k.shape
    if k.dtype != q.dtype:
        raise ApackError(3, "q and k must share a dtype")
    qhs, khs = _heads_rows(q, "q"), _heads_rows(k, "k")
    arr, _keep = _seq_array(seqs)
    n = len(seqs)
    n_kept = (ctypes.c_int64 * max(1, n))()
    if scores is None or kept_rows is None or workspace is None:
        # Output and workspace sizes (the call itself checks what it is given).
        wsb = ctypes.c_size_t(0)
        _check(library().apack_prune_layer_query(n, arr, hq, hkv, d, n_kept, ctypes.byref(wsb)))
        total = sum(int(n_kept[i]) for i in range(n))
        with _alloc_on(stream):
            if scores is None:
                scores = torch.zeros(k_rows, dtype=torch.float32, device=k.device)
            if kept_rows is None:
                kept_rows = torch.empty(max(total, 1), dtype=torch.int32, device=k.device)
            if workspace is None:
                workspace = _workspace(wsb.value, k.device)
    _check(library().apack_prune_layer(
        n, arr, _dtype_code(q), hq, hkv, d, _ptr(q), qhs, q_rows, _ptr(k), khs, k_rows,
        _ptr(scores), _ptr(kept_rows), kept_rows.numel(), n_kept,
        _ptr(workspace), workspace.numel(), _stream(stream)))
    counts = [int(n_kept[i]) for i in range(n)]
    return scores, kept_rows[:sum(counts)], counts


def apack_compact_kv(src_rows, n_in, k_in=(), v_in=(), k_out=(), v_out=(), hidden_in=None,
                     hidden_out=None, pos_in=None, pos_out=None, stream=None):
    """out[i] = in[src_rows[i]] for every K/V layer tensor [Hkv, rows, D],
    the hidden states [rows, H] and the position ids [P, rows]."""
    n_out = int(src_rows.numel())
    n_layers = len(k_in)
    k_only = n_layers > 0 and len(v_in) == 0 and len(v_out) == 0
    if len(k_out) != n_layers or (not k_only and not (len(v_in) == len(v_out) == n_layers)):
        raise ApackError(1, "k_in, v_in, k_out and v_out need one tensor per layer (or empty v_in and v_out)")
    tabs = [(ctypes.c_void_p * max(1, n_layers))() for _ in range(4)]
    hkv = d = 0
    hs_in = hs_out = 0
    code = APACK_BF16
    for l in range(n_layers):
        planes = (k_in[l], k_out[l]) if k_only else (k_in[l], v_in[l], k_out[l], v_out[l])
        for tab, t in zip((tabs[0], tabs[2]) if k_only else tabs, planes):
            tab[l] = t.data_ptr()
        hkv, _, d = k_in[l].shape
        hs_in, hs_out = _heads_rows(k_in[l], "k_in"), _heads_rows(k_out[l], "k_out")
        if not k_only:
            for t in (v_in[l], v_out[l]):
                _heads_rows(t, "v")
        code = _dtype_code(k_in[l])
    hid = 0
    if hidden_in is not None:
        hid = hidden_in.shape[1]
        code = _dtype_code(hidden_in) if n_layers == 0 else code
        if hidden_in.stride(1) != 1 or hidden_in.stride(0) != hid or hidden_out.stride(0) != hid:
            raise ApackError(2, "hidden states must be contiguous [rows, H]")
    prow = 0
    ps_in = ps_out = 0
    if pos_in is not None:
        prow = pos_in.shape[0]
        ps_in, ps_out = pos_in.stride(0), pos_out.stride(0)
        if pos_in.stride(1) != 1 or pos_out.stride(1) != 1:
            raise ApackError(2, "position ids must have unit column stride")
    _check(library().apack_compact_kv(
        n_out, _ptr(src_rows), int(n_in), n_layers, tabs[0], None if k_only else tabs[1], tabs[2],
        None if k_only else tabs[3],
        hkv, d, code, hs_in, hs_out, _ptr(hidden_in), _ptr(hidden_out), hid,
        _ptr(pos_in), _ptr(pos_out), prow, ps_in, ps_out, _stream(stream)))


def apack_compact_kv_inplace_workspace(n_out):
    return int(library().apack_compact_kv_inplace_workspace(int(n_out)))


def _inplace_args(src_rows, k, v, hidden, pos):
    """(n_out, K table, V table, hkv, d, dtype code, head stride, hidden
    width, position rows, position stride) of an in-place compaction."""
    n_out = int(src_rows.numel())
    n_layers = len(k)
    if len(v) not in (0, n_layers):
        raise ApackError(1, "v needs one tensor per layer of k, or none")
    tk = (ctypes.c_void_p * max(1, n_layers))()
    tv = (ctypes.c_void_p * max(1, n_layers))() if len(v) else None
    hkv = d = hs = 0
    code = APACK_BF16
    for l in range(n_layers):
        tk[l] = k[l].data_ptr()
        hkv, _, d = k[l].shape
        hs = _heads_rows(k[l], "k")
        if tv is not None:
            tv[l] = v[l].data_ptr()
            if _heads_rows(v[l], "v") != hs or tuple(v[l].shape) != tuple(k[l].shape):
                raise ApackError(2, "v tensors must match the k tensors' shape and head stride")
        code = _dtype_code(k[l])
    hid = 0
    if hidden is not None:
        hid = hidden.shape[1]
        code = _dtype_code(hidden) if n_layers == 0 else code
        if hidden.stride(1) != 1 or hidden.stride(0) != hid:
            raise ApackError(2, "hidden states must be contiguous [rows, H]")
    prow = ps = 0
    if pos is not None:
        prow, ps = pos.shape[0], pos.stride(0)
        if pos.stride(1) != 1:
            raise ApackError(2, "position ids must have unit column stride")
    return n_out, tk, tv, hkv, d, code, hs, hid, prow, ps


def apack_compact_kv_inplace(src_rows, n_in, k=(), v=(), hidden=None, pos=None, workspace=None, stream=None):
    """x[i] = x[src_rows[i]] in place for every K/V layer tensor [Hkv, rows, D]
    (v may be empty: K planes only), the hidden states [rows, H] and the
    position ids [P, rows]; src_rows must be strictly increasing.  Rows
    [0, n_out) hold the result, later rows keep their contents."""
    n_out, tk, tv, hkv, d, code, hs, hid, prow, ps = _inplace_args(src_rows, k, v, hidden, pos)
    need = apack_compact_kv_inplace_workspace(n_out)
    if workspace is None:
        with _alloc_on(stream):
            workspace = _workspace(need, src_rows.device)
    _check(library().apack_compact_kv_inplace(
        n_out, _ptr(src_rows), int(n_in), len(k), tk, tv, hkv, d, code, hs,
        _ptr(hidden), hid, _ptr(pos), prow, ps, workspace.data_ptr(), workspace.numel(), _stream(stream)))


def apack_compact_kv_inplace_static(src_rows, n_in, k=(), v=(), hidden=None, pos=None, stream=None):
    """apack_compact_kv_inplace with the library's static scratch instead of a
    workspace: allocates nothing (n_out <= 2^20)."""
    n_out, tk, tv, hkv, d, code, hs, hid, prow, ps = _inplace_args(src_rows, k, v, hidden, pos)
    _check(library().apack_compact_kv_inplace_static(
        n_out, _ptr(src_rows), int(n_in), len(k), tk, tv, hkv, d, code, hs,
        _ptr(hidden), hid, _ptr(pos), prow, ps, _stream(stream)))


def apack_compact_kv_inplace_status(workspace, stream=None):
    """True if the last in-place compaction on `workspace` gave up a wait
    (its result is unusable); synchronises the stream."""
    flag = ctypes.c_int32(0)
    _check(library().apack_compact_kv_inplace_status(_ptr(workspace), workspace.numel(), ctypes.byref(flag),
                                                     _stream(stream)))
    return bool(flag.value)


def apack_set_inplace_wait_limit(polls):
    """Sets the bound on one in-place ordering wait; returns the previous one."""
    return int(library().apack_set_inplace_wait_limit(int(polls)))


def apack_layer_flops(n, d_model, d_ffn):
    return float(library().apack_layer_flops(int(n), int(d_model), int(d_ffn)))


def apack_prefill_flops(lengths, n0, d_model, d_ffn):
    """(F_pre, ratio) of a per-layer length schedule."""
    arr = (_I64 * max(1, len(lengths)))(*[int(x) for x in lengths])
    f, r = ctypes.c_double(0), ctypes.c_double(0)
    _check(library().apack_prefill_flops(len(lengths), arr, int(n0), int(d_model), int(d_ffn),
                                         ctypes.byref(f), ctypes.byref(r)))
    return f.value, r.value


def apack_schedule_lengths(n_layers, n_start, prune_layers, n_after):
    """Lengths entering each layer; a prune at layer l takes effect from l + 1."""
    pl = (_I32 * max(1, len(prune_layers)))(*[int(x) for x in prune_layers])
    na = (_I64 * max(1, len(n_after)))(*[int(x) for x in n_after])
    out = (_I64 * max(1, int(n_layers)))()
    if len(prune_layers) != len(n_after):
        raise ApackError(1, "prune_layers and n_after differ in length")
    _check(library().apack_schedule_lengths(int(n_layers), int(n_start), len(prune_layers), pl, na, out))
    return [int(out[i]) for i in range(int(n_layers))]


def apack_dyn_params_default():
    p = DynParams()
    library().apack_dyn_params_default(ctypes.byref(p))
    return p


def _params(params):
    """apack_dyn_params from the defaults and a dict of overrides; the
    alignment scorer may be given by name (see ALIGNMENTS)."""
    p = apack_dyn_params_default()
    for key, val in (params or {}).items():
        if key == "alignment" and isinstance(val, str):
            val = ALIGNMENTS[val]
        setattr(p, key, val)
    return p


def _av_array(seqs):
    arr = (AVSeq * max(1, len(seqs)))()
    for i, s in enumerate(seqs):
        g = s.__getitem__ if isinstance(s, dict) else lambda k, s=s: getattr(s, k)
        arr[i] = AVSeq(int(g("n_frames")), int(g("per_frame")), int(g("n_audio")), int(g("n_query")),
                       int(g("vis_off")), int(g("aud_off")), int(g("qry_off")))
    return arr


def apack_score_dynamics_query(seqs, dim, params=None):
    arr = _av_array(seqs)
    p = _params(params)
    n = len(seqs)
    nk = (ctypes.c_int64 * max(1, n))()
    ws = ctypes.c_size_t(0)
    _check(library().apack_score_dynamics_query(n, arr, dim, ctypes.byref(p), nk, ctypes.byref(ws)))
    return [int(nk[i]) for i in range(n)], int(ws.value)


def apack_score_dynamics(visual, audio, query, seqs, params=None, workspace=None, stream=None):
    """Pre-LLM scorer over a packed batch of clips (Section 3.1).

    visual [rows, dim], audio [rows, dim], query [rows, dim] CUDA tensors
    (bf16 or f32); seqs: descriptors with n_frames, per_frame, n_audio,
    n_query, vis_off, aud_off, qry_off.  Returns a dict of the frame arrays,
    gate flags, kept visual rows and per-clip counts.
    """
    torch = _torch()
    dim = visual.shape[1]
    arr = _av_array(seqs)
    p = _params(params)
    n = len(seqs)
    nk = (ctypes.c_int64 * max(1, n))()
    wsb = ctypes.c_size_t(0)
    _check(library().apack_score_dynamics_query(n, arr, dim, ctypes.byref(p), nk, ctypes.byref(wsb)))
    total = sum(int(nk[i]) for i in range(n))
    frames = sum(int(arr[i].n_frames) for i in range(n))
    dev = visual.device
    with _alloc_on(stream):
        out = {
            "cka": torch.empty(max(frames, 1), dtype=torch.float32, device=dev),
            "score": torch.empty(max(frames, 1), dtype=torch.float32, device=dev),
            "budget": torch.empty(max(frames, 1), dtype=torch.int32, device=dev),
            "segment": torch.empty(max(frames, 1), dtype=torch.int32, device=dev),
            "gate": torch.empty(max(n, 1), dtype=torch.uint8, device=dev),
            "kept": torch.empty(max(total, 1), dtype=torch.int32, device=dev),
        }
        if workspace is None:
            workspace = _workspace(wsb.value, dev)
    for t, name in ((visual, "visual"), (audio, "audio"), (query, "query")):
        if t.dim() != 2 or t.stride(1) != 1 or t.stride(0) != dim:
            raise ApackError(2, f"{name} must be a contiguous [rows, dim] tensor")
    _check(library().apack_score_dynamics(
        n, arr, _dtype_code(visual), dim, _ptr(visual), visual.shape[0], _ptr(audio), audio.shape[0],
        _ptr(query), query.shape[0], ctypes.byref(p), _ptr(out["cka"]), _ptr(out["score"]),
        _ptr(out["budget"]), _ptr(out["segment"]), _ptr(out["gate"]), _ptr(out["kept"]),
        out["kept"].numel(), nk, _ptr(workspace), workspace.numel(), _stream(stream)))
    out["cka"] = out["cka"][:frames]
    out["score"] = out["score"][:frames]
    out["budget"] = out["budget"][:frames]
    out["segment"] = out["segment"][:frames]
    out["gate"] = out["gate"][:n]
    out["kept"] = out["kept"][:total]
    out["n_kept"] = [int(nk[i]) for i in range(n)]
    return out
