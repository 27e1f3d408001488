"""CPU-only checks of the C ABI: symbols, host helpers and validation paths.

Validation runs on the host before anything is enqueued, so every error path
can be forced here with fake device addresses: no call below reaches HIP.
"""

import ctypes
import math
import os
import re
from fractions import Fraction

import pytest

from oracle import prune as OP
from oracle import dynamics as OD
import paper_2608_08794_amd as A
from paper_2608_08794_amd import _lib as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    text = open(os.path.join(ROOT, "include", "apack.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(apack_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = A.library()
    names = _declared_functions()
    assert "apack_prune_layer" in names and "apack_compact_kv" in names and "apack_score_dynamics" in names
    for name in names:
        assert hasattr(lib, name), name
    assert b"gfx950" in lib.apack_version()


def test_keep_count_matches_oracle_decimal_ceiling():
    lib = A.library()
    for pct in range(0, 101, 5):
        keep = pct / 100.0
        for n in list(range(0, 2500)) + [7500, 8640, 17280, 60480, 86400, 93900, 94028, 200000]:
            assert lib.apack_keep_count(keep, n) == OP.keep_count(keep, n), (keep, n)
    for keep in (0.123456, 0.333333, 0.999999, 0.000001):
        for n in (1, 7, 999, 123457, 10**6, 10**8):
            assert lib.apack_keep_count(keep, n) == math.ceil(Fraction(str(keep)) * n), (keep, n)
    assert lib.apack_keep_count(-0.1, 10) == -1
    assert lib.apack_keep_count(1.5, 10) == -1
    assert lib.apack_keep_count(0.5, -1) == -1


def test_visual_budget_matches_oracle():
    lib = A.library()
    for r_pre in (0.35, 0.5, 0.51, 0.365, 0.1, 1.0, 0.0):
        for na, nv in ((1500, 17280), (7500, 86400), (500, 40), (0, 10), (10, 0)):
            assert lib.apack_visual_budget(r_pre, na, nv) == OD.visual_budget(r_pre, na, nv)


def test_default_params_are_table_s1():
    p = A.apack_dyn_params_default()
    got = {f: getattr(p, f) for f, _ in A.DynParams._fields_}
    for key, val in OD.DEFAULTS.items():
        if key == "alignment":   # the library numbers the scorers, the oracle names them
            assert got[key] == L.ALIGNMENTS[val] == 0
            continue
        assert got[key] == val, key
    assert sorted(L.ALIGNMENTS, key=L.ALIGNMENTS.get) == list(OD.ALIGNMENTS)


# -- validation paths (fake, never dereferenced device addresses) ------------

FAKE = 1 << 40


def _seq(spans, n, q_len=4, keep=(0.5, 0.5), basis=(0, 0), tok_off=0, q_off=0, flags=0):
    sp = (L.Span * max(1, len(spans)))(*[L.Span(b, l, m, 0) for b, l, m in spans])
    s = L.Seq(tok_off, n, sp, len(spans), flags, q_off, q_len,
              (ctypes.c_double * 2)(*keep), (ctypes.c_int64 * 2)(*basis))
    return s, sp


def _prune(seqs, hq=4, hkv=2, d=64, dtype=0, q=FAKE, k=FAKE + (1 << 34), scores=FAKE + (2 << 34),
           kept=FAKE + (3 << 34), cap=1 << 20, ws=FAKE + (4 << 34), ws_bytes=1 << 30,
           q_rows=1 << 12, k_rows=1 << 12, qhs=None, khs=None):
    arr = (L.Seq * max(1, len(seqs)))(*seqs)
    qhs = q_rows * d if qhs is None else qhs
    khs = k_rows * d if khs is None else khs
    nk = (ctypes.c_int64 * max(1, len(seqs)))()
    st = A.library().apack_prune_layer(len(seqs), arr, dtype, hq, hkv, d, q, qhs, q_rows, k, khs, k_rows,
                                       scores, kept, cap, nk, ws, ws_bytes, None)
    return st, A.library().apack_last_error().decode()


def test_prune_query_joint_counts_over_both_modalities():
    s, _sp = _seq([(0, 100, 1), (100, 300, 2)], 420, keep=(0.55, 0.0), flags=L.APACK_RANK_JOINT)
    arr = (L.Seq * 1)(s)
    nk = (ctypes.c_int64 * 1)()
    ws = ctypes.c_size_t(0)
    assert A.library().apack_prune_layer_query(1, arr, 8, 2, 128, nk, ctypes.byref(ws)) == 0
    assert nk[0] == 20 + OP.keep_count(0.55, 400)


def test_prune_query_reports_counts_and_workspace():
    s, _sp = _seq([(0, 100, 1), (100, 300, 2)], 420, keep=(0.55, 0.3))
    arr = (L.Seq * 1)(s)
    nk = (ctypes.c_int64 * 1)()
    ws = ctypes.c_size_t(0)
    assert A.library().apack_prune_layer_query(1, arr, 8, 2, 128, nk, ctypes.byref(ws)) == 0
    assert nk[0] == 20 + 55 + 90
    assert ws.value > 0 and ws.value % 256 == 0


@pytest.mark.parametrize("case,status", [
    ("hq_not_multiple", 2), ("bad_d", 7), ("bad_dtype", 3), ("span_outside", 2), ("span_unsorted", 2),
    ("bad_modality", 1), ("keep_range", 1), ("k_exceeds", 1), ("q_len0", 2), ("q_rows", 2),
    ("k_rows", 2), ("overlap_seqs", 2), ("small_ws", 4), ("misaligned_ws", 4), ("null_ws", 4),
    ("small_capacity", 2), ("alias", 5), ("bad_flags", 1), ("misaligned_q", 1), ("null_k", 1),
    ("joint_second_keep", 1), ("joint_second_basis", 1), ("joint_k_exceeds", 1),
])
def test_prune_validation_errors(case, status):
    s, sp = _seq([(0, 10, 1), (10, 20, 2)], 40)
    kw = {}
    seqs = [s]
    if case == "hq_not_multiple":
        kw = dict(hq=6, hkv=4)
    elif case == "bad_d":
        kw = dict(d=96)
    elif case == "bad_dtype":
        kw = dict(dtype=7)
    elif case == "span_outside":
        seqs = [_seq([(30, 20, 2)], 40)[0]]
    elif case == "span_unsorted":
        seqs = [_seq([(10, 5, 2), (0, 5, 1)], 40)[0]]
    elif case == "bad_modality":
        seqs = [_seq([(0, 5, 3)], 40)[0]]
    elif case == "keep_range":
        seqs = [_seq([(0, 5, 1)], 40, keep=(1.2, 0.5))[0]]
    elif case == "k_exceeds":
        seqs = [_seq([(0, 5, 1)], 40, keep=(0.5, 0.5), basis=(20, 0))[0]]
    elif case == "q_len0":
        seqs = [_seq([(0, 5, 1)], 40, q_len=0)[0]]
    elif case == "q_rows":
        kw = dict(q_rows=3)
    elif case == "k_rows":
        kw = dict(k_rows=39)
    elif case == "overlap_seqs":
        seqs = [s, _seq([(0, 10, 2)], 20, tok_off=30)[0]]
    elif case == "small_ws":
        kw = dict(ws_bytes=100)
    elif case == "misaligned_ws":
        kw = dict(ws=FAKE + (4 << 34) + 8)
    elif case == "null_ws":
        kw = dict(ws=None)
    elif case == "small_capacity":
        kw = dict(cap=5)
    elif case == "alias":
        kw = dict(scores=FAKE + (1 << 34) + 64)
    elif case == "bad_flags":
        seqs = [_seq([(0, 5, 1)], 40, flags=2)[0]]
    elif case == "joint_second_keep":
        seqs = [_seq([(0, 5, 1)], 40, keep=(0.5, 0.5), flags=1)[0]]
    elif case == "joint_second_basis":
        seqs = [_seq([(0, 5, 1)], 40, keep=(0.5, 0.0), basis=(0, 3), flags=1)[0]]
    elif case == "joint_k_exceeds":
        seqs = [_seq([(0, 5, 1), (5, 5, 2)], 40, keep=(0.5, 0.0), basis=(30, 0), flags=1)[0]]
    elif case == "misaligned_q":
        kw = dict(q=FAKE + 4)
    elif case == "null_k":
        kw = dict(k=None)
    st, msg = _prune(seqs, **kw)
    assert st == status, msg
    assert msg


def _compact(n_out=10, n_in=20, layers=1, src=FAKE, kin=None, kout=None, hid=(0, 0, 0), pos=(0, 0, 0),
             hkv=2, d=64, dtype=0, hs_in=None, hs_out=None, v_tables=(True, True)):
    P = ctypes.c_void_p * max(1, layers)
    base_in = FAKE + (1 << 34)
    base_out = FAKE + (8 << 34)
    kin = kin or [base_in + l * (1 << 30) for l in range(layers)]
    vin = [base_in + (1 << 33) + l * (1 << 30) for l in range(layers)]
    kout = kout or [base_out + l * (1 << 30) for l in range(layers)]
    vout = [base_out + (1 << 33) + l * (1 << 30) for l in range(layers)]
    hs_in = n_in * d if hs_in is None else hs_in
    hs_out = n_out * d if hs_out is None else hs_out
    vin_t = P(*vin) if v_tables[0] else None
    vout_t = P(*vout) if v_tables[1] else None
    st = A.library().apack_compact_kv(n_out, src, n_in, layers, P(*kin), vin_t, P(*kout), vout_t, hkv, d,
                                      dtype, hs_in, hs_out, hid[0], hid[1], hid[2], pos[0], pos[1], pos[2],
                                      n_in, n_out, None)
    return st, A.library().apack_last_error().decode()


@pytest.mark.parametrize("case,status", [
    ("alias_kv", 5), ("alias_outputs", 5), ("alias_hidden", 5), ("too_many_layers", 1), ("null_src", 1),
    ("bad_dtype", 3), ("stride", 2), ("null_hidden", 1), ("negative", 2), ("half_v_tables", 1),
    ("k_only_alias", 5),
])
def test_compact_validation_errors(case, status):
    kw = {}
    if case == "alias_kv":
        kw = dict(kout=[FAKE + (1 << 34) + 256])
    elif case == "alias_outputs":
        kw = dict(layers=2, kout=[FAKE + (8 << 34), FAKE + (8 << 34) + 512])
    elif case == "alias_hidden":
        kw = dict(hid=(FAKE + (20 << 34), FAKE + (20 << 34) + 64, 512))
    elif case == "too_many_layers":
        kw = dict(layers=65)
    elif case == "null_src":
        kw = dict(src=None)
    elif case == "bad_dtype":
        kw = dict(dtype=9)
    elif case == "stride":
        kw = dict(hs_in=5)
    elif case == "null_hidden":
        kw = dict(hid=(None, FAKE + (30 << 34), 64))
    elif case == "negative":
        kw = dict(n_out=-1)
    elif case == "half_v_tables":
        kw = dict(v_tables=(True, False))
    elif case == "k_only_alias":
        kw = dict(v_tables=(False, False), kout=[FAKE + (1 << 34) + 256])
    st, msg = _compact(**kw)
    assert st == status, msg
    assert msg


def test_compact_k_only_validates_without_device():
    st, msg = _compact(n_out=0, layers=3, v_tables=(False, False))
    assert st == 0, msg


def test_compact_with_nothing_to_copy_is_ok_without_device():
    st, msg = _compact(n_out=0)
    assert st == 0, msg


def _inplace(n_out=10, n_in=20, layers=1, src=FAKE, k=None, v=True, hid=(0, 0), pos=(0, 0, 0), hkv=2, d=64,
             dtype=0, hs=None, ws=FAKE + (40 << 34), ws_bytes=None):
    P = ctypes.c_void_p * max(1, layers)
    base = FAKE + (1 << 34)
    k = k or [base + l * (1 << 30) for l in range(layers)]
    vt = P(*[base + (1 << 33) + l * (1 << 30) for l in range(layers)]) if v else None
    hs = n_in * d if hs is None else hs
    need = A.apack_compact_kv_inplace_workspace(n_out)
    st = A.library().apack_compact_kv_inplace(n_out, src, n_in, layers, P(*k), vt, hkv, d, dtype, hs, hid[0],
                                              hid[1], pos[0], pos[1], pos[2], ws,
                                              need if ws_bytes is None else ws_bytes, None)
    return st, A.library().apack_last_error().decode()


def test_inplace_workspace_size_grows_with_stripes():
    f = A.apack_compact_kv_inplace_workspace
    assert f(-1) == 0
    assert 0 < f(0) <= f(1) == f(64) <= f(65) < f(10**6)
    assert f(10**6) % 256 == 0
    # A 64-byte counter line and a 4-byte reader index per 128 kept rows.
    stripes = -(-10**6 // 128)
    assert stripes * 68 <= f(10**6) <= stripes * 68 + 1024


@pytest.mark.parametrize("case,status", [
    ("more_out_than_in", 2), ("negative", 2), ("null_src", 1), ("bad_dtype", 3), ("stride", 2),
    ("too_many_pos_rows", 7), ("planes_overlap", 5), ("hidden_overlaps_kv", 5), ("src_in_plane", 5),
    ("ws_in_plane", 5), ("ws_over_src", 5), ("small_ws", 4), ("misaligned_ws", 4), ("null_ws", 4),
    ("null_pos", 1), ("too_many_layers", 1),
])
def test_inplace_validation_errors(case, status):
    kw = {}
    if case == "more_out_than_in":
        kw = dict(n_out=21)
    elif case == "negative":
        kw = dict(n_in=-1)
    elif case == "null_src":
        kw = dict(src=None)
    elif case == "bad_dtype":
        kw = dict(dtype=9)
    elif case == "stride":
        kw = dict(hs=64)
    elif case == "too_many_pos_rows":
        kw = dict(pos=(FAKE + (30 << 34), 17, 20))
    elif case == "planes_overlap":
        kw = dict(layers=2, k=[FAKE + (1 << 34), FAKE + (1 << 34) + 1024])
    elif case == "hidden_overlaps_kv":
        kw = dict(hid=(FAKE + (1 << 34) + 4096, 512))
    elif case == "src_in_plane":
        kw = dict(src=FAKE + (1 << 34) + 64)
    elif case == "ws_in_plane":
        kw = dict(ws=FAKE + (1 << 34) + 1024)
    elif case == "ws_over_src":
        kw = dict(src=FAKE + (40 << 34) + 256)
    elif case == "small_ws":
        kw = dict(ws_bytes=16)
    elif case == "misaligned_ws":
        kw = dict(ws=FAKE + (40 << 34) + 4)
    elif case == "null_ws":
        kw = dict(ws=None)
    elif case == "null_pos":
        kw = dict(pos=(None, 3, 20))
    elif case == "too_many_layers":
        kw = dict(layers=65)
    st, msg = _inplace(**kw)
    assert st == status, msg
    assert msg


def test_inplace_with_nothing_to_move_is_ok_without_device():
    assert _inplace(n_out=0, ws=None)[0] == 0
    assert _inplace(n_out=0, layers=0, v=False, ws=None)[0] == 0


def test_inplace_status_validation_without_device():
    lib = A.library()
    flag = ctypes.c_int32(7)
    assert lib.apack_compact_kv_inplace_status(FAKE, 1024, None, None) == 1
    assert lib.apack_compact_kv_inplace_status(None, 1024, ctypes.byref(flag), None) == 4
    assert lib.apack_compact_kv_inplace_status(FAKE + 8, 1024, ctypes.byref(flag), None) == 4
    assert lib.apack_compact_kv_inplace_status(FAKE, 4, ctypes.byref(flag), None) == 4
    assert flag.value == 7   # untouched on error


def test_inplace_static_rejects_more_rows_than_its_scratch_without_device():
    lib = A.library()
    tk = (ctypes.c_void_p * 1)(FAKE + (1 << 34))
    st = lib.apack_compact_kv_inplace_static((1 << 20) + 1, FAKE, (1 << 20) + 2, 1, tk, None, 1, 8, 0,
                                             (1 << 20) + 2 << 3, None, 0, None, 0, 0, None)
    assert st == 7 and "static scratch" in lib.apack_last_error().decode()
    # Nothing to move: returns before touching the device.
    assert lib.apack_compact_kv_inplace_static(0, None, 10, 0, None, None, 0, 0, 0, 0, None, 0, None, 0, 0, None) == 0


def test_inplace_wait_limit_round_trips():
    prev = A.apack_set_inplace_wait_limit(12345)
    try:
        assert prev == 1 << 22
        assert A.apack_set_inplace_wait_limit(0) == 12345
    finally:
        A.apack_set_inplace_wait_limit(prev)


# -- scorer validation (fake device addresses, never dereferenced) ----------

def _av(n_frames=8, per_frame=16, n_audio=100, n_query=4, vis_off=0, aud_off=0, qry_off=0):
    return L.AVSeq(n_frames, per_frame, n_audio, n_query, vis_off, aud_off, qry_off)


def _score(seqs, dim=64, dtype=0, params=None, vis=FAKE, vrows=128, aud=FAKE + (1 << 34), arows=100,
           qry=FAKE + (2 << 34), qrows=4, outs=None, cap=1 << 20, ws=FAKE + (4 << 34), ws_bytes=1 << 30):
    p = A.apack_dyn_params_default()
    for key, val in (params or {}).items():
        setattr(p, key, val)
    arr = (L.AVSeq * max(1, len(seqs)))(*seqs)
    base = FAKE + (8 << 34)
    outs = outs or [base + i * (1 << 30) for i in range(6)]
    nk = (ctypes.c_int64 * max(1, len(seqs)))()
    st = A.library().apack_score_dynamics(len(seqs), arr, dtype, dim, vis, vrows, aud, arows, qry, qrows,
                                          ctypes.byref(p), *outs, cap, nk, ws, ws_bytes, None)
    return st, A.library().apack_last_error().decode(), list(nk)


def test_score_query_reports_budgets_and_workspace():
    seqs = [_av(), _av(n_frames=30, per_frame=144, n_audio=750, vis_off=128, aud_off=100, qry_off=4)]
    arr = (L.AVSeq * 2)(*seqs)
    p = A.apack_dyn_params_default()
    nk = (ctypes.c_int64 * 2)()
    ws = ctypes.c_size_t(0)
    assert A.library().apack_score_dynamics_query(2, arr, 3584, ctypes.byref(p), nk, ctypes.byref(ws)) == 0
    assert list(nk) == [OD.visual_budget(0.5, 100, 128), OD.visual_budget(0.5, 750, 30 * 144)]
    assert ws.value > 0 and ws.value % 256 == 0


def test_score_empty_batch_is_ok_without_device():
    st, msg, _ = _score([])
    assert st == 0, msg


@pytest.mark.parametrize("case,status", [
    ("window0", 1), ("window17", 1), ("dafps_k", 1), ("sigma", 1), ("beta", 1), ("r_pre", 1), ("cover", 1),
    ("power", 1), ("tau_nan", 1), ("dim_odd", 2), ("dim_big", 2), ("per_frame", 2), ("no_audio", 2),
    ("no_query", 2), ("neg_off", 2), ("vis_rows", 2), ("aud_rows", 2), ("qry_rows", 2), ("capacity", 2),
    ("null_visual", 1), ("misaligned", 1), ("null_kept", 1), ("out_in", 5), ("out_out", 5), ("small_ws", 4),
    ("misaligned_ws", 4), ("null_ws", 4), ("dtype", 3), ("alignment", 1), ("alignment_neg", 1),
])
def test_score_validation_errors(case, status):
    kw = {}
    seqs = [_av()]
    base = FAKE + (8 << 34)
    outs = [base + i * (1 << 30) for i in range(6)]
    params = {"window0": {"window": 0}, "window17": {"window": 17}, "dafps_k": {"dafps_k": 33},
              "alignment": {"alignment": 4}, "alignment_neg": {"alignment": -1},
              "sigma": {"sigma": 0.0}, "beta": {"beta": 1.5}, "r_pre": {"r_pre": 1.01},
              "cover": {"cover_thresh": 1.5}, "power": {"dafps_power": -1.0},
              "tau_nan": {"tau_gate": float("nan")}}
    if case in params:
        kw = dict(params=params[case])
    elif case == "dim_odd":
        kw = dict(dim=100)
    elif case == "dim_big":
        kw = dict(dim=16392)
    elif case == "per_frame":
        seqs = [_av(per_frame=257)]
    elif case == "no_audio":
        seqs = [_av(n_audio=0)]
    elif case == "no_query":
        seqs = [_av(n_query=0)]
    elif case == "neg_off":
        seqs = [_av(aud_off=-1)]
    elif case == "vis_rows":
        kw = dict(vrows=127)
    elif case == "aud_rows":
        kw = dict(arows=99)
    elif case == "qry_rows":
        kw = dict(qrows=3)
    elif case == "capacity":
        kw = dict(cap=OD.visual_budget(0.5, 100, 128) - 1)
    elif case == "null_visual":
        kw = dict(vis=None)
    elif case == "misaligned":
        kw = dict(aud=FAKE + (1 << 34) + 8)
    elif case == "null_kept":
        outs[5] = None
        kw = dict(outs=outs)
    elif case == "out_in":
        outs[1] = FAKE + 64
        kw = dict(outs=outs)
    elif case == "out_out":
        outs[3] = outs[0] + 4
        kw = dict(outs=outs)
    elif case == "small_ws":
        kw = dict(ws_bytes=256)
    elif case == "misaligned_ws":
        kw = dict(ws=FAKE + (4 << 34) + 16)
    elif case == "null_ws":
        kw = dict(ws=None)
    elif case == "dtype":
        kw = dict(dtype=4)
    st, msg, nk = _score(seqs, **kw)
    assert st == status, (msg, case)
    assert msg


def test_spatial_alignment_sizes_its_tile_sums():
    # The spatial scorer needs per-frame tile sums; the other scorers do not.
    seqs = [_av(n_frames=30, per_frame=144, n_audio=375)]
    arr = (L.AVSeq * 1)(*seqs)
    sizes = {}
    for name, code in L.ALIGNMENTS.items():
        p = A.apack_dyn_params_default()
        p.alignment = code
        ws = ctypes.c_size_t(0)
        assert A.library().apack_score_dynamics_query(1, arr, 3584, ctypes.byref(p), None, ctypes.byref(ws)) == 0
        sizes[name] = ws.value
    assert sizes["gated_cka"] == sizes["cka"] == sizes["av_cosine"]
    # 13 or 14 audio rows + 144 visual rows -> 10 tiles a side, 55 tiles, 3 sums each, per frame.
    assert sizes["spatial_cka"] - sizes["gated_cka"] >= 30 * 55 * 3 * 8
