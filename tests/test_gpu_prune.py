"""GPU parity of the prune path (Section 3.2, Eq. 5-6) against the fp64 oracle.

Through the C ABI (ctypes binding): scores within the stated tolerance
(2e-3 relative for bf16 inputs, 1e-5 for fp32), kept rows and compacted
K/V/hidden/positions bit-exact.  The generators plant a score gap at every
top-k boundary; each case first certifies that gap with the oracle.
"""

import math
import zlib

import numpy as np
import pytest

import workloads as W
from oracle import prune as OP, widen
from tests.gpu_util import bits, log, raw_bits, score_tol, to_dev

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_08794_amd as A
    A.library()


def _run_prune(case, seqs=None):
    import paper_2608_08794_amd as A
    seqs = seqs or case.seqs
    q = to_dev(case.q, case.dtype)
    k = to_dev(case.k, case.dtype)
    scores, kept, n_kept = A.apack_prune_layer(q, k, seqs)
    torch.cuda.synchronize()
    return scores.cpu().numpy(), kept.cpu().numpy().astype(np.int64), n_kept


def _oracle(case, seqs=None):
    seqs = seqs or case.seqs
    sd = [dict(tok_off=s.tok_off, n_tokens=s.n_tokens, q_off=s.q_off, q_len=s.q_len, tags=s.tags(),
               keep=s.keep, keep_basis=s.keep_basis, joint=s.joint) for s in seqs]
    return OP.prune_batch(widen(case.q, case.dtype), widen(case.k, case.dtype), sd)


def _check_scores(got, want, seqs, dtype):
    tol = score_tol(dtype)
    for s in seqs:
        sl = slice(s.tok_off, s.tok_off + s.n_tokens)
        tags = s.tags()
        g, w = got[sl], want[sl]
        assert np.all(g[tags == 0] == 0.0)
        c = tags != 0
        if c.any():
            rel = np.abs(g[c] - w[c]) / np.abs(w[c])
            assert rel.max() <= tol, f"max rel err {rel.max():.3g} > {tol}"


def _parity(case, seqs=None, min_margin=1e-2):
    seqs = seqs or case.seqs
    log(f"[prune] {case.name} dtype={case.dtype} hq={case.hq} hkv={case.hkv} d={case.d} "
        f"rows={case.k.shape[1]} seqs={len(seqs)}")
    w_scores, w_kept, w_n, margins = _oracle(case, seqs)
    if min_margin:
        assert min(margins) >= min_margin, margins
    g_scores, g_kept, g_n = _run_prune(case, seqs)
    assert g_n == w_n
    np.testing.assert_array_equal(g_kept, w_kept)
    _check_scores(g_scores, w_scores, seqs, case.dtype)
    return g_kept


@pytest.mark.parametrize("fn", [W.prune_cfg1, W.prune_cfg2, W.prune_cfg3])
def test_prune_parity_configs_1_to_3(fn):
    _parity(fn())


def _compact_and_check(cache, kept_rows, n_in):
    import paper_2608_08794_amd as A
    dt = cache.dtype
    src = torch.from_numpy(kept_rows.astype(np.int32)).cuda()
    k_in = [to_dev(x, dt) for x in cache.k_layers]
    v_in = [to_dev(x, dt) for x in cache.v_layers]
    n_out = kept_rows.size
    k_out = [torch.empty((cache.hkv, n_out, cache.d), dtype=k_in[0].dtype, device="cuda") for _ in k_in]
    v_out = [torch.empty_like(x) for x in k_out]
    h_in = to_dev(cache.hidden, dt) if cache.hidden is not None else None
    h_out = torch.empty((n_out, cache.hidden_dim), dtype=h_in.dtype, device="cuda") if h_in is not None else None
    p_in = torch.from_numpy(cache.pos).cuda() if cache.pos is not None else None
    p_out = torch.empty((3, n_out), dtype=torch.int32, device="cuda") if p_in is not None else None
    A.apack_compact_kv(src, n_in, k_in, v_in, k_out, v_out, h_in, h_out, p_in, p_out)
    torch.cuda.synchronize()
    for l in range(len(k_in)):
        np.testing.assert_array_equal(bits(k_out[l]), raw_bits(cache.k_layers[l], dt)[:, kept_rows])
        np.testing.assert_array_equal(bits(v_out[l]), raw_bits(cache.v_layers[l], dt)[:, kept_rows])
    if h_in is not None:
        np.testing.assert_array_equal(bits(h_out), raw_bits(cache.hidden, dt)[kept_rows])
    if p_in is not None:
        np.testing.assert_array_equal(p_out.cpu().numpy(), cache.pos[:, kept_rows])


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_prune_then_compact_configs_1_to_3(cfg):
    case = {1: W.prune_cfg1, 2: W.prune_cfg2, 3: W.prune_cfg3}[cfg]()
    kept = _parity(case)
    cache = W.cfg_cache(cfg, case)
    log(f"[compact] cfg{cfg} rows {case.k.shape[1]} -> {kept.size}")
    _compact_and_check(cache, kept, case.k.shape[1])


def test_compact_k_only_planes():
    # v_in / v_out empty: only the tensors passed as K move (here a K plane
    # and a V plane in the K slots), bit-exactly.
    import paper_2608_08794_amd as A
    case = W.prune_cfg2()
    kept = _parity(case)
    cache = W.cfg_cache(2, case)
    planes_in = [to_dev(cache.k_layers[0], "bf16"), to_dev(cache.v_layers[0], "bf16")]
    src = torch.from_numpy(kept.astype(np.int32)).cuda()
    outs = [torch.empty((x.shape[0], kept.size, x.shape[2]), dtype=x.dtype, device="cuda") for x in planes_in]
    A.apack_compact_kv(src, case.k.shape[1], planes_in, (), outs, ())
    torch.cuda.synchronize()
    np.testing.assert_array_equal(bits(outs[0]), raw_bits(cache.k_layers[0], "bf16")[:, kept])
    np.testing.assert_array_equal(bits(outs[1]), raw_bits(cache.v_layers[0], "bf16")[:, kept])


def _src_rows(kind, n_in, rng):
    """Strictly increasing kept rows of several shapes."""
    if kind == "all":
        return np.arange(n_in)
    if kind == "none":
        return np.zeros(0, np.int64)
    if kind == "one_last":
        return np.array([n_in - 1])
    if kind == "prefix_then_sparse":   # an untouched prefix, then rows far behind their readers
        p = n_in // 3
        return np.concatenate([np.arange(p), np.sort(rng.choice(np.arange(p, n_in), (n_in - p) // 4, replace=False))])
    if kind == "drop_first":
        return np.arange(1, n_in)
    return np.sort(rng.choice(n_in, max(1, int(n_in * float(kind))), replace=False))


@pytest.mark.parametrize("dtype,d,hid,prows,layers,n_in,kind,strided,k_only", [
    ("bf16", 128, 512, 3, 2, 1000, "0.5", False, False),
    ("bf16", 128, 3584, 3, 1, 5000, "prefix_then_sparse", False, False),
    ("bf16", 128, 256, 3, 1, 777, "all", False, False),
    ("bf16", 128, 256, 3, 1, 64, "drop_first", False, False),
    ("bf16", 128, 256, 3, 1, 65, "one_last", False, False),
    ("bf16", 128, 256, 3, 1, 1, "all", False, False),
    ("bf16", 128, 256, 3, 1, 300, "none", False, False),
    ("bf16", 256, 0, 0, 2, 2000, "0.3", True, False),      # two slices per row, strided heads
    ("bf16", 8, 24, 16, 1, 3000, "0.9", False, False),     # one-unit rows, 16 position rows
    ("f32", 3, 5, 1, 1, 1500, "0.7", False, False),        # 4-byte units
    ("f32", 64, 100, 2, 3, 2500, "0.1", True, True),       # K planes only
])
def test_inplace_compaction_matches_gather(dtype, d, hid, prows, layers, n_in, kind, strided, k_only):
    """Rows [0, n_out) equal the oracle's gather of the original rows, rows
    [n_out, n_in) keep their contents, bit for bit; the second call reuses
    the workspace on the compacted cache."""
    import paper_2608_08794_amd as A
    rng = np.random.default_rng(zlib.crc32(repr((dtype, d, n_in, kind)).encode()))
    hkv = 3
    pad = 17 if strided else 0
    cpu = dict(k=[W.payload_bits(rng, (hkv, n_in + pad, d), dtype) for _ in range(layers)],
               v=[] if k_only else [W.payload_bits(rng, (hkv, n_in + pad, d), dtype) for _ in range(layers)],
               h=W.payload_bits(rng, (n_in, hid), dtype) if hid else None,
               p=rng.integers(-2**31, 2**31, size=(prows, n_in + pad), dtype=np.int64).astype(np.int32)
               if prows else None)
    dev = dict(k=[to_dev(x, dtype)[:, :n_in] for x in cpu["k"]], v=[to_dev(x, dtype)[:, :n_in] for x in cpu["v"]],
               h=to_dev(cpu["h"], dtype) if hid else None,
               p=torch.from_numpy(cpu["p"]).cuda()[:, :n_in] if prows else None)
    want = {key: ([x[..., :n_in, :] for x in val] if key in "kv" else val) for key, val in cpu.items()}
    if prows:
        want["p"] = cpu["p"][:, :n_in]
    ws = None
    n = n_in
    for step in range(2):
        src = _src_rows(kind if step == 0 else "0.6", n, rng) if n else np.zeros(0, np.int64)
        log(f"[inplace] {dtype} d={d} hid={hid} pos={prows} layers={layers} step {step}: {n} -> {src.size} ({kind})")
        if ws is None:
            ws = torch.empty(max(256, A.apack_compact_kv_inplace_workspace(src.size)), dtype=torch.uint8,
                             device="cuda")
        A.apack_compact_kv_inplace(torch.from_numpy(src.astype(np.int32)).cuda(), n,
                                   [x[:, :n] for x in dev["k"]], [x[:, :n] for x in dev["v"]],
                                   dev["h"][:n] if hid else None, dev["p"][:, :n] if prows else None, workspace=ws)
        torch.cuda.synchronize()
        m = src.size

        def moved(x, axis):
            y = x.copy()
            idx = [slice(None)] * x.ndim
            idx[axis] = slice(0, m)
            y[tuple(idx)] = OP.compact_rows(x, src, axis=axis)
            return y

        want = dict(k=[moved(x, 1) for x in want["k"]], v=[moved(x, 1) for x in want["v"]],
                    h=moved(want["h"], 0) if hid else None, p=moved(want["p"], 1) if prows else None)
        for l in range(layers):
            np.testing.assert_array_equal(bits(dev["k"][l]), raw_bits(want["k"][l], dtype))
            if not k_only:
                np.testing.assert_array_equal(bits(dev["v"][l]), raw_bits(want["v"][l], dtype))
        if strided:   # the padding rows past n_in stay untouched
            for l in range(layers):
                t = dev["k"][l]
                tail = t.as_strided((hkv, pad, d), t.stride(), t.storage_offset() + n_in * d)
                np.testing.assert_array_equal(bits(tail), raw_bits(cpu["k"][l], dtype)[:, n_in:])
        if hid:
            np.testing.assert_array_equal(bits(dev["h"]), raw_bits(want["h"], dtype))
        if prows:
            np.testing.assert_array_equal(dev["p"].cpu().numpy(), want["p"])
        n = m
        if n == 0:
            break


# -- edge cases ---------------------------------------------------------------


def _synthetic(dtype, hq, hkv, d, seq_specs, seed, zero_keys=False, dup=None, lift=True, joint=(), bases=None):
    """Small packed batch.  seq_specs: list of (spans, n_tokens, q_len, keep);
    sequences listed in ``joint`` rank S jointly with keep[0], and ``bases``
    maps a sequence to its keep basis.  With ``lift`` each sequence's top set
    (per modality, or joint) is planted with a certified gap."""
    rng = np.random.default_rng(seed)
    seqs, tok, qrow = [], 0, 0
    for i, (spans, n, ql, keep) in enumerate(seq_specs):
        basis = (bases or {}).get(i, (0, 0))
        seqs.append(W.PruneSeq(tok, n, spans, qrow, ql, keep, basis, i in joint))
        tok += n
        qrow += ql
    scale = 1.0 if dtype == "f32" else 1.0 / math.sqrt(d)
    qf = rng.standard_normal((hq, max(qrow, 1), d), dtype=np.float32) * np.float32(scale)
    kf = rng.standard_normal((hkv, max(tok, 1), d), dtype=np.float32) * np.float32(scale)
    top = {}
    if lift and not zero_keys:
        qv = W.bf16_bits_to_f32(W.to_bf16_bits(qf)) if dtype == "bf16" else qf
        for i, s in enumerate(seqs):
            if s.joint:
                cand = np.flatnonzero(s.tags() != 0)
                n = s.keep_basis[0] or cand.size
                topi = {"joint": np.sort(rng.choice(cand, size=OP.keep_count(s.keep[0], n), replace=False))}
                rows = topi["joint"]
            else:
                topi = W._planted_sets(rng, s.tags(), s.keep, s.keep_basis)
                rows = np.concatenate([topi[1], topi[2]]).astype(np.int64)
            top[i] = topi
            if s.q_len == 0:
                continue
            dirs = W._group_unit_dirs(qv[:, s.q_off:s.q_off + s.q_len], hkv)
            if dtype == "f32":
                n_rep = hq // hkv
                for g in range(hkv):
                    qf[g * n_rep:(g + 1) * n_rep, s.q_off:s.q_off + s.q_len] += np.float32(3.0) * dirs[g]
                W._lift(kf[:, s.tok_off:s.tok_off + s.n_tokens], dirs, rows, 8.0)
            else:
                W._lift(kf[:, s.tok_off:s.tok_off + s.n_tokens], dirs, rows, W.LIFT_BF16_BOUNDARY)
    if zero_keys:
        kf[:] = 0
    if dup is not None:
        for a, b in dup:
            kf[:, b] = kf[:, a]
    q = W.to_bf16_bits(qf) if dtype == "bf16" else qf
    k = W.to_bf16_bits(kf) if dtype == "bf16" else kf
    return W.PruneCase("synthetic", dtype, hq, hkv, d, q, k, seqs, top)


A_, V_, O_ = 1, 2, 0


@pytest.mark.parametrize("dtype,d", [("bf16", 64), ("bf16", 128), ("f32", 64), ("f32", 128)])
def test_ragged_batch_interleaved_spans(dtype, d):
    specs = [
        ([(0, 50, V_), (50, 13, A_), (63, 70, V_), (133, 12, A_)], 160, 9, (0.5, 0.3)),
        ([(3, 200, A_), (210, 333, V_)], 560, 1, (0.35, 0.8)),          # paper's single query row
        ([], 17, 5, (0.5, 0.5)),                                        # no candidates
        ([(0, 0, A_)], 0, 3, (0.5, 0.5)),                               # empty sequence
        ([(0, 700, V_), (700, 64, A_)], 800, 100, (0.7, 0.15)),         # 700 rows per group: 2 row groups
    ]
    case = _synthetic(dtype, 14, 2, d, specs, seed=11)
    _parity(case)


@pytest.mark.parametrize("dtype,hq,hkv,d,q_len,n", [("bf16", 28, 4, 128, 32, 30011), ("bf16", 8, 2, 128, 40, 40013),
                                                     ("f32", 8, 2, 64, 48, 40013)])
def test_four_wave_workgroups_over_four_stages(dtype, hq, hkv, d, q_len, n):
    # Up to four waves of query rows per group (here 224, 160 and 192 rows)
    # run four-wave workgroups whose key tiles stream through four LDS stages
    # (bf16, and f32 at head dim 64); at these lengths each workgroup's key
    # chunk is three or four tiles, the last one ragged.
    specs = [([(0, 8000, A_), (8000, n - 8200, V_)], n, q_len, (0.5, 0.3))]
    case = _synthetic(dtype, hq, hkv, d, specs, seed=18)
    _parity(case)


@pytest.mark.parametrize("hq,hkv,q_len", [(8, 2, 32), (28, 4, 8), (28, 4, 1)])
def test_row_partials_merged_by_several_threads_per_row(hq, hkv, q_len):
    # Pass 2 starts by combining each query row's per-chunk (max, sum)
    # partials from pass 1.  With 128 rows per group (here 4 x 32) two
    # threads of the four-wave workgroup share a row, with 56 or 7 rows four
    # do, each merging a contiguous run of the chunks before the
    # runs are combined in order (63 to 105 key chunks per group here).
    n = 40013
    specs = [([(0, 8000, A_), (8000, n - 8200, V_)], n, q_len, (0.5, 0.3))]
    case = _synthetic("bf16", hq, hkv, 128, specs, seed=23)
    _parity(case)


@pytest.mark.parametrize("q_len,seed", [(16, 20), (112, 19)])
def test_row_sums_redone_when_a_logit_overflows_the_reference(q_len, seed):
    # Pass 1 sums each query row's exponentials against a fixed reference
    # (its running maximum after the first tile, plus 64) and redoes the
    # chunk with the online maximum when a sum overflows.  One key of KV
    # group 0, in the third tile of its chunk, is set along the first query
    # row so that its logit is ~170-190 (natural units) above the rest: the
    # reference sum of that row overflows and the workgroup (one or seven row
    # waves) takes the second pass.  Scores and kept rows match the oracle.
    n = 40013
    specs = [([(0, 8000, A_), (8000, n - 8200, V_)], n, q_len, (0.5, 0.3))]
    case = _synthetic("bf16", 8, 2, 128, specs, seed=seed)
    q = widen(case.q, "bf16")
    u = q[0, 0] / np.linalg.norm(q[0, 0])
    row = 384 * 10 + 300          # chunks of 384 keys at this length: chunk 10, tile 2
    case.k[0, row] = W.to_bf16_bits((2000.0 * u).astype(np.float32))
    logit = float(q[0, 0] @ widen(case.k, "bf16")[0, row]) / math.sqrt(case.d)
    assert logit > 150.0
    _parity(case)


def test_reference_sums_start_late_after_non_candidate_runs():
    # Chunks whose first tiles hold only non-candidate rows (300 text rows at
    # the start, a 700-row text run in the middle): a wave keeps the online
    # maximum until every lane has seen a candidate key, which here happens
    # one or more tiles into its chunk.
    n = 40013
    spans = [(300, 9000, A_), (10000, n - 10200, V_)]
    case = _synthetic("bf16", 28, 4, 128, [(spans, n, 64, (0.5, 0.3))], seed=21)
    _parity(case)


def test_exact_ties_keep_lowest_rows():
    specs = [([(0, 100, A_), (100, 250, V_)], 400, 7, (0.33, 0.5))]
    case = _synthetic("bf16", 8, 2, 128, specs, seed=12, zero_keys=True)
    w_scores, w_kept, _, _ = _oracle(case)
    g_scores, g_kept, _ = _run_prune(case)
    tags = case.seqs[0].tags()
    # every candidate score is bitwise identical on the GPU
    assert len(set(g_scores[tags != 0].tolist())) == 1
    np.testing.assert_array_equal(g_kept, w_kept)
    assert w_kept.tolist() == list(range(0, 33)) + list(range(100, 225)) + list(range(350, 400))


def test_duplicate_keys_straddling_the_boundary():
    # The lowest-scoring planted audio row `a` gets a twin `b` outside the
    # planted set: the twins tie exactly at the k boundary and the lower row
    # must win.
    spec = [([(0, 64, A_), (64, 128, V_)], 200, 16, (0.5, 0.5))]
    base = _synthetic("bf16", 8, 2, 128, spec, seed=13)
    sc, _, _, _ = _oracle(base)
    top = base.planted[0][A_]
    a = int(top[np.argmin(sc[top])])
    b = int([r for r in range(64) if r not in set(top.tolist())][0])
    case = _synthetic("bf16", 8, 2, 128, spec, seed=13, dup=[(a, b)])
    w_scores, w_kept, _, _ = _oracle(case)
    assert w_scores[a] == w_scores[b]
    assert (min(a, b) in w_kept) and (max(a, b) not in w_kept)
    g_scores, g_kept, _ = _run_prune(case)
    assert g_scores[a] == g_scores[b]
    np.testing.assert_array_equal(g_kept, w_kept)
    _check_scores(g_scores, w_scores, case.seqs, "bf16")


def test_keep_zero_and_keep_all():
    specs = [([(0, 90, A_), (90, 310, V_)], 420, 12, (0.0, 1.0)),
             ([(0, 90, A_), (90, 310, V_)], 420, 12, (1.0, 0.0))]
    case = _synthetic("bf16", 4, 4, 128, specs, seed=14, lift=False)
    _parity(case, min_margin=0)


def test_cumulative_keep_basis():
    """Counts against the original modality lengths (400 audio, 700 visual
    rows before an earlier prune): 120 of the 300 audio and 210 of the 500
    visual rows are kept, planted with a certified gap."""
    case = _synthetic("bf16", 8, 2, 128, [([(0, 300, A_), (300, 500, V_)], 830, 20, (0.3, 0.3))], seed=15,
                      bases={0: (400, 700)})
    kept = _parity(case)
    assert kept.size == 30 + 120 + 210
    want = np.sort(np.concatenate([case.planted[0][A_], case.planted[0][V_], np.arange(800, 830)]))
    np.testing.assert_array_equal(kept, want)


def test_long_sequence_beyond_register_resident_select():
    # 120k rows: longer than the fused select-and-scan kernel holds in
    # registers, so the streaming select and scan kernels run.
    specs = [([(0, 20000, A_), (20000, 99000, V_)], 120000, 3, (0.4, 0.25))]
    case = _synthetic("bf16", 2, 1, 64, specs, seed=16)
    _parity(case)


@pytest.mark.parametrize("n", [16384, 16385])
@pytest.mark.parametrize("ties", [False, True])
def test_select_paths_meet_at_16384_rows(n, ties):
    # Sequences of up to 16384 rows are selected by one workgroup each;
    # longer ones by the tiled kernels.  Both must keep the same rows, with
    # all-equal scores (every key zero) ranked by row.
    specs = [([(0, 3000, A_), (3000, n - 3100, V_)], n, 5, (0.45, 0.3))]
    case = _synthetic("bf16", 4, 1, 64, specs, seed=17, zero_keys=ties)
    if not ties:
        _parity(case)
        return
    w_scores, w_kept, _, _ = _oracle(case)
    g_scores, g_kept, _ = _run_prune(case)
    np.testing.assert_array_equal(g_kept, w_kept)
    k_a, k_v = OP.keep_count(0.45, 3000), OP.keep_count(0.3, n - 3100)
    assert w_kept.tolist() == list(range(k_a)) + list(range(3000, 3000 + k_v)) + list(range(n - 100, n))


# -- Eq. 6 as written: one TopK over S, last query token only ----------------


def test_joint_ranking_last_query_7b_layer():
    _parity(W.prune_joint_layer())


def test_joint_and_per_modality_sequences_in_one_batch():
    # A jointly ranked sequence next to a per-modality one, interleaved spans.
    # Both sequences carry a planted top set (joint for the first), so the
    # kept sets are certified by a gap >= 1e-2.
    specs = [([(0, 60, V_), (60, 40, A_), (100, 90, V_)], 230, 1, (0.85, 0.0)),
             ([(0, 300, A_), (300, 500, V_)], 900, 3, (0.6, 0.25))]
    case = _synthetic("bf16", 28, 4, 128, specs, seed=41, joint=(0,))
    kept = _parity(case)
    s0, s1 = case.seqs
    want0 = np.sort(np.concatenate([case.planted[0]["joint"], np.arange(190, 230)]))
    want1 = s1.tok_off + np.sort(np.concatenate([case.planted[1][A_], case.planted[1][V_], np.arange(800, 900)]))
    np.testing.assert_array_equal(kept, np.concatenate([want0, want1]))


def test_paper_schedule_every_layer_from_l_mid():
    """Algorithm 1's loop: every layer from the first prune layer on keeps
    the top ceil((1-P)|S|) jointly; each step compacts every layer's K/V, the
    hidden states and the positions, and the next step scores the compacted
    cache."""
    import paper_2608_08794_amd as A
    pc = W.paper_schedule_case(n_audio=1500, n_frames=120, n_text=64, n_layers=6, first_layer=2, drop=0.15,
                               hidden_dim=512)
    log(f"[schedule] layers {pc.prune_layers}, drop 0.15")
    n = pc.seq().n_tokens
    tags_all = pc.seq().tags()
    kd = [to_dev(x, "bf16") for x in pc.cache.k_layers]
    vd = [to_dev(x, "bf16") for x in pc.cache.v_layers]
    hd = to_dev(pc.cache.hidden, "bf16")
    pd = torch.from_numpy(pc.cache.pos).cuda()
    rows = np.arange(n)
    gpu_kept, oracle_kept = [], []
    for i, layer in enumerate(pc.prune_layers):
        tags = tags_all[rows]
        spans, b = [], 0
        while b < rows.size:   # maximal runs of one tag in the current order
            e = b
            while e < rows.size and tags[e] == tags[b]:
                e += 1
            if tags[b] != 0:
                spans.append((b, e - b, int(tags[b])))
            b = e
        seq = W.PruneSeq(0, rows.size, spans, 0, 1, (pc.keeps[i], 0.0), (0, 0), True)
        q = to_dev(pc.queries[i], "bf16")
        scores, kept, n_kept = A.apack_prune_layer(q, kd[layer], [seq])
        r = OP.prune_sequence(widen(pc.queries[i], "bf16"), widen(pc.cache.k_layers[layer], "bf16")[:, rows],
                              tags, (pc.keeps[i], 0.0), joint=True)
        assert r["margin"] >= 1e-2
        np.testing.assert_array_equal(kept.cpu().numpy().astype(np.int64), r["kept"])
        m = kept.numel()
        ko = [torch.empty((x.shape[0], m, x.shape[2]), dtype=x.dtype, device="cuda") for x in kd]
        vo = [torch.empty_like(x) for x in ko]
        ho = torch.empty((m, hd.shape[1]), dtype=hd.dtype, device="cuda")
        po = torch.empty((3, m), dtype=torch.int32, device="cuda")
        A.apack_compact_kv(kept, rows.size, kd, vd, ko, vo, hd, ho, pd, po)
        torch.cuda.synchronize()
        rows = rows[r["kept"]]
        for l in range(len(kd)):
            np.testing.assert_array_equal(bits(ko[l]), raw_bits(pc.cache.k_layers[l], "bf16")[:, rows])
        np.testing.assert_array_equal(bits(ho), raw_bits(pc.cache.hidden, "bf16")[rows])
        np.testing.assert_array_equal(po.cpu().numpy(), pc.cache.pos[:, rows])
        kd, vd, hd, pd = ko, vo, ho, po
        gpu_kept.append(n_kept[0])
        oracle_kept.append(r["kept"].size)
        log(f"  layer {layer}: {n_kept[0]} rows kept")
    # Appendix G accounting of the schedule the path produced: the library's
    # ratio from the GPU's kept counts equals the oracle's from its own.
    from oracle import flops as OF
    T, d, m = len(pc.cache.k_layers), 3584, 18944
    lengths = A.apack_schedule_lengths(T, n, list(pc.prune_layers), gpu_kept)
    assert lengths == OF.step_schedule(T, n, list(pc.prune_layers), oracle_kept)
    _, ratio = A.apack_prefill_flops(lengths, n, d, m)
    assert ratio == pytest.approx(float(OF.flops_ratio(lengths, n, d, m)), rel=1e-13)


def test_prune_and_compaction_are_deterministic():
    """Two runs of the 7B post-scorer layer (cross-workgroup partial sums,
    arrival counters, radix histograms) give bit-identical scores, kept rows
    and compacted tensors."""
    import paper_2608_08794_amd as A
    case = W.prune_cfg3()
    cache = W.cfg_cache(3, case)
    q, k = to_dev(case.q, "bf16"), to_dev(case.k, "bf16")
    v = to_dev(cache.v_layers[0], "bf16")
    h = to_dev(cache.hidden, "bf16")
    runs = []
    for _ in range(2):
        scores, kept, n_kept = A.apack_prune_layer(q, k, case.seqs)
        m = n_kept[0]
        ko, vo = (torch.empty((case.hkv, m, case.d), dtype=torch.bfloat16, device="cuda") for _ in range(2))
        ho = torch.empty((m, h.shape[1]), dtype=torch.bfloat16, device="cuda")
        A.apack_compact_kv(kept, case.k.shape[1], [k], [v], [ko], [vo], h, ho)
        torch.cuda.synchronize()
        runs.append([bits(t) for t in (scores, kept, ko, vo, ho)])
    for name, a, b in zip(("scores", "kept", "k", "v", "hidden"), *runs):
        assert np.array_equal(a, b), name


def test_inplace_give_up_is_reported_and_stores_nothing():
    """With the wait bound at 0 every ordering wait gives up at once (no
    kernel spins): the status call reports it, and no ticket that gave up
    stored anything, so rows whose readers sat in earlier stripes keep their
    old contents.  Back at the default bound the same call is exact and the
    status is clear."""
    import paper_2608_08794_amd as A
    rng = np.random.default_rng(77)
    n_in, hkv, d = 5000, 3, 128
    plane = W.payload_bits(rng, (hkv, n_in, d), "bf16")
    src = np.sort(rng.choice(n_in, 1500, replace=False))
    ws = torch.empty(A.apack_compact_kv_inplace_workspace(src.size), dtype=torch.uint8, device="cuda")
    idx = torch.from_numpy(src.astype(np.int32)).cuda()
    prev = A.apack_set_inplace_wait_limit(0)
    try:
        x = to_dev(plane, "bf16")
        A.apack_compact_kv_inplace(idx, n_in, [x], workspace=ws)
        assert A.apack_compact_kv_inplace_status(ws)
    finally:
        assert A.apack_set_inplace_wait_limit(prev) == 0
    got = bits(x)
    moved = OP.compact_rows(plane, src, axis=1)
    # Each output row of each head plane (one work item's unit here) is
    # either moved or untouched, never anything else.
    for h in range(hkv):
        for r in range(src.size):
            assert np.array_equal(got[h, r], moved[h, r]) or np.array_equal(got[h, r], plane[h, r]), (h, r)
    assert not np.array_equal(got[:, :src.size], moved)
    assert np.array_equal(got[:, src.size:], plane[:, src.size:])
    x = to_dev(plane, "bf16")
    A.apack_compact_kv_inplace(idx, n_in, [x], workspace=ws)
    assert not A.apack_compact_kv_inplace_status(ws)
    assert np.array_equal(bits(x)[:, :src.size], moved)


def test_entry_points_on_a_side_stream():
    """Every entry point enqueued on a stream other than torch's current one,
    with the binding allocating outputs and workspaces: results match the
    oracle (the allocations are made on that stream, so their memory is not
    handed out again while the call runs)."""
    import paper_2608_08794_amd as A
    side = torch.cuda.Stream()
    case = W.prune_cfg2()
    cache = W.cfg_cache(2, case)
    w_scores, w_kept, w_n, _ = _oracle(case)
    q, k = to_dev(case.q, "bf16"), to_dev(case.k, "bf16")
    v = to_dev(cache.v_layers[0], "bf16")
    torch.cuda.synchronize()
    with torch.cuda.stream(torch.cuda.Stream()):   # the current stream is yet another one
        scores, kept, n_kept = A.apack_prune_layer(q, k, case.seqs, stream=side)
        side.synchronize()
        junk = [torch.full((1 << 20,), 7, dtype=torch.int32, device="cuda") for _ in range(8)]
        m = n_kept[0]
        vo = torch.empty((case.hkv, m, case.d), dtype=torch.bfloat16, device="cuda")
        A.apack_compact_kv(kept, case.k.shape[1], [v], (), [vo], (), stream=side)
        xi = v.clone()
        torch.cuda.current_stream().synchronize()
        A.apack_compact_kv_inplace(kept, case.k.shape[1], [xi], stream=side)
        dyn = W.dynamics_small("offset")
        xv, xa, xq = (to_dev(x, "bf16") for x in (dyn.xv, dyn.xa, dyn.xq))
        torch.cuda.current_stream().synchronize()
        got = A.apack_score_dynamics(xv, xa, xq, dyn.seqs, dyn.params, stream=side)
        side.synchronize()
        del junk
    assert n_kept == w_n
    np.testing.assert_array_equal(kept.cpu().numpy().astype(np.int64), w_kept)
    _check_scores(scores.cpu().numpy(), w_scores, case.seqs, "bf16")
    np.testing.assert_array_equal(bits(vo), raw_bits(cache.v_layers[0], "bf16")[:, w_kept])
    np.testing.assert_array_equal(bits(xi)[:, :m], raw_bits(cache.v_layers[0], "bf16")[:, w_kept])
    from oracle import dynamics as OD
    s = dyn.seqs[0]
    r = OD.score_sequence(widen(dyn.xv, "bf16"), widen(dyn.xa, "bf16"), widen(dyn.xq, "bf16"), s.n_frames,
                          s.per_frame, dyn.params)
    np.testing.assert_array_equal(got["kept"].cpu().numpy().astype(np.int64), r["kept"])
    np.testing.assert_array_equal(got["budget"].cpu().numpy(), r["frame_budget"])
