"""GPU parity of the pre-LLM scorer (Section 3.1, Eq. 1-4; Algorithm 1)
against the fp64 oracle, through the C ABI.

Discrete outputs (gate, segment ids, frame budgets, kept visual rows) must
be bit-exact; frame CKA and frame scores are fp32 casts of fp64 values and
must agree to fp32 resolution (1e-5 relative where the fp32 gate GEMM feeds
them).  Each case first certifies with the oracle that every decision sits
away from its boundary (1e-9 for fp64 decisions, 1e-4 downstream of the
fp32 gate GEMM).
"""

import numpy as np
import pytest

import workloads as W
from oracle import dynamics as OD, widen
from tests.gpu_util import log, to_dev

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_08794_amd as A
    A.library()


def _oracle(case, dtype="bf16"):
    out = []
    for s in case.seqs:
        xv = widen(case.xv, dtype)[s.vis_off:s.vis_off + s.n_frames * s.per_frame]
        xa = widen(case.xa, dtype)[s.aud_off:s.aud_off + s.n_audio]
        xq = widen(case.xq, dtype)[s.qry_off:s.qry_off + s.n_query]
        out.append(OD.score_sequence(xv, xa, xq, s.n_frames, s.per_frame, case.params))
    return out


def _certify(results):
    for r in results:
        m = r["margins"]
        assert m["cka_degenerate"] > 1.0, m
        assert m["gate"] > 1e-9 and m["segment"] > 1e-9 and m["segment_budget"] > 1e-9, m
        assert m["dafps"] > 1e-9 and m["dedup"] > 1e-9, m
        assert m["frame_budget"] > (1e-4 if r["gate"] else 1e-9), m


def _run(case, dtype="bf16"):
    import paper_2608_08794_amd as A
    xv, xa, xq = (to_dev(x, dtype) for x in (case.xv, case.xa, case.xq))
    out = A.apack_score_dynamics(xv, xa, xq, case.seqs, case.params)
    torch.cuda.synchronize()
    return {k: (v.cpu().numpy() if hasattr(v, "cpu") else v) for k, v in out.items()}


def _compare(case, got, want, dtype="bf16"):
    f0 = 0
    kept_all = []
    for i, (s, r) in enumerate(zip(case.seqs, want)):
        F = s.n_frames
        sl = slice(f0, f0 + F)
        assert bool(got["gate"][i]) == r["gate"], f"clip {i}: gate"
        np.testing.assert_array_equal(got["segment"][sl], r["segment"], err_msg=f"clip {i}: segments")
        np.testing.assert_array_equal(got["budget"][sl], r["frame_budget"], err_msg=f"clip {i}: budgets")
        np.testing.assert_allclose(got["cka"][sl], r["cka"].astype(np.float32), rtol=1e-6, atol=1e-7)
        tol = 1e-5 if r["gate"] else 1e-6
        np.testing.assert_allclose(got["score"][sl], r["score"].astype(np.float32), rtol=tol, atol=1e-7)
        assert got["n_kept"][i] == r["kept"].size
        kept_all.append(r["kept"] + s.vis_off)
        f0 += F
    want_kept = np.concatenate(kept_all) if kept_all else np.zeros(0, np.int64)
    np.testing.assert_array_equal(got["kept"].astype(np.int64), want_kept)


@pytest.mark.parametrize("structure", ["shared", "offset"])
def test_small_clip_parity(structure):
    case = W.dynamics_small(structure)
    log(f"[dynamics] small {structure}")
    want = _oracle(case)
    _certify(want)
    _compare(case, _run(case), want)


@pytest.mark.parametrize("structure", ["shared", "offset"])
def test_small_clip_parity_fp32_inputs(structure):
    case = W.dynamics_small(structure)
    f32 = W.DynamicsCase("f32", case.dim, W.bf16_bits_to_f32(case.xv), W.bf16_bits_to_f32(case.xa),
                         W.bf16_bits_to_f32(case.xq), case.seqs, case.params)
    want = _oracle(f32, "f32")
    _certify(want)
    _compare(f32, _run(f32, "f32"), want, "f32")


@pytest.mark.parametrize("structure", ["shared", "offset"])
def test_7b_shape_60s_clip_parity(structure):
    case = W.dynamics_cfg3(structure)
    log(f"[dynamics] 60 s clip, 3584-d, {structure}")
    want = _oracle(case)
    _certify(want)
    _compare(case, _run(case), want)


def _packed(parts, params, gaps=None):
    """Clips packed one after another; with gaps = (before, between, after),
    rows that belong to no clip (large random values) sit before the first
    clip, between clips and after the last one in all three buffers."""
    rng = np.random.default_rng(99)
    xv, xa, xq, seqs = [], [], [], []
    vo = ao = qo = 0
    dim = parts[0].dim

    def gap(n):
        nonlocal vo, ao, qo
        if n:
            for buf in (xv, xa, xq):
                buf.append(W.to_bf16_bits(rng.uniform(-40.0, 40.0, size=(n, dim)).astype(np.float32)))
            vo, ao, qo = vo + n, ao + n, qo + n

    for i, c in enumerate(parts):
        if gaps:
            gap(gaps[0] if i == 0 else gaps[1])
        s = c.seqs[0]
        seqs.append(W.AVSeq(s.n_frames, s.per_frame, s.n_audio, s.n_query, vo, ao, qo, s.seg_starts, s.structure))
        xv.append(c.xv)
        xa.append(c.xa)
        xq.append(c.xq)
        vo += c.xv.shape[0]
        ao += c.xa.shape[0]
        qo += c.xq.shape[0]
    if gaps:
        gap(gaps[2])
    return W.DynamicsCase("bf16", dim, np.concatenate(xv), np.concatenate(xa), np.concatenate(xq), seqs, params)


def test_ragged_batch_of_clips_with_edge_shapes():
    parts = [
        W.dynamics_small("offset", seed=21, frames=30, per_frame=16, audio=375),
        W.dynamics_small("shared", seed=22, frames=2, per_frame=7, audio=25),      # F < w
        W.dynamics_small("shared", seed=23, frames=1, per_frame=5, audio=9),       # one frame
        W.dynamics_small("offset", seed=24, frames=20, per_frame=70, audio=250),   # P not a multiple of 64
        W.dynamics_small("shared", seed=25, frames=12, per_frame=256, audio=150),  # largest P
        W.dynamics_small("offset", seed=27, frames=8, per_frame=160, audio=80),    # DA-FPS rows past LDS
        W.dynamics_small("shared", seed=28, frames=7, per_frame=151, audio=70),    # odd P * P, rows past LDS
    ]
    case = _packed(parts, {"window": 3, "r_pre": 0.5})
    want = _oracle(case)
    _certify(want)
    _compare(case, _run(case), want)


def test_rows_outside_every_clip_are_ignored():
    """Buffers longer than the clips need: rows before, between and after
    the clips (in X_V, X_A and X_Q alike) change nothing, and the norms and
    max-cosine slots are sized by the clips' rows, not by the buffers'."""
    parts = [
        W.dynamics_small("offset", seed=51, frames=16, per_frame=12, audio=60),
        W.dynamics_small("shared", seed=52, frames=9, per_frame=20, audio=40),
    ]
    case = _packed(parts, {"window": 3, "r_pre": 0.5}, gaps=(5, 37, 300))
    want = _oracle(case)
    _certify(want)
    _compare(case, _run(case), want)


def test_long_clips_on_both_plan_paths():
    """The per-clip plan keeps its per-frame arrays in LDS up to 1023 frames
    and in global memory past that: one clip at the LDS limit, one past it
    (112 segments, the gate fired)."""
    parts = [
        W.dynamics_small("shared", seed=42, frames=1023, per_frame=3, audio=2046),
        W.dynamics_small("offset", seed=43, frames=1500, per_frame=8, audio=3000),
    ]
    case = _packed(parts, {"window": 3, "r_pre": 0.5})
    want = _oracle(case)
    _certify(want)
    _compare(case, _run(case), want)


@pytest.mark.parametrize("window", [1, 2, 5, 9, 16])
def test_window_sizes(window):
    """Every window bucket of the band and CKA kernels (up to the largest
    window, 16), on a 20-frame clip."""
    case = W.dynamics_small("offset", seed=61, frames=20, per_frame=16, audio=100, window=window)
    want = _oracle(case)
    _certify(want)
    _compare(case, _run(case), want)


@pytest.mark.parametrize("dafps_k", [1, 2, 3, 4, 6, 7, 8, 12, 32])
def test_dafps_density_list_lengths(dafps_k):
    """Every length of the DA-FPS density list (its mean over the dafps_k
    largest cosines), on 40-token frames, so that 32 < P - 1."""
    case = W.dynamics_small("offset", seed=81, frames=24, per_frame=40, audio=150)
    case.params = {"window": 3, "r_pre": 0.5, "dafps_k": dafps_k}
    want = _oracle(case)
    _certify(want)
    _compare(case, _run(case), want)


def test_dafps_list_longer_than_the_frame():
    """dafps_k = 32 on 16-token frames: the mean runs over the P - 1 others."""
    case = W.dynamics_small("offset", seed=81, frames=24, per_frame=16, audio=150)
    case.params = {"window": 3, "r_pre": 0.5, "dafps_k": 32}
    want = _oracle(case)
    _certify(want)
    _compare(case, _run(case), want)


@pytest.mark.parametrize("cover,power", [(0.5, 1.0), (0.95, 0.0), (0.8, 2.0)])
def test_dafps_cover_and_power(cover, power):
    case = W.dynamics_small("shared", seed=84, frames=24, per_frame=24, audio=150)
    case.params = {"window": 3, "r_pre": 0.5, "cover_thresh": cover, "dafps_power": power}
    want = _oracle(case)
    _certify(want)
    _compare(case, _run(case), want)


@pytest.mark.parametrize("r_pre", [1.0, 0.05, 0.6])
def test_budget_extremes(r_pre):
    case = W.dynamics_small("offset", seed=31)
    case.params = {"window": 3, "r_pre": r_pre}
    want = _oracle(case)
    _certify(want)
    _compare(case, _run(case), want)


# -- alternative alignment scorers (the supplement's scorer comparison) -------

@pytest.mark.parametrize("alignment", ["gated_cka", "cka", "av_cosine", "spatial_cka"])
@pytest.mark.parametrize("structure", ["shared", "offset"])
def test_alignment_scorers_small_clips(structure, alignment):
    case = W.dynamics_small(structure, seed=8)
    case.params = dict(case.params, alignment=alignment)
    log(f"[dynamics] small {structure}, {alignment}")
    want = _oracle(case)
    _certify(want)
    _compare(case, _run(case), want)


@pytest.mark.parametrize("alignment", ["cka", "av_cosine", "spatial_cka"])
@pytest.mark.parametrize("structure", ["shared", "offset"])
def test_alignment_scorers_7b_shape_60s_clip(structure, alignment):
    case = W.dynamics_cfg3(structure)
    case.params = dict(case.params, alignment=alignment)
    log(f"[dynamics] 60 s clip, 3584-d, {structure}, {alignment}")
    want = _oracle(case)
    _certify(want)
    _compare(case, _run(case), want)


def test_spatial_cka_ragged_batch_with_edge_shapes():
    # Bins of one audio token (N_A = F), a frame with more audio rows than a
    # tile, P not a multiple of the 16-row tile, and the largest P.
    parts = [
        W.dynamics_small("offset", seed=21, frames=30, per_frame=16, audio=375),
        W.dynamics_small("shared", seed=26, frames=10, per_frame=9, audio=10),     # one audio row per bin
        W.dynamics_small("shared", seed=23, frames=1, per_frame=5, audio=40),      # 40 audio rows, one frame
        W.dynamics_small("offset", seed=24, frames=20, per_frame=70, audio=250),
        W.dynamics_small("shared", seed=25, frames=12, per_frame=256, audio=150),
    ]
    case = _packed(parts, {"window": 3, "r_pre": 0.5, "alignment": "spatial_cka"})
    want = _oracle(case)
    _certify(want)
    got = _run(case)
    _compare(case, got, want)
    f0 = sum(p.seqs[0].n_frames for p in parts[:1])
    assert np.all(got["cka"][f0:f0 + 10] == 0.0)   # one-token bins have no audio covariance


# -- degenerate inputs: zero frame, static scene, duplicate and zero tokens --

@pytest.mark.parametrize("alignment", ["gated_cka", "cka", "av_cosine", "spatial_cka"])
@pytest.mark.parametrize("structure", ["shared", "offset"])
def test_degenerate_inputs_parity(structure, alignment):
    """A zero frame, a static scene (repeated frames and audio), duplicate
    tokens in an anchor frame and zero tokens and audio rows: zero CKA on
    degenerate windows, cosine exactly 1 between repeated tokens and 0 for
    zero ones, so the ties these inputs create fall the same way (lower
    index) on both sides."""
    case = W.dynamics_edge(structure)
    case.params = dict(case.params, alignment=alignment)
    log(f"[dynamics] edge clip {structure}, {alignment}")
    want = _oracle(case)
    _certify(want)
    _compare(case, _run(case), want)


def test_degenerate_inputs_parity_fp32_and_wide_dim():
    """The same degenerate clip at the 7B embedding width (the 256-tile gate
    GEMM) and with fp32 inputs (the fp32 gate GEMM)."""
    case = W.dynamics_edge("offset", dim=3584, frames=40, per_frame=24, audio=500)
    log("[dynamics] edge clip, 3584-d, bf16")
    want = _oracle(case)
    _certify(want)
    _compare(case, _run(case), want)
    f32 = W.DynamicsCase("f32", case.dim, W.bf16_bits_to_f32(case.xv), W.bf16_bits_to_f32(case.xa),
                         W.bf16_bits_to_f32(case.xq), case.seqs, case.params)
    log("[dynamics] edge clip, 3584-d, fp32")
    want = _oracle(f32, "f32")
    _certify(want)
    _compare(f32, _run(f32, "f32"), want, "f32")


def test_scorer_is_deterministic():
    """Two runs of the 60 s 7B-shape clip with the gate fired (atomic
    maxima, split-K Grams, cross-workgroup sums) give the same bits."""
    case = W.dynamics_cfg3("offset")
    a, b = _run(case), _run(case)
    for key in ("cka", "score", "budget", "segment", "gate", "kept"):
        assert np.array_equal(a[key].view(np.uint8), b[key].view(np.uint8)), key
    assert a["n_kept"] == b["n_kept"]
