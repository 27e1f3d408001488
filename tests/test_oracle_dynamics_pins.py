"""Pins of the pre-LLM scorer oracle (Section 3.1, Eq. 1-4; Algorithm 1).

Each check ties the oracle to something other than itself: library routines
(torch adaptive pooling, scipy Gaussian filtering), the HSIC form of linear
CKA and Eq. 1 written in feature space, closed forms of rank-one windows,
hand-computed examples, brute-force enumeration, and the scene structure the
generators plant.
"""

import itertools
import math

import numpy as np
import pytest
import scipy.ndimage
import torch

import workloads as W
from oracle import dynamics as OD, widen


# -- coarse pass


def test_audio_resample_is_adaptive_avg_pool():
    rng = np.random.default_rng(0)
    for n_audio, n_frames in ((1500, 120), (25, 2), (7, 5), (13, 13), (3, 8)):
        xa = rng.standard_normal((n_audio, 6))
        ours = OD.resample_audio(xa, n_frames)
        ref = torch.nn.functional.adaptive_avg_pool1d(
            torch.from_numpy(xa.T.copy())[None], n_frames)[0].T.numpy()
        np.testing.assert_allclose(ours, ref, rtol=1e-13, atol=1e-15)


def test_frame_pool_is_mean_over_tokens():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((5 * 7, 3))
    v = OD.pool_frames(x, 5, 7)
    for f in range(5):
        np.testing.assert_allclose(v[f], sum(x[f * 7 + p] for p in range(7)) / 7, rtol=1e-14)


def test_window_rows():
    assert OD.window_rows(0, 10, 3) == (0, 3)
    assert OD.window_rows(5, 10, 3) == (4, 7)
    assert OD.window_rows(9, 10, 3) == (7, 10)
    # Even window: the extra frame lies in the past.
    assert OD.window_rows(5, 10, 4) == (3, 7)
    assert OD.window_rows(2, 2, 3) == (0, 2)


# -- Eq. 1


def _eq1_feature_space(a, v):
    a = a - a.mean(axis=0)
    v = v - v.mean(axis=0)
    num = np.linalg.norm(v.T @ a, "fro") ** 2
    return num / (np.linalg.norm(a.T @ a, "fro") * np.linalg.norm(v.T @ v, "fro"))


def _hsic_cka(a, v):
    """Kornblith et al. linear CKA: HSIC(K, L) / sqrt(HSIC(K, K) HSIC(L, L))
    with K = A A^T, L = V V^T on the raw rows and H the centring matrix."""
    n = a.shape[0]
    h = np.eye(n) - np.ones((n, n)) / n
    k, l = a @ a.T, v @ v.T

    def hsic(x, y):
        return np.trace(x @ h @ y @ h)

    return hsic(k, l) / math.sqrt(hsic(k, k) * hsic(l, l))


def test_cka_equals_eq1_in_feature_space_and_hsic_form():
    rng = np.random.default_rng(2)
    for w in (2, 3, 4, 6):
        for _ in range(5):
            a = rng.standard_normal((w, 11))
            v = rng.standard_normal((w, 11)) + 0.5 * a
            c = OD.linear_cka(a, v)
            assert c == pytest.approx(_eq1_feature_space(a, v), rel=1e-12)
            assert c == pytest.approx(_hsic_cka(a, v), rel=1e-12)
            assert 0.0 <= c <= 1.0 + 1e-15


def test_cka_invariances_and_special_cases():
    rng = np.random.default_rng(3)
    a = rng.standard_normal((4, 9))
    v = rng.standard_normal((4, 9))
    c = OD.linear_cka(a, v)
    assert OD.linear_cka(a, a) == pytest.approx(1.0, rel=1e-14)
    q, _ = np.linalg.qr(rng.standard_normal((9, 9)))
    assert OD.linear_cka(a @ q, v) == pytest.approx(c, rel=1e-12)
    assert OD.linear_cka(3.7 * a, v) == pytest.approx(c, rel=1e-12)
    assert OD.linear_cka(a + rng.standard_normal(9), v) == pytest.approx(c, rel=1e-12)
    # Two centred rows are always collinear: CKA = 1.
    assert OD.linear_cka(a[:2], v[:2]) == pytest.approx(1.0, rel=1e-12)
    # A constant stack has zero centred Gram: CKA defined as 0.
    assert OD.linear_cka(np.ones((3, 5)), v[:3]) == 0.0


def test_cka_rank_one_closed_form():
    """A = u a^T, V = t b^T: CKA = (u_c . t_c)^2 / (|u_c|^2 |t_c|^2)."""
    rng = np.random.default_rng(4)
    a_dir, b_dir = rng.standard_normal(16), rng.standard_normal(16)
    spike, trend = np.array([-1.0, 1.0, -1.0]), np.array([0.0, 1.0, 2.0])
    assert OD.linear_cka(np.outer(spike, a_dir), np.outer(trend, b_dir)) == pytest.approx(0.0, abs=1e-15)
    alt4, trend4 = np.array([1.0, -1.0, 1.0, -1.0]), np.arange(4.0)
    # centred: alt4 -> (1,-1,1,-1), trend4 -> (-1.5,-.5,.5,1.5): (u.t)^2 = 4, |u|^2 |t|^2 = 4*5
    assert OD.linear_cka(np.outer(alt4, a_dir), np.outer(trend4, b_dir)) == pytest.approx(0.2, rel=1e-13)
    u, t = rng.standard_normal(5), rng.standard_normal(5)
    uc, tc = u - u.mean(), t - t.mean()
    want = (uc @ tc) ** 2 / ((uc @ uc) * (tc @ tc))
    assert OD.linear_cka(np.outer(u, a_dir), np.outer(t, b_dir)) == pytest.approx(want, rel=1e-12)


def test_frame_cka_uses_clamped_windows():
    rng = np.random.default_rng(5)
    a, v = rng.standard_normal((7, 5)), rng.standard_normal((7, 5))
    c = OD.frame_cka(a, v, 3)
    assert c[0] == pytest.approx(_eq1_feature_space(a[0:3], v[0:3]), rel=1e-12)
    assert c[3] == pytest.approx(_eq1_feature_space(a[2:5], v[2:5]), rel=1e-12)
    assert c[6] == pytest.approx(_eq1_feature_space(a[4:7], v[4:7]), rel=1e-12)


# -- Eq. 2: direct distance and gate


def test_direct_distance_closed_form():
    xa = np.array([[1.0, 0.0, 0.0], [0.0, 1.0, 0.0]])
    xv = np.array([[2.0, 0.0, 0.0],    # parallel to audio 0: cos 1
                   [0.0, 0.0, 5.0],    # orthogonal to both: cos 0
                   [1.0, 1.0, 0.0],    # 45 degrees: cos sqrt(1/2)
                   [-1.0, -1.0, 0.0]])  # best match cos = -sqrt(1/2)
    d, best = OD.direct_distance(xv, xa, 2, 2)
    np.testing.assert_allclose(best, [1.0, 0.0, math.sqrt(0.5), -math.sqrt(0.5)], atol=1e-15)
    np.testing.assert_allclose(d, [0.5, 1.0], atol=1e-15)
    np.testing.assert_allclose(OD.minmax(np.array([2.0, 4.0, 3.0])), [0.0, 1.0, 0.5])
    assert np.all(OD.minmax(np.array([1.0, 1.0])) == 0)


def test_gate_switches_on_cka_mean():
    case = W.dynamics_small("offset")
    s = case.seqs[0]
    r = OD.score_sequence(widen(case.xv, "bf16"), widen(case.xa, "bf16"), widen(case.xq, "bf16"),
                          s.n_frames, s.per_frame, case.params)
    assert r["gate"] and r["cbar"] < 0.78
    b = 0.90
    np.testing.assert_allclose(r["alpha"], (1 - b) * r["cka"] + b * (1 - r["dhat"]), rtol=1e-15)
    case = W.dynamics_small("shared")
    s = case.seqs[0]
    r = OD.score_sequence(widen(case.xv, "bf16"), widen(case.xa, "bf16"), widen(case.xq, "bf16"),
                          s.n_frames, s.per_frame, case.params)
    assert not r["gate"] and r["cbar"] > 0.78
    np.testing.assert_array_equal(r["alpha"], r["cka"])


# -- segmentation


@pytest.mark.parametrize("n", [1, 2, 3, 5, 9, 40, 119])
def test_smoothing_matches_scipy(n):
    rng = np.random.default_rng(n)
    x = rng.uniform(0.8, 1.0, size=n)
    for sigma in (1.0, 0.7, 2.0):
        ref = scipy.ndimage.gaussian_filter1d(x, sigma, mode="reflect", truncate=4.0)
        np.testing.assert_allclose(OD.gaussian_smooth(x, sigma), ref, rtol=1e-13)


def test_single_hard_cut_gives_five_low_positions_and_one_cut():
    cs = np.full(30, 0.99)
    cs[12] = 0.0
    sm = OD.gaussian_smooth(cs, 1.0)
    assert np.flatnonzero(sm < 0.97).tolist() == [10, 11, 12, 13, 14]
    seg, _ = OD.segment_ids(sm, 31, 0.97)
    assert seg.tolist() == [0] * 13 + [1] * 18


def test_segments_from_hand_built_runs():
    sm = np.array([0.99, 0.5, 0.4, 0.6, 0.99, 0.99, 0.1, 0.99, 0.95])
    seg, margin = OD.segment_ids(sm, 10, 0.97)
    # runs {1,2,3} (min at 2) and {6} and {8}: cuts after frames 2, 6, 8
    assert seg.tolist() == [0, 0, 0, 1, 1, 1, 1, 2, 2, 3]
    assert margin == pytest.approx(0.02)
    seg, _ = OD.segment_ids(np.full(5, 0.99), 6, 0.97)
    assert seg.tolist() == [0] * 6


# -- Eq. 3 and the frame score


def test_relevance_and_segment_score_closed_forms():
    qbar = np.array([1.0, 0.0])
    v = np.array([[2.0, 0.0], [-1.0, 0.0], [0.0, 3.0]])
    np.testing.assert_allclose(OD.relevance(v, qbar), [1.0, 0.0, 0.5])
    r = np.array([0.2, 0.8, 0.5, 0.4])
    seg = np.array([0, 0, 0, 1])
    g = OD.segment_scores(r, seg, 0.5)
    assert g[0] == pytest.approx(math.sqrt(3) * (0.5 * 0.8 + 0.5 * 0.5))
    assert g[1] == pytest.approx(0.4)


# -- Eq. 4 and the frame budgets


def test_visual_budget_hand_values():
    assert OD.visual_budget(0.5, 1500, 17280) == 7890
    assert OD.visual_budget(0.35, 1500, 17280) == 5073
    assert OD.visual_budget(0.1, 1500, 1000) == 0
    assert OD.visual_budget(1.0, 10, 20) == 20


def _brute_apportion(total, q, caps):
    best, best_key = None, None
    for alloc in itertools.product(*[range(c + 1) for c in caps]):
        if sum(alloc) != total:
            continue
        key = (sum((a - x) ** 2 for a, x in zip(alloc, q)),
               tuple(-a for a in alloc))   # on equal error, favour lower indices
        if best_key is None or key < best_key:
            best, best_key = alloc, key
    return list(best)


def test_apportion_is_l2_closest_integer_vector_without_binding_caps():
    rng = np.random.default_rng(6)
    for _ in range(200):
        n = int(rng.integers(1, 5))
        w = rng.uniform(0.05, 1.0, size=n)
        total = int(rng.integers(0, 9))
        caps = [total] * n
        q = [total * x / w.sum() for x in w]
        alloc, _ = OD.apportion(total, w, caps)
        assert alloc.tolist() == _brute_apportion(total, q, caps)


def _waterfill(total, w, caps):
    """q*_i = min(cap_i, lam * w_i) with sum q* = total, lam by bisection."""
    lo, hi = 0.0, 1.0
    while sum(min(c, hi * x) for x, c in zip(w, caps)) < total:
        hi *= 2.0
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        if sum(min(c, mid * x) for x, c in zip(w, caps)) < total:
            lo = mid
        else:
            hi = mid
    return [min(c, hi * x) for x, c in zip(w, caps)]


def test_apportion_with_caps_matches_waterfill_brute_force():
    alloc, _ = OD.apportion(8, [10.0, 1.0, 1.0], [2, 5, 5])
    assert alloc.tolist() == [2, 3, 3]
    rng = np.random.default_rng(7)
    for _ in range(300):
        n = int(rng.integers(1, 5))
        w = rng.uniform(0.05, 1.0, size=n) ** 2
        caps = rng.integers(0, 6, size=n).tolist()
        total = int(rng.integers(0, sum(caps) + 1))
        alloc, _ = OD.apportion(total, w, caps)
        assert int(alloc.sum()) == total
        assert np.all(alloc >= 0) and np.all(alloc <= caps)
        qstar = _waterfill(total, w.tolist(), caps)
        assert alloc.tolist() == _brute_apportion(total, qstar, caps)


def test_apportion_is_scale_invariant():
    # Table S1 writes the segment weight as twice Eq. 3 at lambda = 0.5.
    w = np.array([0.3, 0.9, 0.45, 0.7])
    a1, _ = OD.apportion(37, w, [20] * 4)
    a2, _ = OD.apportion(37, 2 * w, [20] * 4)
    assert a1.tolist() == a2.tolist()


# -- token selection


def test_dafps_hand_example():
    """Four unit tokens at 0, 10, 25 and 90 degrees; density k = 2, coverage 0.8.

    rho = (2.8367, 2.9261, 2.8084, 0.2981): first pick token 1; then
    (1 - sim) * sqrt(rho) = (0.0256, -, 0.0571, 0.4512) -> token 3; then
    token 2 (0.0571 > 0.0256); then token 0.
    """
    ang = np.radians([0.0, 10.0, 25.0, 90.0])
    x = np.stack([np.cos(ang), np.sin(ang)], axis=1) * np.array([[1.0], [2.0], [0.5], [3.0]])
    picks, margin = OD.dafps(x, 4, 2, 0.8, 0.5)
    assert picks == [1, 3, 2, 0]
    assert margin > 0.01
    assert OD.dafps(x, 2, 2, 0.8, 0.5)[0] == [1, 3]
    assert OD.dafps(x, 0, 2, 0.8, 0.5)[0] == []


def _dafps_loops(x, k, dk, cover, power):
    p = len(x)
    norm = [math.sqrt(sum(v * v for v in row)) for row in x]
    s = [[sum(a * b for a, b in zip(x[i], x[j])) / (norm[i] * norm[j]) for j in range(p)] for i in range(p)]
    rho = []
    for i in range(p):
        others = sorted((s[i][j] for j in range(p) if j != i), reverse=True)
        knn = sum(others[:dk]) / len(others[:dk])
        cov = sum(1 for j in range(p) if j != i and s[i][j] >= cover)
        rho.append(max(knn, 0.0) * (1 + cov))
    picks = [max(range(p), key=lambda i: (rho[i], -i))]
    while len(picks) < k:
        cand = [i for i in range(p) if i not in picks]
        val = {i: (1 - max(s[i][j] for j in picks)) * rho[i] ** power for i in cand}
        picks.append(max(cand, key=lambda i: (val[i], -i)))
    return picks


def test_dafps_brute_force_loops():
    rng = np.random.default_rng(8)
    for trial in range(20):
        p = int(rng.integers(2, 9))
        x = rng.standard_normal((p, 4)) + (0.8 if trial % 2 else 0.0)
        k = int(rng.integers(1, p + 1))
        assert OD.dafps(x, k, 3, 0.8, 0.5)[0] == _dafps_loops(x.tolist(), k, 3, 0.8, 0.5)


def test_dedup_keeps_least_anchor_similar_positions():
    rng = np.random.default_rng(9)
    anchor = rng.standard_normal((10, 6))
    x = anchor + rng.uniform(0, 2, size=(10, 1)) * rng.standard_normal((10, 6))
    sims = [float(x[i] @ anchor[i] / np.linalg.norm(x[i]) / np.linalg.norm(anchor[i])) for i in range(10)]
    for k in range(11):
        want = sorted(sorted(range(10), key=lambda i: (sims[i], i))[:k])
        assert OD.dedup(x, anchor, k)[0] == want


# -- whole scorer on planted clips


@pytest.mark.parametrize("structure", ["shared", "offset"])
def test_scorer_recovers_planted_scenes_and_budgets(structure):
    case = W.dynamics_small(structure)
    s = case.seqs[0]
    r = OD.score_sequence(widen(case.xv, "bf16"), widen(case.xa, "bf16"), widen(case.xq, "bf16"),
                          s.n_frames, s.per_frame, case.params)
    starts = [0] + (np.flatnonzero(np.diff(r["segment"])) + 1).tolist()
    assert starts == s.seg_starts
    assert r["gate"] == (structure == "offset")
    bv = OD.visual_budget(0.5, s.n_audio, s.n_frames * s.per_frame)
    assert r["visual_budget"] == bv == r["kept"].size == int(r["frame_budget"].sum())
    assert np.all(r["frame_budget"] <= s.per_frame)
    kept = r["kept"]
    assert np.all(np.diff(kept) > 0) and kept.min() >= 0 and kept.max() < s.n_frames * s.per_frame
    per_frame = np.bincount(kept // s.per_frame, minlength=s.n_frames)
    np.testing.assert_array_equal(per_frame, r["frame_budget"])
    for key, m in r["margins"].items():
        assert m > 1e-9, key


# -- alternative alignment scorers -------------------------------------------

def _spatial_by_covariance(xv, xa, F, P):
    """Spatial CKA the long way: explicit d x d feature covariances of each
    frame's centred patches and centred co-timed audio tokens, compared by
    their Frobenius cosine."""
    out = []
    for f, (lo, hi) in enumerate(OD.audio_bins(xa.shape[0], F)):
        v = xv[f * P:(f + 1) * P]
        a = xa[lo:hi]
        cv = (v - v.mean(0)).T @ (v - v.mean(0))
        ca = (a - a.mean(0)).T @ (a - a.mean(0))
        den = np.linalg.norm(cv) * np.linalg.norm(ca)
        out.append(float(np.sum(cv * ca) / den) if den else 0.0)
    return np.array(out)


def test_spatial_cka_equals_feature_covariance_alignment():
    rng = np.random.default_rng(41)
    for F, P, NA, d in ((5, 7, 23, 6), (3, 16, 9, 11), (8, 4, 40, 3)):
        xv = rng.standard_normal((F * P, d))
        xa = rng.standard_normal((NA, d))
        np.testing.assert_allclose(OD.spatial_cka(xv, xa, F, P), _spatial_by_covariance(xv, xa, F, P),
                                   rtol=1e-12, atol=1e-15)


def test_spatial_cka_rank_one_is_squared_cosine():
    # Patches varying along w only and audio along u only: c = cos^2(u, w).
    rng = np.random.default_rng(42)
    d, P = 9, 12
    u, w = rng.standard_normal(d), rng.standard_normal(d)
    base_v, base_a = rng.standard_normal(d), rng.standard_normal(d)
    xv = base_v + np.outer(rng.standard_normal(P), w)
    xa = base_a + np.outer(rng.standard_normal(6), u)     # one frame, bin of all 6 audio rows
    want = (u @ w) ** 2 / ((u @ u) * (w @ w))
    assert OD.spatial_cka(xv, xa, 1, P)[0] == pytest.approx(want, rel=1e-12)


def test_spatial_cka_invariances_and_degenerate_bins():
    rng = np.random.default_rng(43)
    F, P, NA, d = 4, 10, 30, 7
    xv = rng.standard_normal((F * P, d))
    xa = rng.standard_normal((NA, d))
    c = OD.spatial_cka(xv, xa, F, P)
    q, _ = np.linalg.qr(rng.standard_normal((d, d)))
    np.testing.assert_allclose(OD.spatial_cka(xv @ q, xa @ q, F, P), c, rtol=1e-11)       # shared rotation
    np.testing.assert_allclose(OD.spatial_cka(3.5 * xv, 0.2 * xa, F, P), c, rtol=1e-12)   # scales
    shift = np.repeat(rng.standard_normal((F, d)), P, axis=0)
    np.testing.assert_allclose(OD.spatial_cka(xv + shift, xa + 5.0, F, P), c, rtol=1e-9)  # per-frame shifts
    perm = np.concatenate([f * P + rng.permutation(P) for f in range(F)])
    np.testing.assert_allclose(OD.spatial_cka(xv[perm], xa, F, P), c, rtol=1e-12)         # patch order
    assert np.all((c >= 0.0) & (c <= 1.0 + 1e-12))
    # A bin of one audio token has no covariance: c = 0.
    assert np.all(OD.spatial_cka(xv, xa[:F], F, P) == 0.0)


def test_alignment_modes_select_their_frame_scores():
    case = W.dynamics_small("offset", seed=44)
    s = case.seqs[0]
    xv, xa, xq = (widen(x, "bf16") for x in (case.xv, case.xa, case.xq))
    base = OD.score_sequence(xv, xa, xq, s.n_frames, s.per_frame, case.params)
    cka = OD.score_sequence(xv, xa, xq, s.n_frames, s.per_frame, dict(case.params, alignment="cka"))
    assert base["gate"] and not cka["gate"]
    np.testing.assert_array_equal(cka["alpha"], cka["cka"])
    av = OD.score_sequence(xv, xa, xq, s.n_frames, s.per_frame, dict(case.params, alignment="av_cosine"))
    assert av["gate"]
    np.testing.assert_array_equal(av["alpha"], 1.0 - av["dhat"])
    np.testing.assert_array_equal(av["dhat"], base["dhat"])
    sp = OD.score_sequence(xv, xa, xq, s.n_frames, s.per_frame, dict(case.params, alignment="spatial_cka"))
    np.testing.assert_array_equal(sp["cka"], OD.spatial_cka(xv, xa, s.n_frames, s.per_frame))
    with pytest.raises(ValueError):
        OD.score_sequence(xv, xa, xq, s.n_frames, s.per_frame, dict(case.params, alignment="ot"))


# -- frame scores and budgets, composed by hand (Eq. 2-4; Algorithm 1) -------
#
# Five frames, two tokens per frame (P = 2), segments G_0 = {0, 1, 2} and
# G_1 = {3, 4}; lambda = 0.5, gamma = 0.9, beta = 0.9; N_A = 5 audio tokens
# and R_pre = 0.8, so B_v = ceil(0.8 * (5 + 10)) - 5 = 12 - 5 = 7.
#
#   r = (0.5, 0.9, 0.7 | 0.3, 0.6)
#   g_0 = sqrt(3) (0.5 * 0.9 + 0.5 * 0.7) = 0.8 sqrt(3)   = 1.3856406460551018
#   g_1 = sqrt(2) (0.5 * 0.6 + 0.5 * 0.45) = 0.525 sqrt(2) = 0.7424621202458749
#   u = (1, 1, 1, g_1/g_0, g_1/g_0),  g_1/g_0 = 0.65625 sqrt(2/3) = 0.5358258812338203
#   c = (0.2, 0.2, 0.6, 0.9, 0.1)       (frames 0 and 1 share a clamped window)
#   dhat = (0, 0.5, 1, 0.25, 0.75)
#
# Segment budgets (Eq. 4) by g with caps (6, 4): quotas 7 g_m / (g_0 + g_1)
# = (4.5578, 2.4422) -> floors (4, 2), the one leftover unit to the larger
# fractional part .5578 -> B = (5, 2).  The same with or without the gate.

_HAND = dict(r=[0.5, 0.9, 0.7, 0.3, 0.6], c=[0.2, 0.2, 0.6, 0.9, 0.1],
             dhat=[0.0, 0.5, 1.0, 0.25, 0.75], seg=[0, 0, 0, 1, 1])
_G = [1.3856406460551018, 0.7424621202458749]
_U1 = 0.5358258812338203


def _hand(fired):
    alpha = OD.frame_alpha(_HAND["c"], _HAND["dhat"], fired, 0.9)
    g, u, s = OD.frame_scores(alpha, _HAND["r"], np.array(_HAND["seg"]), 0.9, 0.5)
    bv = OD.visual_budget(0.8, 5, 5 * 2)
    bm, kf, _ = OD.budgets(bv, g, s, np.array(_HAND["seg"]), 2)
    return bv, alpha, g, u, s, bm, kf


def test_frame_scores_and_budgets_by_hand_gate_off():
    # alpha = c.  s = 0.9 u + 0.1 c:
    #   (0.9 + 0.02, 0.9 + 0.02, 0.9 + 0.06, 0.9 * 0.5358258812 + 0.09, ... + 0.01)
    # Frames of G_0 share B_0 = 5 by s, caps 2: quotas 5 s / 2.8 =
    # (1.642857, 1.642857, 1.714286) -> floors (1, 1, 1); two leftover units
    # to the largest fractional parts: frame 2 (.714), then frame 0 (ties
    # with frame 1 at .642857 go to the lower index) -> (2, 1, 2).
    # G_1: B_1 = 2, quotas 2 s / 1.0644865862 = (1.07515, 0.92485) -> (1, 1).
    bv, alpha, g, u, s, bm, kf = _hand(False)
    assert bv == 7
    np.testing.assert_allclose(alpha, [0.2, 0.2, 0.6, 0.9, 0.1], rtol=0, atol=0)
    np.testing.assert_allclose(g, _G, rtol=1e-14)
    np.testing.assert_allclose(u, [1.0, 1.0, 1.0, _U1, _U1], rtol=1e-14)
    np.testing.assert_allclose(s, [0.92, 0.92, 0.96, 0.5722432931104383, 0.4922432931104383], rtol=1e-14)
    assert bm.tolist() == [5, 2]
    assert kf.tolist() == [2, 1, 2, 1, 1]


def test_frame_scores_and_budgets_by_hand_gate_fired():
    # alpha = 0.1 c + 0.9 (1 - dhat) = (0.92, 0.47, 0.06, 0.765, 0.235);
    # s = 0.9 u + 0.1 alpha = (0.992, 0.947, 0.906, 0.4822432931 + 0.0765,
    # 0.4822432931 + 0.0235).  G_0: quotas 5 s / 2.845 =
    # (1.743409, 1.664323, 1.592267) -> floors (1, 1, 1), leftover units to
    # frames 0 and 1 -> (2, 2, 1).  G_1: quotas (1.04978, 0.95022) -> (1, 1).
    bv, alpha, g, u, s, bm, kf = _hand(True)
    np.testing.assert_allclose(alpha, [0.92, 0.47, 0.06, 0.765, 0.235], rtol=1e-14)
    np.testing.assert_allclose(g, _G, rtol=1e-14)
    np.testing.assert_allclose(s, [0.992, 0.947, 0.906, 0.5587432931104383, 0.5057432931104383], rtol=1e-14)
    assert bm.tolist() == [5, 2]
    assert kf.tolist() == [2, 2, 1, 1, 1]


@pytest.mark.parametrize("structure", ["shared", "offset"])
def test_score_sequence_composes_the_hand_pinned_steps(structure):
    """The whole scorer's frame scores and budgets are the composition pinned
    above, applied to its own CKA, distance, relevance and segments."""
    case = W.dynamics_small(structure)
    s = case.seqs[0]
    r = OD.score_sequence(widen(case.xv, "bf16"), widen(case.xa, "bf16"), widen(case.xq, "bf16"),
                          s.n_frames, s.per_frame, case.params)
    alpha = OD.frame_alpha(r["cka"], r["dhat"], r["gate"], OD.DEFAULTS["beta"])
    g, u, sc = OD.frame_scores(alpha, r["relevance"], r["segment"], OD.DEFAULTS["gamma"], 0.5)
    bm, kf, _ = OD.budgets(r["visual_budget"], g, sc, r["segment"], s.per_frame)
    np.testing.assert_array_equal(r["score"], sc)
    np.testing.assert_array_equal(r["segment_budget"], bm)
    np.testing.assert_array_equal(r["frame_budget"], kf)


# -- degenerate inputs: repeated frames, zero tokens, duplicate tokens -------


def test_repeated_rows_make_a_degenerate_window():
    rng = np.random.default_rng(60)
    # Column means of three copies of a row are not always the row itself,
    # so the centred stack is rounding noise rather than 0; the window is
    # degenerate and its CKA is defined as 0.
    noisy = 0
    for _ in range(50):
        x = rng.standard_normal(40)
        a = np.stack([x, x, x])
        v = rng.standard_normal((3, 40))
        noisy += int(np.any(a - a.mean(axis=0) != 0))
        assert OD.linear_cka(a, v) == 0.0
        assert OD.linear_cka(v, a) == 0.0
    assert noisy > 0
    assert OD.linear_cka(np.zeros((3, 5)), rng.standard_normal((3, 5))) == 0.0
    # Variation well above the bound is compared by Eq. 1 as usual; far
    # below it the window counts as degenerate.
    base, trend = rng.standard_normal(30), rng.standard_normal(30)
    v = rng.standard_normal((4, 30))
    a = base + 1e-2 * np.outer(np.arange(4.0), trend)
    assert OD.linear_cka(a, v) == pytest.approx(_eq1_feature_space(a, v), rel=1e-9)
    a = base + 1e-7 * np.outer(np.arange(4.0), trend)
    c, margin = OD.linear_cka(a, v, with_margin=True)
    assert c == 0.0 and margin > 1.0


def test_static_run_gives_zero_frame_cka():
    rng = np.random.default_rng(61)
    a, v = rng.standard_normal((12, 8)), rng.standard_normal((12, 8))
    v[4:9] = v[4]
    c = OD.frame_cka(a, v, 3)
    # Windows lying inside frames 4..8: those of frames 5, 6, 7.
    assert c[5] == c[6] == c[7] == 0.0
    assert np.all(c[[0, 1, 2, 3, 10, 11]] != 0.0)


def test_cosine_of_a_bitwise_copy_is_exactly_one():
    rng = np.random.default_rng(62)
    x = widen(W.to_bf16_bits(rng.standard_normal((400, 3584)).astype(np.float32)), "bf16")
    sqrt_twice = 0
    for row in x:
        assert OD.cosine(row, row.copy()) == 1.0
        n = math.sqrt(float(row @ row))
        sqrt_twice += int(float(row @ row) / (n * n) != 1.0)
    assert sqrt_twice > 0   # the sqrt(n) sqrt(n) form misses 1 on some rows
    assert OD.cosine(x[0], np.zeros(3584)) == 0.0
    assert OD.cosine(x[0], x[1]) == pytest.approx(float(x[0] @ x[1]) / np.linalg.norm(x[0]) / np.linalg.norm(x[1]),
                                                  rel=1e-13)


def test_cosine_gram_with_duplicates_and_zero_rows():
    rng = np.random.default_rng(63)
    x = rng.standard_normal((10, 50))
    x[[3, 7]] = x[1]
    x[5] = 0.0
    s = OD.cosine_gram(x)
    assert np.array_equal(s, s.T)
    for i in (1, 3, 7):
        for j in (1, 3, 7):
            assert s[i, j] == 1.0
    assert np.all(s[5] == 0.0) and np.all(s[:, 5] == 0.0)
    u = x / np.maximum(np.linalg.norm(x, axis=1, keepdims=True), 1e-300)
    np.testing.assert_allclose(s, u @ u.T, rtol=1e-13, atol=1e-15)


def test_dedup_of_a_repeated_frame_takes_zero_tokens_then_lowest_positions():
    rng = np.random.default_rng(64)
    anchor = widen(W.to_bf16_bits(rng.standard_normal((16, 64)).astype(np.float32)), "bf16")
    anchor[6] = 0.0
    frame = anchor.copy()
    frame[11] = 0.0
    for k in range(17):
        picks, margin = OD.dedup(frame, anchor, k)
        assert picks == sorted(([6, 11] + [p for p in range(16) if p not in (6, 11)])[:k])
        assert margin >= 1.0   # only exact ties sit at a cut, or the gap from 0 to 1


def test_dafps_duplicate_tokens_tie_to_the_lowest_index():
    rng = np.random.default_rng(65)
    x = rng.standard_normal((12, 6)) + 2.0     # all cosines positive
    x[[4, 8, 9]] = x[2]
    picks, _ = OD.dafps(x, 12, 3, 0.8, 0.5)
    # The copies are one point: once one of them is picked, the others have
    # distance 0 to the picked set and come last, in index order.
    first = min(i for i in (2, 4, 8, 9) if i in picks[:-3])
    assert picks[-3:] == sorted({2, 4, 8, 9} - {first})
    assert sorted(picks) == list(range(12))


def test_direct_distance_of_repeated_frames_is_equal():
    rng = np.random.default_rng(66)
    xv = rng.standard_normal((6 * 5, 9))
    xv[10:15] = xv[5:10]
    xv[20:25] = xv[5:10]
    d, best = OD.direct_distance(xv, rng.standard_normal((7, 9)), 6, 5, chunk=4)
    assert d[1] == d[2] == d[4]
    np.testing.assert_array_equal(best[5:10], best[20:25])


@pytest.mark.parametrize("structure", ["shared", "offset"])
def test_scorer_on_degenerate_inputs(structure):
    """Zero frame, static scene, duplicate and zero tokens (the edge clip):
    planted segments recovered (frame 0 alone), zero CKA inside the static
    scene, and the static non-anchor frames keep the zero token's position
    and then the lowest positions, with every decision certified."""
    case = W.dynamics_edge(structure)
    s = case.seqs[0]
    r = OD.score_sequence(widen(case.xv, "bf16"), widen(case.xa, "bf16"), widen(case.xq, "bf16"),
                          s.n_frames, s.per_frame, case.params)
    starts = [0] + (np.flatnonzero(np.diff(r["segment"]) != 0) + 1).tolist()
    assert starts == s.seg_starts
    assert r["gate"] == (structure == "offset")
    xv = case.xv.reshape(s.n_frames, s.per_frame, -1)
    static = [m for m in range(1, len(starts))
              if all(np.array_equal(xv[f], xv[starts[m]])
                     for f in range(starts[m], (starts + [s.n_frames])[m + 1]))]
    assert len(static) == 1
    s0, s1 = starts[static[0]], (starts + [s.n_frames])[static[0] + 1]
    assert np.all(r["cka"][s0 + 1:s1 - 1] == 0.0)
    kept = r["kept"]
    for f in range(s0 + 1, s1):
        got = (kept[(kept >= f * s.per_frame) & (kept < (f + 1) * s.per_frame)] - f * s.per_frame).tolist()
        k = int(r["frame_budget"][f])
        assert got == sorted(([3] + [p for p in range(s.per_frame) if p != 3])[:k])
    for key, m in r["margins"].items():
        assert m > (1.0 if key == "cka_degenerate" else 1e-9), key
