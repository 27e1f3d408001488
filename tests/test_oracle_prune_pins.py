"""Pins of the prune oracle (Section 3.2, Eq. 5-6) to things other than itself.

Library routines (torch softmax, scaled-dot-product attention with GQA),
closed forms, invariants, exact decimal arithmetic, brute force on tiny
inputs, and the structure the generators plant.
"""

import math
from fractions import Fraction

import numpy as np
import pytest
import torch

import workloads as W
from oracle import prune as OP, widen

AUDIO, VISUAL, OTHER = 1, 2, 0


def _rand_case(rng, hq, hkv, t, d, tags):
    q = rng.standard_normal((hq, t, d))
    k = rng.standard_normal((hkv, len(tags), d))
    return q, k, np.asarray(tags)


# -- counts (Eq. 6): ceil(keep * n) for the decimal ratio the caller means


def test_keep_count_matches_exact_decimal_ceiling():
    for pct in range(5, 100, 5):
        keep_str = f"0.{pct:02d}"
        exact = Fraction(keep_str)
        for n in list(range(0, 3000)) + [7500, 8640, 17280, 86400, 93900, 94028]:
            want = math.ceil(exact * n)
            assert OP.keep_count(float(keep_str), n) == want, (keep_str, n)


def test_keep_count_known_values():
    # 0.7 * 86400 evaluates to 60479.99999999999 in binary64; the ceiling is 60480.
    assert OP.keep_count(0.7, 86400) == 60480
    # 0.55 * 100 evaluates to 55.00000000000001 in binary64; the decimal ceiling is 55.
    assert OP.keep_count(0.55, 100) == 55
    assert OP.keep_count(0.3, 17280) == 5184
    assert OP.keep_count(0.3, 7890) == 2367
    assert OP.keep_count(0.0, 10) == 0 and OP.keep_count(1.0, 10) == 10
    # A float32 ratio widened to double is a different number: 0.3f*17280 -> 5185.
    assert OP.keep_count(float(np.float32(0.3)), 17280) == 5185


# -- Eq. 5 against library routines


def test_single_head_single_query_is_torch_softmax():
    rng = np.random.default_rng(1)
    tags = [AUDIO] * 5 + [OTHER] * 2 + [VISUAL] * 6
    q, k, tags = _rand_case(rng, 1, 1, 1, 16, tags)
    cand = tags != OTHER
    s = OP.attention_mass(q, k, cand)
    ref = torch.softmax(torch.from_numpy(q[0, 0] @ k[0, cand].T / 4.0), dim=0).numpy()
    np.testing.assert_allclose(s[cand], ref, rtol=1e-13, atol=0)
    assert np.all(s[~cand] == 0)


def test_gqa_mean_equals_sdpa_probabilities():
    """SDPA with V = identity returns the probabilities; enable_gqa fixes the
    head-to-group mapping (query head h reads key head h // (Hq/Hkv))."""
    rng = np.random.default_rng(2)
    hq, hkv, t, d = 6, 2, 5, 8
    tags = [AUDIO] * 7 + [OTHER] + [VISUAL] * 9 + [OTHER] * 3
    q, k, tags = _rand_case(rng, hq, hkv, t, d, tags)
    cand = tags != OTHER
    s = OP.attention_mass(q, k, cand)
    ks = torch.from_numpy(np.ascontiguousarray(k[:, cand]))
    eye = torch.eye(int(cand.sum()), dtype=torch.float64).expand(hkv, -1, -1).contiguous()
    out = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[None], ks[None], eye[None], enable_gqa=True)[0]
    ref = out.mean(dim=(0, 1)).numpy()
    np.testing.assert_allclose(s[cand], ref, rtol=1e-12, atol=1e-15)
    # A wrong mapping (h % Hkv) gives a different answer on this input.
    q_perm = q[[0, 3, 1, 4, 2, 5]]
    s_bad = OP.attention_mass(q_perm, k, cand)
    assert not np.allclose(s_bad[cand], ref, rtol=1e-6)


def test_brute_force_python_loops():
    rng = np.random.default_rng(3)
    hq, hkv, t, d = 4, 2, 2, 3
    tags = [VISUAL, OTHER, AUDIO, AUDIO, VISUAL, OTHER, VISUAL]
    q, k, tags = _rand_case(rng, hq, hkv, t, d, tags)
    s = OP.attention_mass(q, k, tags != OTHER)
    cands = [j for j in range(len(tags)) if tags[j] != OTHER]
    want = {j: 0.0 for j in cands}
    for h in range(hq):
        g = h // (hq // hkv)
        for tt in range(t):
            lg = {j: sum(q[h, tt, x] * k[g, j, x] for x in range(d)) / math.sqrt(d) for j in cands}
            z = sum(math.exp(v) for v in lg.values())
            for j in cands:
                want[j] += math.exp(lg[j]) / z / (hq * t)
    for j in cands:
        assert s[j] == pytest.approx(want[j], rel=1e-12)


# -- closed forms and invariants


def test_hand_example_one_quarter_three_quarters():
    # D = 4, q = 2 e0; k0 = 0, k2 = ln(3) e0 -> logits 0 and ln 3 -> p = (1/4, 3/4).
    q = np.zeros((1, 1, 4))
    q[0, 0, 0] = 2.0
    k = np.zeros((1, 3, 4))
    k[0, 2, 0] = math.log(3.0)
    k[0, 1] = 123.0  # a text row between them is never scored
    s = OP.attention_mass(q, k, np.array([True, False, True]))
    assert s[0] == pytest.approx(0.25, rel=1e-14)
    assert s[2] == pytest.approx(0.75, rel=1e-14)
    assert s[1] == 0.0


def test_equal_keys_give_uniform_mass():
    rng = np.random.default_rng(4)
    q = rng.standard_normal((4, 3, 8))
    k = np.tile(rng.standard_normal(8), (2, 10, 1))
    s = OP.attention_mass(q, k, np.ones(10, bool))
    np.testing.assert_allclose(s, 0.1, rtol=1e-14)


def test_mass_sums_to_one_and_is_shift_and_permutation_invariant():
    rng = np.random.default_rng(5)
    hq, hkv, t, d = 8, 2, 4, 16
    tags = rng.choice([AUDIO, VISUAL, OTHER], size=40, p=[0.3, 0.6, 0.1])
    q, k, tags = _rand_case(rng, hq, hkv, t, d, tags)
    cand = tags != OTHER
    s = OP.attention_mass(q, k, cand)
    assert s.sum() == pytest.approx(1.0, rel=1e-13)
    # Adding one vector to every key of a group shifts each row's logits by a constant.
    k2 = k + rng.standard_normal((hkv, 1, d))
    np.testing.assert_allclose(OP.attention_mass(q, k2, cand), s, rtol=1e-11)
    # Permuting rows permutes scores.
    perm = rng.permutation(len(tags))
    sp = OP.attention_mass(q, k[:, perm], cand[perm])
    np.testing.assert_allclose(sp, s[perm], rtol=1e-12)
    # Non-candidate keys do not matter.
    k3 = k.copy()
    k3[:, ~cand] = 1e3
    np.testing.assert_allclose(OP.attention_mass(q, k3, cand), s, rtol=0, atol=0)


# -- top-k (Eq. 6 per modality) and the kept list


def test_topk_brute_force_and_tie_break():
    rng = np.random.default_rng(6)
    scores = rng.integers(0, 5, size=30).astype(np.float64) / 7.0   # many exact ties
    rows = np.arange(3, 27)
    for kk in range(0, rows.size + 1):
        want = sorted(sorted(rows.tolist(), key=lambda j: (-np.float32(scores[j]), j))[:kk])
        assert OP.topk_rows(scores, rows, kk).tolist() == want


def test_equal_scores_keep_lowest_rows_per_modality():
    q = np.ones((2, 1, 4))
    k = np.zeros((1, 12, 4))
    tags = np.array([AUDIO] * 4 + [VISUAL] * 6 + [OTHER] * 2)
    r = OP.prune_sequence(q, k, tags, (0.5, 0.5))
    assert r["kept"].tolist() == [0, 1, 4, 5, 6, 10, 11]


def test_duplicate_keys_tie_exactly_and_lower_row_wins():
    rng = np.random.default_rng(7)
    hq, hkv, t, d = 4, 2, 3, 8
    tags = np.array([VISUAL] * 10)
    q, k, _ = _rand_case(rng, hq, hkv, t, d, tags)
    k[:, 6] = k[:, 2]
    s = OP.attention_mass(q, k, tags != OTHER)
    assert s[2] == s[6]
    order = sorted(range(10), key=lambda j: (-s[j], j))
    kk = order.index(2) + 1          # boundary falls between the twins
    kept = OP.topk_rows(s, np.arange(10), kk)
    assert 2 in kept and 6 not in kept


def test_kept_list_invariants():
    rng = np.random.default_rng(8)
    tags = rng.choice([AUDIO, VISUAL, OTHER], size=200, p=[0.2, 0.7, 0.1])
    q, k, tags = _rand_case(rng, 4, 1, 5, 8, tags)
    r = OP.prune_sequence(q, k, tags, (0.35, 0.6))
    kept = r["kept"]
    assert np.all(np.diff(kept) > 0)
    assert set(np.flatnonzero(tags == OTHER)) <= set(kept.tolist())
    for m, keep in ((AUDIO, 0.35), (VISUAL, 0.6)):
        n = int(np.sum(tags == m))
        assert int(np.sum(tags[kept] == m)) == math.ceil(Fraction(str(keep)) * n)
    x = rng.integers(0, 2**16, size=(3, 200, 5)).astype(np.uint16)
    assert np.array_equal(OP.compact_rows(x, kept, axis=1), x[:, kept])


# -- joint ranking (Eq. 6 as written: one TopK over S)


def test_joint_ranking_brute_force():
    rng = np.random.default_rng(17)
    hq, hkv, t, d = 4, 2, 1, 3
    tags = np.array([VISUAL, OTHER, AUDIO, AUDIO, VISUAL, OTHER, VISUAL, AUDIO, VISUAL, VISUAL])
    q, k, tags = _rand_case(rng, hq, hkv, t, d, tags)
    cands = [j for j in range(len(tags)) if tags[j] != OTHER]
    mass = {j: 0.0 for j in cands}
    for h in range(hq):
        g = h // (hq // hkv)
        lg = {j: sum(q[h, 0, x] * k[g, j, x] for x in range(d)) / math.sqrt(d) for j in cands}
        z = sum(math.exp(v) for v in lg.values())
        for j in cands:
            mass[j] += math.exp(lg[j]) / z / hq
    for keep in (0.0, 0.1, 0.5, 0.85, 0.9, 1.0):
        kk = math.ceil(Fraction(str(keep)) * len(cands))
        top = sorted(cands, key=lambda j: (-np.float32(mass[j]), j))[:kk]
        want = sorted([j for j in range(len(tags)) if tags[j] == OTHER] + top)
        r = OP.prune_sequence(q, k, tags, (keep, 0.0), joint=True)
        assert r["kept"].tolist() == want, keep
        assert r["k"] == {"joint": kk}


def test_joint_equals_per_modality_with_one_modality():
    rng = np.random.default_rng(18)
    tags = np.array([AUDIO] * 9 + [OTHER] * 3)
    q, k, tags = _rand_case(rng, 4, 2, 2, 5, tags)
    for keep in (0.2, 0.5, 0.77):
        a = OP.prune_sequence(q, k, tags, (keep, 0.3))
        b = OP.prune_sequence(q, k, tags, (keep, 0.0), joint=True)
        assert a["kept"].tolist() == b["kept"].tolist()


def test_joint_schedule_counts_follow_the_drop_ratio():
    # Repeated Eq. 6 with drop P keeps ceil((1-P)|S|) of the current set.
    n = 1000
    for p_drop in ("0.10", "0.15"):
        keep = 1 - float(p_drop)
        cur = n
        for _ in range(14):
            nxt = OP.keep_count(keep, cur)
            assert nxt == math.ceil((1 - Fraction(p_drop)) * cur)
            cur = nxt
    assert OP.keep_count(0.9, 94028 - 128) == 84510


def test_keep_basis_counts_against_original_length():
    q = np.ones((1, 1, 2))
    k = np.zeros((1, 10, 2))
    tags = np.array([VISUAL] * 10)
    r = OP.prune_sequence(q, k, tags, (0.0, 0.5), keep_basis=(0, 16))
    assert r["k"]["visual"] == 8
    with pytest.raises(ValueError):
        OP.prune_sequence(q, k, tags, (0.0, 0.7), keep_basis=(0, 16))


# -- the generators' planted structure predicts the oracle's kept sets


@pytest.mark.parametrize("fn", [W.prune_cfg1, W.prune_cfg2, W.prune_cfg3])
def test_planted_top_sets_are_recovered_with_margin(fn):
    c = fn()
    s = c.seqs[0]
    r = OP.prune_sequence(widen(c.q, c.dtype), widen(c.k, c.dtype), s.tags(), s.keep)
    top = c.planted[0]
    tags = s.tags()
    for m in (AUDIO, VISUAL):
        kept_m = r["kept"][tags[r["kept"]] == m]
        assert np.array_equal(kept_m, top[m])
    assert r["margin"] >= 1e-2
    assert r["scores"].sum() == pytest.approx(1.0, rel=1e-12)
