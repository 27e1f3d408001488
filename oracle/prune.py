"""fp64 oracle of the in-LLM query-conditioned prune (Section 3.2).

TEST INFRASTRUCTURE ONLY -- see the package docstring.  Parity pins live in
``tests/test_oracle_prune_pins.py``.

What one prune step computes, for one sequence (Section 3.2, Eq. 5 and Eq. 6;
the inner loop of Algorithm 1), in the readings listed below:

1. Candidates S: the rows whose modality tag is audio or visual.  Text and
   other rows are never scored and always kept.
2. Logits: for every query head h, query row t and candidate j,
   l[h,t,j] = q[h,t] . k[g(h), j] / sqrt(D), with the grouped-query mapping
   g(h) = h // (Hq / Hkv) and D the key (head) dimension.
3. Eq. 5: for each (h, t), p[h,t,:] is the softmax of l[h,t,:] over S.
4. Head and query mean: I_j = mean over all (h, t) of p[h,t,j].  The paper
   averages over heads and scores with the last query token; a query span of
   one row reproduces that, and longer spans average every query row.
5. Per-modality top-k (Eq. 6 applied within each modality): k_m is
   ceil(keep_m * n_m) in exact decimal arithmetic (keep_m is the decimal
   ratio the caller means), with n_m the modality's current candidate count
   or an explicit basis.  T_m is
   the first k_m rows of modality m in the order (score descending, row
   ascending); the ranking uses the fp32-rounded score, the precision of the
   GPU path.
6. Kept rows: the ascending union of non-candidates, T_audio and T_visual.
7. Compaction: every per-row array is gathered at the kept rows.
"""

import math
from fractions import Fraction

import numpy as np

AUDIO = 1
VISUAL = 2
OTHER = 0


def exact_ratio(keep):
    """The decimal a keep ratio denotes, as an exact fraction.

    A float is taken as the decimal of its shortest round-trip form (0.55
    means 55/100, not the nearest binary64 value).
    """
    if isinstance(keep, Fraction):
        return keep
    if isinstance(keep, (float, np.floating)):
        return Fraction(repr(float(keep)))
    return Fraction(keep)


def keep_count(keep, n):
    """k = ceil(keep * n) in exact decimal arithmetic (Eq. 6's count)."""
    r = exact_ratio(keep)
    n = int(n)
    if not (0 <= r <= 1):
        raise ValueError("keep ratio must lie in [0, 1]")
    if n < 0:
        raise ValueError("count must be non-negative")
    return int(math.ceil(r * n))


def logits(q, k):
    """Scaled query-key logits of one sequence (Eq. 5 numerator exponent).

    q: [Hq, T, D] fp64 query rows; k: [Hkv, J, D] fp64 keys.
    Returns [Hq, T, J]: l[h,t,j] = q[h,t] . k[h // (Hq/Hkv), j] / sqrt(D).
    """
    hq, _, d = q.shape
    hkv = k.shape[0]
    if hq % hkv != 0:
        raise ValueError("query heads must be a multiple of key heads")
    n_rep = hq // hkv
    out = np.empty((hq, q.shape[1], k.shape[1]), dtype=np.float64)
    for h in range(hq):
        out[h] = q[h] @ k[h // n_rep].T
    return out / math.sqrt(d)


def softmax_rows(x):
    """Softmax along the last axis with the row maximum subtracted first."""
    m = np.max(x, axis=-1, keepdims=True)
    e = np.exp(x - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def attention_mass(q, k, cand, row_chunk=256):
    """I_j of Eq. 5 averaged over heads and query rows, for j in S.

    q: [Hq, T, D]; k: [Hkv, N, D]; cand: boolean [N] marking S.
    Returns an [N] fp64 array: I_j for candidates, 0 elsewhere.
    Rows (h, t) are processed in chunks so the [rows, |S|] probability block
    stays small; the sum over rows is accumulated in a fixed order.
    """
    hq, t_len, _ = q.shape
    hkv = k.shape[0]
    n_rep = hq // hkv
    idx = np.flatnonzero(cand)
    scores = np.zeros(k.shape[1], dtype=np.float64)
    if idx.size == 0:
        return scores
    ks = k[:, idx, :]
    acc = np.zeros(idx.size, dtype=np.float64)
    for h in range(hq):
        for t0 in range(0, t_len, row_chunk):
            l = logits(q[h:h + 1, t0:t0 + row_chunk], ks[h // n_rep:h // n_rep + 1])
            p = softmax_rows(l[0])
            acc += p.sum(axis=0)
    scores[idx] = acc / float(hq * t_len)
    return scores


def topk_rows(scores, rows, k):
    """First k of ``rows`` ordered by (fp32 score descending, row ascending)."""
    rows = np.asarray(rows, dtype=np.int64)
    if k > rows.size:
        raise ValueError("k exceeds the candidate count")
    s32 = scores[rows].astype(np.float32)
    order = np.lexsort((rows, -s32.astype(np.float64)))
    return np.sort(rows[order[:k]])


def boundary_gap(scores, rows, k):
    """Relative gap at the k boundary: (s_(k) - s_(k+1)) / s_(k), fp64.

    s_(i) is the i-th largest score among ``rows``.  Returns +inf when the
    boundary is empty (k == 0 or k == |rows|).
    """
    if k <= 0 or k >= len(rows):
        return math.inf
    s = np.sort(scores[np.asarray(rows)])[::-1]
    if s[k - 1] <= 0:
        return 0.0
    return float((s[k - 1] - s[k]) / s[k - 1])


def prune_sequence(q, k, tags, keep, keep_basis=(0, 0), joint=False):
    """One prune step of one sequence.

    q: [Hq, T, D] fp64; k: [Hkv, N, D] fp64; tags: [N] int (0 other,
    1 audio, 2 visual); keep: (keep_audio, keep_visual);
    keep_basis: n used in ceil(keep*n) per modality, 0 = current count.
    joint: rank the audio and visual candidates together, as Eq. 6 is
    written (S <- TopK of ceil((1-P)|S|) over the whole candidate set), with
    keep[0] = 1 - P and keep_basis[0] its n; keep[1] and keep_basis[1] are
    unused.

    Returns a dict with ``scores`` [N] fp64 (0 for non-candidates), ``kept``
    (ascending sequence-local rows), ``k`` (per-modality counts, or the joint
    count under "joint") and ``margin`` (the smallest relative boundary gap).
    """
    tags = np.asarray(tags)
    cand = (tags == AUDIO) | (tags == VISUAL)
    scores = attention_mass(q, k, cand)
    kept = [np.flatnonzero(~cand)]
    ks = {}
    margin = math.inf
    if joint:
        rows = np.flatnonzero(cand)
        kj = keep_count(keep[0], int(keep_basis[0]) or rows.size)
        kept.append(topk_rows(scores, rows, kj))
        kept = np.sort(np.concatenate(kept))
        return {"scores": scores, "kept": kept, "k": {"joint": kj}, "margin": boundary_gap(scores, rows, kj)}
    for m, name in ((AUDIO, "audio"), (VISUAL, "visual")):
        rows = np.flatnonzero(tags == m)
        basis = int(keep_basis[m - 1]) or rows.size
        km = keep_count(keep[m - 1], basis)
        ks[name] = km
        kept.append(topk_rows(scores, rows, km))
        margin = min(margin, boundary_gap(scores, rows, km))
    kept = np.sort(np.concatenate(kept))
    return {"scores": scores, "kept": kept, "k": ks, "margin": margin}


def prune_batch(q, k, seqs, q_off_key="q_off"):
    """Prune step over a packed ragged batch.

    q: [Hq, sum T, D] fp64; k: [Hkv, sum N, D] fp64.
    seqs: list of dicts with tok_off, n_tokens, q_off, q_len, tags [n_tokens],
    keep (pair), optional keep_basis (pair) and optional joint (bool).
    Returns (scores [sum N], kept_rows: packed absolute rows, sequences in
    order, ascending within each; n_kept per sequence; margins).
    """
    total = k.shape[1]
    scores = np.zeros(total, dtype=np.float64)
    kept_all, n_kept, margins = [], [], []
    for s in seqs:
        o, n = s["tok_off"], s["n_tokens"]
        qo, ql = s[q_off_key], s["q_len"]
        r = prune_sequence(q[:, qo:qo + ql], k[:, o:o + n], s["tags"], s["keep"],
                           s.get("keep_basis", (0, 0)), s.get("joint", False))
        scores[o:o + n] = r["scores"]
        kept_all.append(r["kept"] + o)
        n_kept.append(r["kept"].size)
        margins.append(r["margin"])
    kept_rows = np.concatenate(kept_all) if kept_all else np.zeros(0, np.int64)
    return scores, kept_rows, n_kept, margins


def compact_rows(x, kept_rows, axis):
    """Gather of the kept rows along ``axis`` on raw bits (no arithmetic)."""
    return np.take(x, np.asarray(kept_rows, dtype=np.int64), axis=axis)
