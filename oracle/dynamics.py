"""fp64 oracle of the pre-LLM local audio-visual dynamics scorer (Section 3.1).

TEST INFRASTRUCTURE ONLY -- see the package docstring.  Parity pins live in
``tests/test_oracle_dynamics_pins.py``.

The scorer is a heuristic with no closed-form target, so this module follows
the method's steps in the paper's order and notation (Section 3.1 "Coarse
pass", "Gated fine pass", "Segmentation and token selection"; the first loop
of Algorithm 1; the supplement's pre-LLM compression details and Table S1).
Where the paper leaves a step open, the reading used here is stated at the
step:

* audio resampling onto the frame axis: adaptive average-pool bins,
  [floor(f*N_A/F), ceil((f+1)*N_A/F));
* window: exactly w consecutive frames, centred on f (the extra frame of an
  even w lies in the past), clamped inside [0, F); all F frames when F < w;
* centring: subtract each window stack's column means (linear CKA);
* a degenerate window gives 0: one whose centred Gram has a Frobenius norm
  of at most CKA_DEGENERATE times the trace of the raw Gram, on the audio
  or the visual side (a window of repeated frames, or of zero frames, has
  no variation for Eq. 1 to compare; its centred Gram is pure rounding);
* cosines are dot(x, y) / sqrt(dot(x, x) dot(y, y)) with every dot product
  summed by the same rule, so a token and a bitwise copy of it have cosine
  exactly 1 (the square root of a correctly rounded square is its argument);
  a zero-norm cosine gives 0;
* gate: fires when the clip-mean CKA is strictly below tau (Eq. 2);
* the gate blends the CKA term, and the frame score is
  s_f = gamma * u_f + (1 - gamma) * alpha_f, with alpha_f the Eq. 2 blend;
* direct distance d_f: one minus the frame mean of each visual token's
  strongest cosine match over all audio tokens (the "AV cosine" frame
  score of the alignment-scorer comparison), min-max normalised over frames;
* frame-query relevance r_f = (1 + cos(v_f, mean query embedding)) / 2;
* segmentation: Gaussian smoothing of consecutive-frame cosines (sigma,
  truncated at 4 sigma, half-sample-symmetric reflection at the ends); each
  maximal run below tau_sim puts one cut after the run's minimum;
* u_f = g_m(f) / max_m g_m;
* budgets: B_v = clamp(ceil(R_pre * (N_A + F*P)) - N_A, 0, F*P); segment
  budgets apportion B_v by g_m (Eq. 4) with caps |G_m| * P, frame budgets
  apportion B_m by s_f within the segment with caps P; apportionment is
  capped water-filling followed by largest remainders (lowest index first);
* DA-FPS density: rho_i = max(mean of the top-k cosines to other tokens, 0)
  * (1 + number of other tokens with cosine >= the coverage threshold); the
  DA-FPS power applies to rho;
* non-anchor frames keep exactly their budget of least-anchor-similar
  positions; ties go to the lower index everywhere.

Alternative alignment scorers (the supplement's comparison of alignment-
scoring rules and the window sweep), selected by ``alignment``, with the
rest of the compressor unchanged:

* ``"gated_cka"`` (default): Eq. 1 and the gate of Eq. 2;
* ``"cka"``: local-window CKA alone, alpha_f = c_f, never gated;
* ``"av_cosine"``: alpha_f = 1 - d_hat_f for every clip, the token-wise
  match of each visual token to its strongest audio token over the whole
  clip (the "static" similarity that ignores time);
* ``"spatial_cka"``: the w = 1 variant that compares, within each frame,
  the covariance of the visual patches with that of the co-timed audio
  tokens (the frame's adaptive-pool bin):
  c_f = ||A~ V~^T||_F^2 / (||A~ A~^T||_F ||V~ V~^T||_F), each token set
  centred by its own mean (so a bin of one audio token gives 0); this c_f
  then enters the gate of Eq. 2 in place of the window CKA.

Every helper also reports the margins of its discrete decisions so tests can
certify that the seeded inputs sit away from every decision boundary.
"""

import math
from fractions import Fraction

import numpy as np


DEFAULTS = {
    # Table S1 defaults (pre-LLM stage).
    "window": 3,
    "dafps_k": 5,
    "tau_gate": 0.78,
    "beta": 0.90,
    "gamma": 0.9,
    "tau_sim": 0.97,
    "sigma": 1.0,
    "lambda_seg": 0.5,
    "cover_thresh": 0.8,
    "dafps_power": 0.5,
    "r_pre": 0.50,
    # Alignment scorer (see the module docstring); the paper's is gated CKA.
    "alignment": "gated_cka",
}

ALIGNMENTS = ("gated_cka", "cka", "av_cosine", "spatial_cka")

# A centred Gram whose Frobenius norm is at most this fraction of the raw
# Gram's trace marks a degenerate CKA input (see the module docstring).
CKA_DEGENERATE = 1e-8


# --------------------------------------------------------------------------
# Coarse pass: frame-level pairs (a_f, v_f)
# --------------------------------------------------------------------------

def pool_frames(xv, n_frames, per_frame):
    """v_f: mean of frame f's visual tokens.  xv: [F*P, d]."""
    return xv.reshape(n_frames, per_frame, -1).mean(axis=1)


def audio_bins(n_audio, n_frames):
    """Adaptive average-pool bin [lo, hi) of audio rows for each frame."""
    return [((f * n_audio) // n_frames, -((-(f + 1) * n_audio) // n_frames))
            for f in range(n_frames)]


def resample_audio(xa, n_frames):
    """a_f: mean of the audio rows in frame f's bin.  xa: [N_A, d]."""
    out = np.zeros((n_frames, xa.shape[1]), dtype=np.float64)
    for f, (lo, hi) in enumerate(audio_bins(xa.shape[0], n_frames)):
        if hi > lo:
            out[f] = xa[lo:hi].mean(axis=0)
    return out


def window_rows(f, n_frames, w):
    """Rows [lo, hi) of frame f's CKA window (w frames, clamped)."""
    if n_frames <= w:
        return 0, n_frames
    lo = min(max(f - w // 2, 0), n_frames - w)
    return lo, lo + w


def degenerate_ratio(k_centred, raw_trace):
    """||K||_F / tr(G) of a centred Gram K against its raw Gram G (0 when
    the raw trace is 0: the rows are all zero)."""
    nk = math.sqrt(float(np.sum(k_centred * k_centred)))
    return nk / raw_trace if raw_trace > 0.0 else 0.0


def degenerate_margin(ratio):
    """Distance of a degeneracy ratio from CKA_DEGENERATE as |ln(ratio / eps)|
    (infinite for an exact 0)."""
    return math.inf if ratio == 0.0 else abs(math.log(ratio / CKA_DEGENERATE))


def linear_cka(a, v, with_margin=False):
    """Eq. 1 on column-centred stacks A, V in R^{w x d}.

    ||V^T A||_F^2 / (||A^T A||_F ||V^T V||_F) equals
    <A A^T, V V^T>_F / (||A A^T||_F ||V V^T||_F) by the trace identity
    tr(A^T V V^T A) = tr(V V^T A A^T); the w x w form is evaluated here.
    A degenerate side (centred Gram at most CKA_DEGENERATE of the raw
    trace) gives 0.  With ``with_margin`` also returns the degeneracy
    decision's margin.
    """
    tr_a, tr_v = float(np.sum(a * a)), float(np.sum(v * v))
    a = a - a.mean(axis=0, keepdims=True)
    v = v - v.mean(axis=0, keepdims=True)
    ka = a @ a.T
    kv = v @ v.T
    ra, rv = degenerate_ratio(ka, tr_a), degenerate_ratio(kv, tr_v)
    margin = min(degenerate_margin(ra), degenerate_margin(rv))
    if ra <= CKA_DEGENERATE or rv <= CKA_DEGENERATE:
        c = 0.0
    else:
        c = float(np.sum(ka * kv)) / (math.sqrt(float(np.sum(ka * ka))) * math.sqrt(float(np.sum(kv * kv))))
    return (c, margin) if with_margin else c


def frame_cka(a, v, w, with_margin=False):
    """c_f for every frame (Eq. 1 over the clamped window of frame f)."""
    n = a.shape[0]
    out = np.zeros(n, dtype=np.float64)
    margin = math.inf
    for f in range(n):
        lo, hi = window_rows(f, n, w)
        out[f], m = linear_cka(a[lo:hi], v[lo:hi], with_margin=True)
        margin = min(margin, m)
    return (out, margin) if with_margin else out


# --------------------------------------------------------------------------
# Gated fine pass (Eq. 2)
# --------------------------------------------------------------------------

def spatial_cka(xv, xa, n_frames, per_frame, with_margin=False):
    """Per-frame spatial CKA at w = 1 (reading above): linear CKA between the
    feature covariances of the frame's P visual tokens and of the audio
    tokens of its adaptive-pool bin, each centred by its own mean.  A
    degenerate side (as in linear_cka: a bin of one token, or a frame of
    identical tokens) gives 0."""
    lo_hi = audio_bins(xa.shape[0], n_frames)
    out = np.zeros(n_frames)
    margin = math.inf
    for f in range(n_frames):
        v = xv[f * per_frame:(f + 1) * per_frame]
        lo, hi = lo_hi[f]
        a = xa[lo:hi]
        if a.shape[0] == 0 or v.shape[0] == 0:
            continue
        vc = v - v.mean(axis=0)
        ac = a - a.mean(axis=0)
        kaa, kvv = ac @ ac.T, vc @ vc.T
        ra = degenerate_ratio(kaa, float(np.sum(a * a)))
        rv = degenerate_ratio(kvv, float(np.sum(v * v)))
        margin = min(margin, degenerate_margin(ra), degenerate_margin(rv))
        if ra <= CKA_DEGENERATE or rv <= CKA_DEGENERATE:
            continue
        num = float(np.sum((ac @ vc.T) ** 2))
        out[f] = num / (float(np.linalg.norm(kaa)) * float(np.linalg.norm(kvv)))
    return (out, margin) if with_margin else out


def dot(x, y):
    """x . y summed by one rule for every pair of vectors (NumPy's pairwise
    sum of the elementwise products): equal vectors give equal sums."""
    return float(np.sum(x * y))


def cosine(x, y):
    """dot(x, y) / sqrt(dot(x, x) dot(y, y)); 0 when either norm is 0.  A
    vector and a bitwise copy of it give exactly 1."""
    nx, ny = dot(x, x), dot(y, y)
    if nx == 0.0 or ny == 0.0:
        return 0.0
    return dot(x, y) / math.sqrt(nx * ny)


def cosine_gram(x):
    """Cosines of every pair of rows of x, S_ij = G_ij / sqrt(G_ii G_jj) from
    the Gram G of the distinct rows (a bitwise-repeated row is the same row,
    so its cosine with its copy is exactly 1), made exactly symmetric; 0
    where a norm is 0."""
    uniq, inv = np.unique(x, axis=0, return_inverse=True)
    g = uniq @ uniq.T
    g = np.triu(g) + np.triu(g, 1).T
    n = np.diag(g).copy()
    den = np.sqrt(np.outer(n, n))
    s = np.zeros_like(g)
    nz = den > 0.0
    s[nz] = g[nz] / den[nz]
    inv = np.asarray(inv).reshape(-1)
    return s[np.ix_(inv, inv)]


def unit_rows(x):
    """Rows divided by their norms; zero rows stay zero (cosine 0)."""
    n = np.sqrt(np.sum(x * x, axis=1))
    out = np.zeros_like(x)
    nz = n > 0
    out[nz] = x[nz] / n[nz, None]
    return out


def direct_distance(xv, xa, n_frames, per_frame, chunk=4096):
    """d_f = 1 - mean over frame f's tokens of max_j cos(x_V, x_A[j]).

    Returns (d [F], best [F*P]) where best holds each visual token's maximum
    cosine over all audio tokens.  The maximum is computed once per distinct
    visual token, so bitwise-repeated tokens (a frame that repeats another)
    get the same value.
    """
    ua = unit_rows(xa)
    uniq, inv = np.unique(xv, axis=0, return_inverse=True)
    best_u = np.empty(uniq.shape[0], dtype=np.float64)
    for i in range(0, uniq.shape[0], chunk):
        uv = unit_rows(uniq[i:i + chunk])
        best_u[i:i + chunk] = (uv @ ua.T).max(axis=1)
    best = best_u[np.asarray(inv).reshape(-1)]
    d = 1.0 - best.reshape(n_frames, per_frame).mean(axis=1)
    return d, best


def minmax(d):
    lo, hi = float(np.min(d)), float(np.max(d))
    if hi == lo:
        return np.zeros_like(d)
    return (d - lo) / (hi - lo)


# --------------------------------------------------------------------------
# Segmentation (Algorithm 1, second step; supplement pre-LLM details)
# --------------------------------------------------------------------------

def gaussian_smooth(x, sigma, truncate=4.0):
    """Gaussian-weighted moving average with half-sample-symmetric ends."""
    x = np.asarray(x, dtype=np.float64)
    n = x.size
    if n == 0:
        return x.copy()
    radius = int(truncate * float(sigma) + 0.5)
    offs = np.arange(-radius, radius + 1)
    wts = np.exp(-0.5 * (offs / float(sigma)) ** 2)
    wts = wts / wts.sum()
    out = np.zeros(n, dtype=np.float64)
    for i in range(n):
        acc = 0.0
        for o, wt in zip(offs, wts):
            j = (i + o) % (2 * n)
            if j >= n:
                j = 2 * n - 1 - j
            acc += wt * x[j]
        out[i] = acc
    return out


def continuity(v):
    """cs_f = cos(v_f, v_{f+1}) for f < F-1."""
    return np.array([cosine(v[f], v[f + 1]) for f in range(v.shape[0] - 1)],
                    dtype=np.float64)


def segment_ids(smoothed, n_frames, tau_sim):
    """Segment id of every frame.

    Each maximal run of positions with smoothed cosine below tau_sim puts a
    single cut between frames f* and f*+1, f* being the run's minimum
    (lowest index on ties).  Returns (seg [F] int, margin), where margin is
    the smallest |smoothed - tau_sim| and in-run argmin gap.
    """
    seg = np.zeros(n_frames, dtype=np.int64)
    margin = math.inf
    cuts = []
    f = 0
    m = len(smoothed)
    while f < m:
        margin = min(margin, abs(smoothed[f] - tau_sim))
        if smoothed[f] < tau_sim:
            g = f
            while g + 1 < m and smoothed[g + 1] < tau_sim:
                g += 1
                margin = min(margin, abs(smoothed[g] - tau_sim))
            run = smoothed[f:g + 1]
            best = int(np.argmin(run))
            if run.size > 1:
                others = np.delete(run, best)
                margin = min(margin, float(np.min(others) - run[best]))
            cuts.append(f + best)
            f = g + 1
        else:
            f += 1
    for c in cuts:
        seg[c + 1:] += 1
    return seg, margin


# --------------------------------------------------------------------------
# Segment and frame scores (Eq. 3, Eq. 2, Algorithm 1 third-fifth steps)
# --------------------------------------------------------------------------

def relevance(v, qbar):
    """r_f = (1 + cos(v_f, mean query embedding)) / 2."""
    return np.array([(1.0 + cosine(v[f], qbar)) / 2.0 for f in range(v.shape[0])],
                    dtype=np.float64)


def segment_scores(r, seg, lam):
    """g_m = sqrt(|G_m|) (lam max_{G_m} r + (1 - lam) mean_{G_m} r)  (Eq. 3)."""
    n_seg = int(seg.max()) + 1 if seg.size else 0
    g = np.zeros(n_seg, dtype=np.float64)
    for m in range(n_seg):
        rm = r[seg == m]
        g[m] = math.sqrt(rm.size) * (lam * float(rm.max()) + (1.0 - lam) * float(rm.mean()))
    return g


def frame_alpha(c, dhat, fired, beta):
    """The alignment term of frame f (Eq. 2): alpha_f = (1 - beta) c_f +
    beta (1 - dhat_f) when the gate fired, else c_f."""
    c = np.asarray(c, dtype=np.float64)
    if not fired:
        return c.copy()
    return (1.0 - beta) * c + beta * (1.0 - np.asarray(dhat, dtype=np.float64))


def frame_scores(alpha, r, seg, gamma, lam):
    """Segment scores and frame scores (Eq. 3; Algorithm 1, scoring steps).

    g_m from segment_scores, the broadcast u_f = g_m(f) / max_m g_m and the
    frame score s_f = gamma u_f + (1 - gamma) alpha_f.  Returns (g, u, s).
    """
    seg = np.asarray(seg)
    g = segment_scores(np.asarray(r, dtype=np.float64), seg, lam)
    u = g[seg] / float(g.max()) if seg.size else np.zeros(0)
    s = gamma * u + (1.0 - gamma) * np.asarray(alpha, dtype=np.float64)
    return g, u, s


# --------------------------------------------------------------------------
# Budgets (Eq. 4; Algorithm 1 sixth step; supplement pre-LLM details)
# --------------------------------------------------------------------------

def keep_count(ratio, n):
    """ceil(ratio * n) in exact decimal arithmetic (a float ratio is the
    decimal of its shortest round-trip form)."""
    if isinstance(ratio, (float, np.floating)):
        ratio = Fraction(repr(float(ratio)))
    return int(math.ceil(Fraction(ratio) * int(n)))


def visual_budget(r_pre, n_audio, n_visual):
    """B_v = clamp(ceil(R_pre (N_A + N_V)) - N_A, 0, N_V): all audio is kept."""
    b = keep_count(r_pre, n_audio + n_visual) - n_audio
    return max(0, min(b, n_visual))


def apportion(total, weights, caps):
    """Capped largest-remainder apportionment of ``total`` by ``weights``.

    Water-filling first: items whose proportional quota exceeds their cap are
    fixed at the cap and the rest is re-shared among the others, until no
    quota exceeds its cap.  Then each free item gets floor(quota) and the
    leftover units go to the largest fractional parts, lowest index first on
    ties.  All-zero weights among the free items share equally.

    Returns (alloc int array, margin).  The only decision that can change
    the allocation under a tiny perturbation of the quotas is the order of
    fractional parts at the remainder cut, so margin is the gap between the
    last fractional part that receives a unit and the first that does not.
    A quota just below an integer has fractional part near 1 and receives a
    unit that restores its floor, and a quota at its cap ends at the cap
    whether it is fixed or free, so neither is a decision boundary.
    """
    w = np.asarray(weights, dtype=np.float64)
    caps = np.asarray(caps, dtype=np.int64)
    n = w.size
    if total < 0 or total > int(caps.sum()):
        raise ValueError("total outside [0, sum(caps)]")
    fixed = np.zeros(n, dtype=bool)
    margin = math.inf
    while True:
        free = ~fixed
        remaining = total - int(caps[fixed].sum())
        wf = w[free]
        sw = float(wf.sum())
        quota = np.zeros(n, dtype=np.float64)
        if sw > 0.0:
            quota[free] = remaining * w[free] / sw
        elif free.any():
            quota[free] = remaining / float(free.sum())
        over = free & (quota > caps)
        if not over.any():
            break
        fixed |= over
    alloc = np.zeros(n, dtype=np.int64)
    alloc[fixed] = caps[fixed]
    free_idx = np.flatnonzero(~fixed)
    if free_idx.size:
        fl = np.floor(quota[free_idx])
        alloc[free_idx] = fl.astype(np.int64)
        frac = quota[free_idx] - fl
        left = total - int(alloc.sum())
        order = sorted(range(free_idx.size), key=lambda i: (-frac[i], i))
        for i in order[:left]:
            alloc[free_idx[i]] += 1
        if 0 < left < free_idx.size:
            margin = min(margin, _cut_gap([frac[i] for i in order], left))
    return alloc, margin


def _cut_gap(desc, k):
    """Gap between the k-th largest value of ``desc`` (sorted descending) and
    the largest value below it.  Values exactly equal to the k-th are split
    by index on both sides of any comparison: such ties arise from identical
    computations (frames sharing a clamped window, identical tokens), which
    an implementation reproduces bit for bit."""
    kth = desc[k - 1]
    below = [x for x in desc[k:] if x < kth]
    return float(kth - below[0]) if below else math.inf


def budgets(bv, g, s, seg, per_frame):
    """Segment and frame budgets (Eq. 4; Algorithm 1, allocation step).

    B_m apportions the visual budget bv by the segment scores g_m with caps
    |G_m| P; then k_f apportions B_m over the frames of segment m by their
    frame scores s_f with caps P.  Returns (B [n_seg], k [F], margins) with
    the margins of the two apportionments.
    """
    seg = np.asarray(seg)
    n_seg = len(g)
    seg_len = np.array([int(np.sum(seg == m)) for m in range(n_seg)], dtype=np.int64)
    if n_seg:
        bm, m_seg = apportion(bv, g, seg_len * per_frame)
    else:
        bm, m_seg = np.zeros(0, np.int64), math.inf
    kf = np.zeros(seg.size, dtype=np.int64)
    m_frame = math.inf
    for m in range(n_seg):
        frames = np.flatnonzero(seg == m)
        alloc, mg = apportion(int(bm[m]), np.asarray(s)[frames], np.full(frames.size, per_frame))
        kf[frames] = alloc
        m_frame = min(m_frame, mg)
    return bm, kf, {"segment_budget": m_seg, "frame_budget": m_frame}


# --------------------------------------------------------------------------
# Token selection (Algorithm 1 loop over segments)
# --------------------------------------------------------------------------

def dafps(x, k, density_k, cover_thresh, power):
    """Density-aware farthest-point sampling on one anchor frame.

    x: [P, d] tokens.  rho_i = max(mean of the density_k largest cosines to
    other tokens, 0) * (1 + #{j != i : cos_ij >= cover_thresh}).  The first
    pick is argmax rho; each later pick maximises
    (1 - max cosine to the picked set) * rho^power over the unpicked tokens.
    Returns (picks in pick order, margin).
    """
    p = x.shape[0]
    k = min(k, p)
    s = cosine_gram(x)
    margin = math.inf
    rho = np.zeros(p, dtype=np.float64)
    for i in range(p):
        others = np.delete(s[i], i)
        if others.size:
            margin = min(margin, float(np.min(np.abs(others - cover_thresh))))
            top = np.sort(others)[::-1][:density_k]
            knn = float(top.mean())
            cov = int(np.sum(others >= cover_thresh))
        else:
            knn, cov = 0.0, 0
        rho[i] = max(knn, 0.0) * (1.0 + cov)
    picks = []
    if k == 0:
        return picks, margin
    first, gap = _argmax_lowest(rho)
    margin = min(margin, gap)
    picks.append(first)
    sim_max = s[first].copy()
    taken = np.zeros(p, dtype=bool)
    taken[first] = True
    weight = rho ** power
    while len(picks) < k:
        val = (1.0 - sim_max) * weight
        val[taken] = -math.inf
        nxt, gap = _argmax_lowest(val)
        margin = min(margin, gap)
        picks.append(nxt)
        taken[nxt] = True
        sim_max = np.maximum(sim_max, s[nxt])
    return picks, margin


def _argmax_lowest(v):
    """Index of the maximum (lowest index on ties) and the gap to the largest
    value below it (exact ties are split by index, see _cut_gap)."""
    i = int(np.argmax(v))
    rest = v[np.isfinite(v) & (v < v[i])]
    gap = float(v[i] - rest.max()) if rest.size else math.inf
    return i, gap


def dedup(x, anchor, k):
    """Non-anchor frame: the k positions least similar to the anchor token at
    the same position (lowest position on ties).  Returns (picks, margin)."""
    p = x.shape[0]
    sim = np.array([cosine(x[i], anchor[i]) for i in range(p)], dtype=np.float64)
    order = sorted(range(p), key=lambda i: (sim[i], i))
    picks = sorted(order[:k])
    margin = math.inf
    if 0 < k < p:
        margin = _cut_gap([-sim[i] for i in order], k)
    return picks, margin


# --------------------------------------------------------------------------
# The whole scorer for one sequence
# --------------------------------------------------------------------------

def score_sequence(xv, xa, xq, n_frames, per_frame, params=None):
    """Pre-LLM scorer for one clip (Section 3.1; first loop of Algorithm 1).

    xv: [F*P, d] visual tokens, xa: [N_A, d] audio tokens, xq: [n_q, d]
    query-span embeddings, all fp64.  Returns a dict of every intermediate,
    the kept visual rows (sequence-local, ascending) and the decision margins.
    """
    p = dict(DEFAULTS)
    if params:
        p.update(params)
    F, P = n_frames, per_frame
    n_audio = xa.shape[0]
    margins = {}

    v = pool_frames(xv, F, P)
    a = resample_audio(xa, F)
    qbar = xq.mean(axis=0)

    # Local-window CKA and the gate (Eq. 1, Eq. 2), or an alternative scorer.
    mode = p["alignment"]
    if mode not in ALIGNMENTS:
        raise ValueError(f"unknown alignment {mode!r}")
    if mode == "spatial_cka":
        c, margins["cka_degenerate"] = spatial_cka(xv, xa, F, P, with_margin=True)
    else:
        c, margins["cka_degenerate"] = frame_cka(a, v, p["window"], with_margin=True)
    cbar = float(c.mean()) if F else 0.0
    if mode in ("gated_cka", "spatial_cka"):
        fired = bool(F > 0 and cbar < p["tau_gate"])
        margins["gate"] = abs(cbar - p["tau_gate"]) if F else math.inf
    else:
        fired = bool(F > 0 and mode == "av_cosine")
        margins["gate"] = math.inf
    beta = 1.0 if mode == "av_cosine" else p["beta"]
    if fired:
        d, _ = direct_distance(xv, xa, F, P)
        dhat = minmax(d)
    else:
        d = np.zeros(F)
        dhat = np.zeros(F)
    alpha = frame_alpha(c, dhat, fired, beta)

    # Segmentation.
    cs = continuity(v)
    sm = gaussian_smooth(cs, p["sigma"])
    seg, margins["segment"] = segment_ids(sm, F, p["tau_sim"])

    # Segment score, broadcast and frame score (Eq. 3; Algorithm 1).
    r = relevance(v, qbar)
    g, u, s = frame_scores(alpha, r, seg, p["gamma"], p["lambda_seg"])

    # Budgets (Eq. 4 at segment level, then frames within each segment).
    bv = visual_budget(p["r_pre"], n_audio, F * P)
    n_seg = g.size
    bm, kf, mb = budgets(bv, g, s, seg, P)
    margins.update(mb)

    # Token selection: DA-FPS on each anchor, dedup on the other frames.
    keep = np.zeros(F * P, dtype=bool)
    m_fps, m_dd = math.inf, math.inf
    for m in range(n_seg):
        frames = np.flatnonzero(seg == m)
        anchor = int(frames[0])
        xa_f = xv[anchor * P:(anchor + 1) * P]
        picks, mg = dafps(xa_f, int(kf[anchor]), p["dafps_k"], p["cover_thresh"],
                          p["dafps_power"])
        m_fps = min(m_fps, mg)
        keep[anchor * P + np.asarray(picks, dtype=np.int64)] = True
        for f in frames[1:]:
            picks, mg = dedup(xv[f * P:(f + 1) * P], xa_f, int(kf[f]))
            m_dd = min(m_dd, mg)
            keep[f * P + np.asarray(picks, dtype=np.int64)] = True
    margins["dafps"] = m_fps
    margins["dedup"] = m_dd
    kept = np.flatnonzero(keep)

    return {
        "v": v, "a": a, "qbar": qbar, "cka": c, "cbar": cbar, "gate": fired,
        "d": d, "dhat": dhat, "alpha": alpha, "continuity": cs, "smoothed": sm,
        "segment": seg, "relevance": r, "g": g, "u": u, "score": s,
        "visual_budget": bv, "segment_budget": bm, "frame_budget": kf,
        "kept": kept, "margins": margins,
    }
