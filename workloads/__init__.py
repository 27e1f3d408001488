"""Seeded synthetic workloads for the A-PACK hot path.

This module holds shapes and seeded input generators only.  It contains no
step of the method's arithmetic (no attention mass, softmax, top-k, CKA,
segmentation, budget or token selection): it only draws the inputs, with
the token shapes of the paper's workloads (25 audio tokens per second, two
frames per second of 144 visual tokens, the Qwen2.5-Omni thinker head
shapes) and planted structure that keeps every discrete decision of the
method away from its boundary.  The tests, the benchmark and the smoke check
all draw their inputs here; the CPU oracle never imports it.

All values are drawn with ``numpy.random.default_rng(seed)`` in float32 and,
for bf16 workloads, rounded to bf16 with round-to-nearest-even.  The rounded
bit patterns are the single source of truth for both the oracle and the GPU.
"""

import math
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

AUDIO = 1
VISUAL = 2
OTHER = 0

AUDIO_PER_SECOND = 25
FRAMES_PER_SECOND = 2
TOKENS_PER_FRAME = 144


# --------------------------------------------------------------------------
# bf16 bit handling (generator side)
# --------------------------------------------------------------------------

def to_bf16_bits(x):
    """float32 -> bf16 bit patterns (uint16), round to nearest even."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounding = np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))
    return ((b + rounding) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(bits):
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


def payload_bits(rng, shape, dtype):
    """Unique-content payload rows for bit copies (values never used).

    bf16: random finite bit patterns with |value| < 2 (exponent top bit
    cleared).  f32: standard normal values.
    """
    if dtype == "bf16":
        n = int(np.prod(shape))
        words = rng.bit_generator.random_raw((n + 3) // 4).view(np.uint16)[:n]
        return (words & np.uint16(0xBFFF)).reshape(shape)
    return rng.standard_normal(shape, dtype=np.float32)


def _round(x, dtype):
    return to_bf16_bits(x) if dtype == "bf16" else np.asarray(x, dtype=np.float32)


def _values(x, dtype):
    """float32 values of raw generator output (for building lifts)."""
    return bf16_bits_to_f32(x) if dtype == "bf16" else x


# --------------------------------------------------------------------------
# Prune-step workloads (in-LLM stage)
# --------------------------------------------------------------------------

@dataclass
class PruneSeq:
    tok_off: int
    n_tokens: int
    spans: List[tuple]          # (begin, len, modality), sequence-local rows
    q_off: int
    q_len: int
    keep: tuple                 # (audio, visual); (joint, 0) with joint ranking
    keep_basis: tuple = (0, 0)  # n in ceil(keep * n); 0 = current count
    joint: bool = False         # rank audio and visual together

    def tags(self):
        t = np.zeros(self.n_tokens, dtype=np.int8)
        for b, n, m in self.spans:
            t[b:b + n] = m
        return t


@dataclass
class PruneCase:
    """One prune step: Q of the query span and K of the prune layer."""
    name: str
    dtype: str                  # "bf16" or "f32"
    hq: int
    hkv: int
    d: int
    q: np.ndarray               # [Hq, sum q_len, D] raw (uint16 bits or float32)
    k: np.ndarray               # [Hkv, sum N, D] raw
    seqs: List[PruneSeq]
    planted: dict = field(default_factory=dict)   # modality -> planted top set per seq


@dataclass
class CacheCase:
    """Payload to compact: per-layer K/V, hidden states and positions."""
    dtype: str
    hkv: int
    d: int
    hidden_dim: int
    k_layers: List[np.ndarray]  # each [Hkv, N, D] raw
    v_layers: List[np.ndarray]
    hidden: Optional[np.ndarray]  # [N, H] raw
    pos: Optional[np.ndarray]     # [3, N] int32


def _group_unit_dirs(qv, hkv):
    """Unit mean query direction of every KV group (float32)."""
    hq = qv.shape[0]
    n_rep = hq // hkv
    dirs = []
    for g in range(hkv):
        m = qv[g * n_rep:(g + 1) * n_rep].reshape(-1, qv.shape[-1]).mean(axis=0)
        dirs.append(m / np.linalg.norm(m))
    return np.stack(dirs).astype(np.float32)


def _lift(kv, dirs, rows, amount):
    """K[g, rows] += amount * dirs[g] (float32, before rounding)."""
    if len(rows) == 0:
        return
    rows = np.asarray(rows)
    for g in range(kv.shape[0]):
        kv[g, rows] += np.float32(amount) * dirs[g]


def _ceil_keep(keep, n):
    # Generator-side count, used only to size the planted sets: the ceiling
    # of keep * n for the decimal ratio written as `keep`.
    from fractions import Fraction
    return int(math.ceil(Fraction(repr(float(keep))) * n))


def _single_seq(n_audio, n_visual, n_text, q_len, keep, basis=(0, 0)):
    spans = [(0, n_audio, AUDIO), (n_audio, n_visual, VISUAL)]
    n = n_audio + n_visual + n_text
    return PruneSeq(0, n, spans, 0, q_len, keep, basis)


def _planted_sets(rng, tags, keep, basis, high=None):
    """Random top set of size ceil(keep*n) per modality (containing ``high``)."""
    out = {}
    for m in (AUDIO, VISUAL):
        rows = np.flatnonzero(tags == m)
        n = basis[m - 1] or rows.size
        k = _ceil_keep(keep[m - 1], n)
        must = np.intersect1d(rows, high) if high is not None else np.zeros(0, np.int64)
        must = must[:k]
        rest = np.setdiff1d(rows, must)
        extra = rng.choice(rest, size=k - must.size, replace=False) if k > must.size else np.zeros(0, np.int64)
        out[m] = np.sort(np.concatenate([must, extra]).astype(np.int64))
    return out


# Planted lifts (multiples of the unit group-mean query direction).  Chosen
# so that the relative score gap at every top-k boundary is >= 1e-2.
LIFT_F32_BOUNDARY = 8.0
QUERY_TOPIC_F32 = 3.0
LIFT_BF16_BOUNDARY = 12.0
LIFT_BF16_HIGH = 60.0


def prune_cfg1(seed=0):
    """Tiny fp32 step: 8/2 heads, D=64; 256 audio + 16x64 visual + 32 text."""
    rng = np.random.default_rng(seed)
    hq, hkv, d = 8, 2, 64
    seq = _single_seq(256, 1024, 32, 32, (0.5, 0.5))
    q = rng.standard_normal((hq, seq.q_len, d), dtype=np.float32)
    k = rng.standard_normal((hkv, seq.n_tokens, d), dtype=np.float32)
    # Planted structure: every query row of a KV group shares a topic
    # direction, and the planted top rows' keys are lifted along it.
    dirs = _unit(rng, (hkv,), d)
    n_rep = hq // hkv
    for g in range(hkv):
        q[g * n_rep:(g + 1) * n_rep] += np.float32(QUERY_TOPIC_F32) * dirs[g]
    top = _planted_sets(rng, seq.tags(), seq.keep, seq.keep_basis)
    _lift(k, dirs, np.concatenate([top[AUDIO], top[VISUAL]]), LIFT_F32_BOUNDARY)
    return PruneCase("cfg1", "f32", hq, hkv, d, q, k, [seq], {0: top})


def _bf16_step(rng, hq, hkv, d, seq, high_frac=0.0):
    scale = np.float32(1.0 / math.sqrt(d))
    qf = rng.standard_normal((hq, seq.q_len, d), dtype=np.float32) * scale
    q = to_bf16_bits(qf)
    kf = rng.standard_normal((hkv, seq.n_tokens, d), dtype=np.float32) * scale
    dirs = _group_unit_dirs(bf16_bits_to_f32(q), hkv)
    tags = seq.tags()
    cand = np.flatnonzero(tags != OTHER)
    high = None
    if high_frac > 0:
        n_high = _ceil_keep(high_frac, cand.size)
        high = np.sort(rng.choice(cand, size=n_high, replace=False))
        _lift(kf, dirs, high, LIFT_BF16_HIGH)
    top = _planted_sets(rng, tags, seq.keep, seq.keep_basis, high)
    _lift(kf, dirs, np.concatenate([top[AUDIO], top[VISUAL]]), LIFT_BF16_BOUNDARY)
    return q, to_bf16_bits(kf), top


def prune_cfg2(seed=1):
    """Qwen2.5-Omni-3B-shaped layer: 16/2 heads, D=128; 30 s clip."""
    rng = np.random.default_rng(seed)
    hq, hkv, d = 16, 2, 128
    seq = _single_seq(750, 60 * 144, 64, 64, (0.6, 0.4))
    q, k, top = _bf16_step(rng, hq, hkv, d, seq, high_frac=0.05)
    return PruneCase("cfg2", "bf16", hq, hkv, d, q, k, [seq], {0: top})


def prune_cfg3(seed=2):
    """Qwen2.5-Omni-7B-shaped layer after the pre-LLM stage: 28/4 heads.

    60 s clip: 1500 audio + the pre-LLM visual budget of 7890 tokens
    (R_pre = 0.5 over 1500 + 120*144) + 64 text tokens; keep 0.5 / 0.3.
    """
    rng = np.random.default_rng(seed)
    hq, hkv, d = 28, 4, 128
    seq = _single_seq(1500, 7890, 64, 64, (0.5, 0.3))
    q, k, top = _bf16_step(rng, hq, hkv, d, seq, high_frac=0.05)
    return PruneCase("cfg3", "bf16", hq, hkv, d, q, k, [seq], {0: top})


def prune_joint_layer(seed=5, keep=0.85):
    """Eq. 6 as the paper writes it: the last query token only (q_len = 1)
    and one TopK over all audio and visual candidates.  7B shape after the
    pre-LLM stage (1500 audio + 7890 visual + 64 text); the planted top set
    of size ceil(keep * |S|) is drawn from both modalities together."""
    rng = np.random.default_rng(seed)
    hq, hkv, d = 28, 4, 128
    n_a, n_v, n_t = 1500, 7890, 64
    spans = [(0, n_a, AUDIO), (n_a, n_v, VISUAL)]
    seq = PruneSeq(0, n_a + n_v + n_t, spans, 0, 1, (keep, 0.0), (0, 0), True)
    scale = np.float32(1.0 / math.sqrt(d))
    qf = rng.standard_normal((hq, 1, d), dtype=np.float32) * scale
    q = to_bf16_bits(qf)
    kf = rng.standard_normal((hkv, seq.n_tokens, d), dtype=np.float32) * scale
    dirs = _group_unit_dirs(bf16_bits_to_f32(q), hkv)
    cand = np.flatnonzero(seq.tags() != OTHER)
    top = np.sort(rng.choice(cand, size=_ceil_keep(keep, cand.size), replace=False))
    _lift(kf, dirs, top, LIFT_BF16_BOUNDARY)
    return PruneCase("joint", "bf16", hq, hkv, d, q, to_bf16_bits(kf), [seq], {0: {"joint": top}})


def cache_payload(rng, dtype, n_layers, hkv, d, n, hidden_dim, with_pos=True):
    k = [payload_bits(rng, (hkv, n, d), dtype) for _ in range(n_layers)]
    v = [payload_bits(rng, (hkv, n, d), dtype) for _ in range(n_layers)]
    hid = payload_bits(rng, (n, hidden_dim), dtype) if hidden_dim else None
    pos = None
    if with_pos:
        t = np.arange(n, dtype=np.int32)
        pos = np.stack([t, (t * 7) % 1013, (t * 13) % 2039]).astype(np.int32)
    return CacheCase(dtype, hkv, d, hidden_dim, k, v, hid, pos)


def cfg_cache(cfg, case: PruneCase, seed_offset=100):
    """Payload for a single-layer compaction of configs 1-3."""
    rng = np.random.default_rng(case_seed(cfg) + seed_offset)
    hidden = {1: 512, 2: 2048, 3: 3584}[cfg]
    n = case.k.shape[1]
    cc = cache_payload(rng, case.dtype, 1, case.hkv, case.d, n, hidden)
    cc.k_layers[0] = case.k      # the prune layer's own keys are compacted too
    return cc


def case_seed(cfg):
    return {1: 0, 2: 1, 3: 2, 4: 3, 5: 4}[cfg]


# --------------------------------------------------------------------------
# Config 4: long 7B-shaped progressive pruning over a 28-layer cache
# --------------------------------------------------------------------------

CFG4_LAYERS = 28
CFG4_PRUNE_LAYERS = (14, 18, 22)
CFG4_KEEP = (0.7, 0.5, 0.3)


@dataclass
class ProgressiveCase:
    dtype: str
    hq: int
    hkv: int
    d: int
    hidden_dim: int
    n_audio: int
    n_visual: int
    n_text: int
    q_len: int
    prune_layers: tuple
    keeps: tuple
    queries: List[np.ndarray]   # per prune step [Hq, q_len, D] bits
    cache: CacheCase            # full-length cache (prune layers' K included)
    planted: List[dict]         # per step: modality -> planted rows (original numbering)

    def seq(self):
        return _single_seq(self.n_audio, self.n_visual, self.n_text, self.q_len, (0.0, 0.0))


def progressive_case(seed=3, n_audio=7500, n_frames=600, n_text=128, q_len=128,
                     n_layers=CFG4_LAYERS, prune_layers=CFG4_PRUNE_LAYERS,
                     keeps=CFG4_KEEP, hq=28, hkv=4, d=128, hidden_dim=3584,
                     payload=True):
    """5-min clip: 7500 audio + 600x144 visual + 128 text tokens, 28 layers.

    Prune layers 14, 18, 22 keep the cumulative fractions 0.7, 0.5, 0.3 of
    the original audio and visual counts.  The planted top sets are nested:
    each step's set is drawn inside the previous one, and only the prune
    layer of that step carries its lift, so every step's boundary is planted
    on exactly the rows that survive to it.
    """
    rng = np.random.default_rng(seed)
    n_visual = n_frames * TOKENS_PER_FRAME
    n = n_audio + n_visual + n_text
    seq = _single_seq(n_audio, n_visual, n_text, q_len, (0, 0))
    tags = seq.tags()
    scale = np.float32(1.0 / math.sqrt(d))
    if payload:
        cache = cache_payload(rng, "bf16", n_layers, hkv, d, n, hidden_dim)
    else:
        cache = CacheCase("bf16", hkv, d, hidden_dim, [None] * n_layers,
                          [None] * n_layers, None, None)
    queries, planted = [], []
    prev = {m: np.flatnonzero(tags == m) for m in (AUDIO, VISUAL)}
    basis = {m: prev[m].size for m in (AUDIO, VISUAL)}
    for layer, keep in zip(prune_layers, keeps):
        qf = rng.standard_normal((hq, q_len, d), dtype=np.float32) * scale
        qb = to_bf16_bits(qf)
        dirs = _group_unit_dirs(bf16_bits_to_f32(qb), hkv)
        kf = rng.standard_normal((hkv, n, d), dtype=np.float32) * scale
        top = {}
        for m in (AUDIO, VISUAL):
            kk = _ceil_keep(keep, basis[m])
            top[m] = np.sort(rng.choice(prev[m], size=kk, replace=False))
        _lift(kf, dirs, np.concatenate([top[AUDIO], top[VISUAL]]), LIFT_BF16_BOUNDARY)
        cache.k_layers[layer] = to_bf16_bits(kf)
        queries.append(qb)
        planted.append(top)
        prev = top
    return ProgressiveCase("bf16", hq, hkv, d, hidden_dim, n_audio, n_visual, n_text,
                           q_len, tuple(prune_layers), tuple(keeps), queries, cache, planted)


def paper_schedule_case(seed=6, n_audio=7500, n_frames=600, n_text=128, n_layers=CFG4_LAYERS,
                        first_layer=14, drop=0.10, hq=28, hkv=4, d=128, hidden_dim=3584, payload=True):
    """The paper's inner-LLM schedule (Algorithm 1; Section 3.2; Section 4.1
    implementation details): from `first_layer` on, every layer keeps the
    top ceil((1 - drop) |S|) of the current candidates, ranked jointly by the
    last query token's attention.  The planted sets are nested over all
    candidates, each lifted only at its own layer."""
    rng = np.random.default_rng(seed)
    n_visual = n_frames * TOKENS_PER_FRAME
    n = n_audio + n_visual + n_text
    seq = _single_seq(n_audio, n_visual, n_text, 1, (0, 0))
    tags = seq.tags()
    scale = np.float32(1.0 / math.sqrt(d))
    if payload:
        cache = cache_payload(rng, "bf16", n_layers, hkv, d, n, hidden_dim)
    else:
        cache = CacheCase("bf16", hkv, d, hidden_dim, [None] * n_layers, [None] * n_layers, None, None)
    layers = tuple(range(first_layer, n_layers))
    keep = 1.0 - drop
    prev = np.flatnonzero(tags != OTHER)
    queries, planted = [], []
    for layer in layers:
        qb = to_bf16_bits(rng.standard_normal((hq, 1, d), dtype=np.float32) * scale)
        dirs = _group_unit_dirs(bf16_bits_to_f32(qb), hkv)
        kf = rng.standard_normal((hkv, n, d), dtype=np.float32) * scale
        top = np.sort(rng.choice(prev, size=_ceil_keep(keep, prev.size), replace=False))
        _lift(kf, dirs, top, LIFT_BF16_BOUNDARY)
        cache.k_layers[layer] = to_bf16_bits(kf)
        queries.append(qb)
        planted.append({"joint": top})
        prev = top
    return ProgressiveCase("bf16", hq, hkv, d, hidden_dim, n_audio, n_visual, n_text, 1, layers,
                           tuple([keep] * len(layers)), queries, cache, planted)


# --------------------------------------------------------------------------
# Pre-LLM dynamics workloads (local audio-visual structure)
# --------------------------------------------------------------------------

@dataclass
class AVSeq:
    n_frames: int
    per_frame: int
    n_audio: int
    n_query: int
    vis_off: int
    aud_off: int
    qry_off: int
    seg_starts: List[int]       # planted scene starts (frame index)
    structure: str              # "shared" (gate off) or "offset" (gate on)


@dataclass
class DynamicsCase:
    dtype: str
    dim: int
    xv: np.ndarray              # [sum F*P, dim] raw
    xa: np.ndarray              # [sum N_A, dim] raw
    xq: np.ndarray              # [sum n_q, dim] raw
    seqs: List[AVSeq]
    params: dict


def _scene_lengths(rng, n_frames, lo=8, hi=24):
    """Planted scene lengths, each >= lo frames (so smoothed cuts stay apart)."""
    if n_frames < 2 * lo:
        return [n_frames]
    out = []
    left = n_frames
    while left > 0:
        if left < 2 * lo:
            out.append(left)
            break
        L = int(rng.integers(lo, min(hi, left - lo) + 1))
        out.append(L)
        left -= L
    return out


def _unit(rng, shape, dim):
    x = rng.standard_normal(shape + (dim,), dtype=np.float32)
    return x / np.linalg.norm(x, axis=-1, keepdims=True)


def av_clip(rng, n_frames, per_frame, n_audio, n_query, dim, structure,
            n_objects=8, drift_step=0.10, audio_swing=0.30):
    """Embeddings of one clip with planted scenes and local dynamics.

    Visual token (f, p) of scene m: 0.6 scene_m + object_{m, c(p)} +
    0.2 detail_{m, p} + drift_V(f) b_m + 0.3 noise.  Tokens of one object
    cluster are close (cosine about 0.9) and clusters are far apart (about
    0.25), so coverage counts sit away from their threshold.  Audio token n
    of scene m: 0.5 scene_m + audio_m + drift_A(f(n)) a_m + 0.3 noise.

    ``shared``: drift_A = drift_V = a per-scene random walk (local
    co-variation, high window CKA).  ``offset``: audio swings +-audio_swing
    on alternate frames while the visual drift is a per-scene linear trend
    (orthogonal temporal patterns, low window CKA).

    The query embeds scene cues from one or two scenes plus noise.
    """
    lens = _scene_lengths(rng, n_frames)
    starts = np.cumsum([0] + lens[:-1]).tolist()
    n_sc = len(lens)
    scene = _unit(rng, (n_sc,), dim)
    objects = _unit(rng, (n_sc, n_objects), dim)
    detail = _unit(rng, (n_sc, per_frame), dim)
    bdir = _unit(rng, (n_sc,), dim)
    adir = _unit(rng, (n_sc,), dim)
    audio_sc = _unit(rng, (n_sc,), dim)
    cluster = rng.integers(0, n_objects, size=(n_sc, per_frame))
    frame_scene = np.repeat(np.arange(n_sc), lens)
    drift_v = np.zeros(n_frames, dtype=np.float32)
    drift_a = np.zeros(n_frames, dtype=np.float32)
    for m, (s0, L) in enumerate(zip(starts, lens)):
        f = np.arange(L, dtype=np.float32)
        if structure == "shared":
            walk = np.cumsum(rng.standard_normal(L).astype(np.float32)) * drift_step
            walk -= walk.mean()
            drift_v[s0:s0 + L] = walk
            drift_a[s0:s0 + L] = walk
        else:
            drift_v[s0:s0 + L] = (f - (L - 1) / 2.0) * drift_step
            drift_a[s0:s0 + L] = np.where(np.arange(L) % 2 == 0, -audio_swing, audio_swing)
    xv = np.empty((n_frames, per_frame, dim), dtype=np.float32)
    for f in range(n_frames):
        m = frame_scene[f]
        xv[f] = (0.6 * scene[m] + objects[m, cluster[m]] + 0.2 * detail[m]
                 + drift_v[f] * bdir[m]
                 + 0.3 * _unit(rng, (per_frame,), dim))
    xv = xv.reshape(n_frames * per_frame, dim)
    # Audio rows follow the frame axis at n_audio / n_frames rows per frame.
    af = np.minimum((np.arange(n_audio) * n_frames) // max(n_audio, 1), n_frames - 1)
    am = frame_scene[af]
    xa = (0.5 * scene[am] + audio_sc[am] + drift_a[af, None] * adir[am]
          + 0.3 * _unit(rng, (n_audio,), dim)).astype(np.float32)
    picks = rng.choice(n_sc, size=min(2, n_sc), replace=False)
    cue = scene[picks].sum(axis=0) + objects[picks[0], 0]
    xq = (cue[None, :] + 0.8 * _unit(rng, (n_query,), dim)).astype(np.float32)
    return xv, xa, xq, starts


def dynamics_cfg3(structure="offset", seed=2, dim=3584, window=4, seconds=60,
                  n_query=64):
    """60 s clip at the 7B shape: 1500 audio + 120x144 visual, 64 query rows."""
    rng = np.random.default_rng(seed + (0 if structure == "shared" else 500))
    F = seconds * FRAMES_PER_SECOND
    NA = seconds * AUDIO_PER_SECOND
    xv, xa, xq, starts = av_clip(rng, F, TOKENS_PER_FRAME, NA, n_query, dim, structure)
    seq = AVSeq(F, TOKENS_PER_FRAME, NA, n_query, 0, 0, 0, starts, structure)
    params = {"window": window, "r_pre": 0.5}
    return DynamicsCase("bf16", dim, to_bf16_bits(xv), to_bf16_bits(xa), to_bf16_bits(xq),
                        [seq], params)


def dynamics_small(structure="offset", seed=7, dim=64, frames=24, per_frame=16,
                   audio=300, n_query=8, window=3):
    """Reduced clip with the same recipe, sized for CPU-speed parity cases."""
    rng = np.random.default_rng(seed + (0 if structure == "shared" else 500))
    xv, xa, xq, starts = av_clip(rng, frames, per_frame, audio, n_query, dim, structure)
    seq = AVSeq(frames, per_frame, audio, n_query, 0, 0, 0, starts, structure)
    return DynamicsCase("bf16", dim, to_bf16_bits(xv), to_bf16_bits(xa), to_bf16_bits(xq),
                        [seq], {"window": window, "r_pre": 0.5})


def dynamics_edge(structure="offset", seed=75, dim=64, frames=64, per_frame=16, audio=600,
                  n_query=8, window=3):
    """A clip with the scorer's degenerate inputs, built on the planted-scene
    recipe (raw bits are copied, so repeats are bitwise):

    - frame 0 is all zeros (zero-norm frame: its own segment, cosines 0);
    - the shortest scene after the first is static: every frame repeats the
      scene's first frame, and its audio rows repeat one audio token, so its
      CKA windows have no variation and its non-anchor frames equal their
      anchor;
    - the first dynamic anchor repeats its token 0 in tokens 1-4 (exact
      duplicates inside a DA-FPS frame);
    - single zero tokens in the static anchor, in a dynamic anchor and in a
      non-anchor frame, and two zero audio rows.
    """
    rng = np.random.default_rng(seed + (0 if structure == "shared" else 500))
    xv, xa, xq, starts = av_clip(rng, frames, per_frame, audio, n_query, dim, structure)
    xv = to_bf16_bits(xv).reshape(frames, per_frame, dim)
    xa = to_bf16_bits(xa)
    lens = [b - a for a, b in zip(starts, starts[1:] + [frames])]
    st = min(range(1, len(starts)), key=lambda m: (lens[m], m))
    s0, L = starts[st], lens[st]
    xv[s0][3] = 0                                   # zero token in the static anchor
    xv[s0 + 1:s0 + L] = xv[s0]
    af = np.minimum((np.arange(audio) * frames) // audio, frames - 1)
    rows = np.flatnonzero((af >= s0) & (af < s0 + L))
    xa[rows] = xa[rows[0]]
    dyn = starts[1] if st != 1 else starts[2]
    xv[dyn][1:5] = xv[dyn][0]                       # duplicates inside an anchor frame
    xv[dyn][9] = 0                                  # zero token in a dynamic anchor
    xv[dyn + 2][5] = 0                              # zero token in a non-anchor frame
    xa[[3, audio // 2]] = 0                         # zero audio rows
    xv[0] = 0                                       # zero frame: a segment of its own
    seg_starts = sorted(set([0, 1] + starts[1:]))
    seq = AVSeq(frames, per_frame, audio, n_query, 0, 0, 0, seg_starts, structure)
    return DynamicsCase("bf16", dim, xv.reshape(frames * per_frame, dim), xa, to_bf16_bits(xq),
                        [seq], {"window": window, "r_pre": 0.5})


# --------------------------------------------------------------------------
# Config 5: ragged batch of 8 clips (scorer + one prune + compaction)
# --------------------------------------------------------------------------

@dataclass
class RaggedCase:
    seconds: List[int]
    dynamics: DynamicsCase
    prune: PruneCase
    cache: CacheCase


def ragged_batch(seed=4, n_seq=8, t_lo=20, t_hi=300, q_lo=32, q_hi=128, dim=3584,
                 hq=28, hkv=4, d=128, hidden_dim=3584, window=3, r_pre=0.5,
                 keep=(0.5, 0.3), payload=True):
    """Ragged batch at the 7B shape.

    Clip lengths T_i ~ U{t_lo..t_hi} s and query spans ~ U{q_lo..q_hi}; even
    clips carry the shared-drift structure (gate stays off), odd clips the
    offset structure (gate fires).  The prune step sees each clip as
    2-second chunks of [visual | audio] followed by the text span, with the
    pre-LLM visual budget spread evenly over the chunks.
    """
    rng = np.random.default_rng(seed)
    secs = rng.integers(t_lo, t_hi + 1, size=n_seq).tolist()
    nqs = rng.integers(q_lo, q_hi + 1, size=n_seq).tolist()
    xv_l, xa_l, xq_l, av = [], [], [], []
    vo = ao = qo = 0
    for i, (T, nq) in enumerate(zip(secs, nqs)):
        F, NA = T * FRAMES_PER_SECOND, T * AUDIO_PER_SECOND
        structure = "shared" if i % 2 == 0 else "offset"
        xv, xa, xq, starts = av_clip(rng, F, TOKENS_PER_FRAME, NA, nq, dim, structure)
        xv_l.append(to_bf16_bits(xv))
        xa_l.append(to_bf16_bits(xa))
        xq_l.append(to_bf16_bits(xq))
        av.append(AVSeq(F, TOKENS_PER_FRAME, NA, nq, vo, ao, qo, starts, structure))
        vo += F * TOKENS_PER_FRAME
        ao += NA
        qo += nq
    dyn = DynamicsCase("bf16", dim, np.concatenate(xv_l), np.concatenate(xa_l),
                       np.concatenate(xq_l), av, {"window": window, "r_pre": r_pre})
    # Stage-2 layout.
    seqs, tok = [], 0
    qrow = 0
    for T, nq in zip(secs, nqs):
        F, NA = T * FRAMES_PER_SECOND, T * AUDIO_PER_SECOND
        bv = max(0, min(_ceil_keep(r_pre, NA + F * TOKENS_PER_FRAME) - NA, F * TOKENS_PER_FRAME))
        n_chunks = max(1, T // 2)
        vis = [bv // n_chunks + (1 if c < bv % n_chunks else 0) for c in range(n_chunks)]
        aud = [NA // n_chunks + (1 if c < NA % n_chunks else 0) for c in range(n_chunks)]
        spans, row = [], 0
        for c in range(n_chunks):
            if vis[c]:
                spans.append((row, vis[c], VISUAL))
                row += vis[c]
            if aud[c]:
                spans.append((row, aud[c], AUDIO))
                row += aud[c]
        n = row + nq
        seqs.append(PruneSeq(tok, n, spans, qrow, nq, keep))
        tok += n
        qrow += nq
    scale = np.float32(1.0 / math.sqrt(d))
    qf = rng.standard_normal((hq, qrow, d), dtype=np.float32) * scale
    qb = to_bf16_bits(qf)
    qv = bf16_bits_to_f32(qb)
    kf = rng.standard_normal((hkv, tok, d), dtype=np.float32) * scale
    top_all = {}
    for i, s in enumerate(seqs):
        dirs = _group_unit_dirs(qv[:, s.q_off:s.q_off + s.q_len], hkv)
        top = _planted_sets(rng, s.tags(), s.keep, s.keep_basis)
        rows = s.tok_off + np.concatenate([top[AUDIO], top[VISUAL]])
        sub = kf[:, s.tok_off:s.tok_off + s.n_tokens]
        _lift(sub, dirs, rows - s.tok_off, LIFT_BF16_BOUNDARY)
        top_all[i] = top
    kb = to_bf16_bits(kf)
    prune = PruneCase("cfg5", "bf16", hq, hkv, d, qb, kb, seqs, top_all)
    if payload:
        cache = cache_payload(rng, "bf16", 1, hkv, d, tok, hidden_dim)
        cache.k_layers[0] = kb
    else:
        cache = None
    return RaggedCase(secs, dyn, prune, cache)
