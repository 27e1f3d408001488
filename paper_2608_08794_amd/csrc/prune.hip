// In-LLM query-conditioned prune (Section 3.2, Eq. 5 and Eq. 6) on gfx950.
//
// Per sequence and prune layer:
//   I_j = 1/(Hq*T) * sum_{h,t} softmax_{j in S}( q[h,t] . k[h/(Hq/Hkv), j] / sqrt(D) )
// followed by a per-modality top-k with the lower row winning ties, and the
// ascending list of kept rows.
//
// Kernels (all on the caller's stream, no host synchronisation):
//   k_rowstats   pass 1: per query row, online (max, sum exp2) over a chunk
//                of keys; logits from MFMA with Q fragments resident in VGPRs
//                and K tiles staged through padded, double-buffered LDS.
//   k_rowreduce  combines the chunk partials of every query row (fixed order)
//                into b_r = max_r + log2(Z_r).
//   k_colsum     pass 2: recomputes the logits with the roles of the MFMA
//                operands swapped so the per-key sum over query rows is
//                lane-local, then a fixed-order cross-wave sum through LDS.
//   k_finalize   sums the per-group partials in a fixed order into I_j.
//   k_select     per (sequence, modality): 4-pass 8-bit radix select over the
//                fp32 score bits (scores are >= 0, so the bits are ordered).
//   k_scan       per sequence: keep mask and ordered compaction of kept rows.
#include <cfloat>
#include <cmath>
#include <vector>

#include "common.hpp"
#include "prune_plan.hpp"

namespace apack {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned short bf16_t;

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// Element traits: the MFMA used for each input type.
//   bf16: v_mfma_f32_32x32x16_bf16, 8 consecutive k per lane and k-step.
//   f32 : v_mfma_f32_32x32x2_f32,   1 k per lane and k-step.
// In both, lane l supplies row (l % 32) of A / column (l % 32) of B for the
// k half selected by l / 32, and the 32x32 result puts column (l % 32) and
// rows 8*(e/4) + 4*(l/32) + (e%4) in accumulator element e.
// ---------------------------------------------------------------------------
template <class T> struct Mma;

template <> struct Mma<bf16_t> {
  using frag = bf16x8;
  static constexpr int kstep = 16;        // k per MFMA
  static constexpr int lane_k = 8;        // k per lane per MFMA
  static __device__ __forceinline__ f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ frag zero() { return frag{}; }
};

template <> struct Mma<float> {
  using frag = float;
  static constexpr int kstep = 2;
  static constexpr int lane_k = 1;
  static __device__ __forceinline__ f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ frag zero() { return 0.0f; }
};

template <class T, int D>
struct TileGeom {
  static constexpr int kRowBytes = D * (int)sizeof(T);
  static constexpr int kPitch = kRowBytes + 16;      // padded LDS row (bytes)
  static constexpr int kUnits = kRowBytes / 16;      // 16-byte units per row
  static constexpr int kTileBytes = kKeyTile * kPitch;
  static constexpr int kSteps = D / Mma<T>::kstep;
};

// Query fragments of the 64 rows a wave owns (two blocks of 32), loaded once.
template <class T, int D>
struct QFrags {
  typename Mma<T>::frag v[2][TileGeom<T, D>::kSteps];
};

template <class T, int D>
__device__ __forceinline__ void load_q(QFrags<T, D>& qfr, const T* q, int64_t q_hs, const SeqDev& sq, int g,
                                       int n_rep, int row0, int lane) {
  using M = Mma<T>;
  auto& qf = qfr.v;
  const int rows = n_rep * sq.q_len;
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    const int rho = row0 + rb * 32 + (lane & 31);
    const bool ok = rho < rows;
    const int h = g * n_rep + (ok ? rho / sq.q_len : 0);
    const int t = ok ? rho % sq.q_len : 0;
    const T* src = q + (int64_t)h * q_hs + (sq.q_off + t) * (int64_t)D + (lane >> 5) * M::lane_k;
#pragma unroll
    for (int ks = 0; ks < TileGeom<T, D>::kSteps; ++ks)
      qf[rb][ks] = ok ? *reinterpret_cast<const typename M::frag*>(src + ks * M::kstep) : M::zero();
  }
}

// Global -> register staging of one key tile (kKeyTile rows of D elements).
template <class T, int D, int NW>
struct KStage {
  using G = TileGeom<T, D>;
  static constexpr int kPer = (kKeyTile * G::kUnits + NW * kWave - 1) / (NW * kWave);
  uint4 r[kPer];
  __device__ __forceinline__ void load(const T* kbase, int64_t row0, int64_t n_rows, int tid) {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int u = tid + i * NW * kWave;
      const int row = u / G::kUnits, col = u % G::kUnits;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (row < kKeyTile && row0 + row < n_rows)
        v = *reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(kbase + (row0 + row) * D) + col * 16);
      r[i] = v;
    }
  }
  __device__ __forceinline__ void store(char* lds, int tid) const {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int u = tid + i * NW * kWave;
      const int row = u / G::kUnits, col = u % G::kUnits;
      if (row < kKeyTile) *reinterpret_cast<uint4*>(lds + row * G::kPitch + col * 16) = r[i];
    }
  }
};

template <class T, int D>
__device__ __forceinline__ typename Mma<T>::frag lds_frag(const char* lds, int key, int ks, int lane) {
  using M = Mma<T>;
  const char* p = lds + key * TileGeom<T, D>::kPitch + (ks * M::kstep + (lane >> 5) * M::lane_k) * (int)sizeof(T);
  return *reinterpret_cast<const typename M::frag*>(p);
}

__device__ __forceinline__ void row_of(const SeqDev& sq, int g, int n_rep, int rho, int& r) {
  const int h = g * n_rep + rho / sq.q_len;
  r = h * sq.q_len + rho % sq.q_len;
}

// ---------------------------------------------------------------------------
// Pass 1: per query row, online max and sum of exp2 over one key chunk.
// ---------------------------------------------------------------------------
template <class T, int D, int NW>
__global__ __launch_bounds__(NW * kWave) void k_rowstats(const SeqDev* __restrict__ seqs,
                                                         const TileDev* __restrict__ tiles,
                                                         const uint8_t* __restrict__ tags,
                                                         const T* __restrict__ q, int64_t q_hs,
                                                         const T* __restrict__ k, int64_t k_hs,
                                                         int n_rep, float scale_log2,
                                                         float2* __restrict__ stats) {
  using G = TileGeom<T, D>;
  using M = Mma<T>;
  __shared__ __attribute__((aligned(16))) char lds[2][G::kTileBytes];
  __shared__ uint8_t ltag[2][kKeyTile];

  const TileDev tl = tiles[blockIdx.x];
  const SeqDev sq = seqs[tl.seq];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int rows_g = n_rep * sq.q_len;
  const int row0 = tl.rg * sq.rows_per_rg + wave * 64;
  const bool active = row0 < rows_g && row0 < (tl.rg + 1) * sq.rows_per_rg;

  QFrags<T, D> qfr;
  auto& qf = qfr.v;
  if (active) load_q<T, D>(qfr, q, q_hs, sq, tl.g, n_rep, row0, lane);

  const int64_t key_begin = (int64_t)tl.chunk * sq.chunk;
  int64_t key_end = key_begin + sq.chunk;
  if (key_end > sq.n_tokens) key_end = sq.n_tokens;
  const int n_tiles = (int)((key_end - key_begin + kKeyTile - 1) / kKeyTile);
  const T* kbase = k + (int64_t)tl.g * k_hs + sq.tok_off * D;
  const uint8_t* tg = tags + sq.tag_off;

  float m_run[2] = {-FLT_MAX, -FLT_MAX}, s_run[2] = {0.f, 0.f};

  KStage<T, D, NW> st;
  st.load(kbase, key_begin, key_end, tid);
  for (int it = 0; it < n_tiles; ++it) {
    const int buf = it & 1;
    const int64_t t0 = key_begin + (int64_t)it * kKeyTile;
    st.store(lds[buf], tid);
    if (tid < kKeyTile) ltag[buf][tid] = (t0 + tid < key_end) ? tg[t0 + tid] : 0;
    __syncthreads();
    if (it + 1 < n_tiles) st.load(kbase, t0 + kKeyTile, key_end, tid);
    if (active) {
#pragma unroll
      for (int kb = 0; kb < kKeyTile / 32; ++kb) {
        f32x16 acc[2] = {f32x16{}, f32x16{}};
#pragma unroll
        for (int ks = 0; ks < G::kSteps; ++ks) {
          const auto kf = lds_frag<T, D>(lds[buf], kb * 32 + (lane & 31), ks, lane);
          acc[0] = M::mma(kf, qf[0][ks], acc[0]);
          acc[1] = M::mma(kf, qf[1][ks], acc[1]);
        }
        // acc[rb][e]: query column (lane % 32) of block rb, key row
        // kb*32 + 8*(e/4) + 4*(lane/32) + e%4.
        bool valid[16];
#pragma unroll
        for (int e = 0; e < 16; ++e)
          valid[e] = ltag[buf][kb * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3)] != 0;
#pragma unroll
        for (int rb = 0; rb < 2; ++rb) {
          float x[16];
          float lmax = -FLT_MAX;
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            x[e] = valid[e] ? acc[rb][e] * scale_log2 : -INFINITY;
            lmax = fmaxf(lmax, x[e]);
          }
          const float m_new = fmaxf(m_run[rb], lmax);
          float s = s_run[rb] * exp2f(m_run[rb] - m_new);
#pragma unroll
          for (int e = 0; e < 16; ++e) s += exp2f(x[e] - m_new);
          s_run[rb] = s;
          m_run[rb] = m_new;
        }
      }
    }
  }
  if (!active) return;
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    const float mo = __shfl_xor(m_run[rb], 32);
    const float so = __shfl_xor(s_run[rb], 32);
    const float mm = fmaxf(m_run[rb], mo);
    const float ss = s_run[rb] * exp2f(m_run[rb] - mm) + so * exp2f(mo - mm);
    const int rho = row0 + rb * 32 + lane;
    if (lane < 32 && rho < rows_g && rho < (tl.rg + 1) * sq.rows_per_rg) {
      int r;
      row_of(sq, tl.g, n_rep, rho, r);
      stats[sq.stats_off + (int64_t)r * sq.n_chunks + tl.chunk] = make_float2(mm, ss);
    }
  }
}

// ---------------------------------------------------------------------------
// Combine chunk partials of every query row: b_r = M_r + log2(Z_r).
// One wave per row; lanes stride the chunks; fixed-order tree merge.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void merge(float& m, float& s, float mo, float so) {
  const float mm = fmaxf(m, mo);
  s = s * exp2f(m - mm) + so * exp2f(mo - mm);
  m = mm;
}

__global__ __launch_bounds__(256) void k_rowreduce(const SeqDev* __restrict__ seqs, int n_seq,
                                                   int64_t total_rows, const float2* __restrict__ stats,
                                                   float* __restrict__ bias) {
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= total_rows) return;
  int lo = 0, hi = n_seq - 1;
  while (lo < hi) {  // last sequence whose bias_off <= row
    const int mid = (lo + hi + 1) >> 1;
    if (seqs[mid].bias_off <= row) lo = mid; else hi = mid - 1;
  }
  const SeqDev& sq = seqs[lo];
  const int64_t r = row - sq.bias_off;
  const float2* p = stats + sq.stats_off + r * sq.n_chunks;
  float m = -FLT_MAX, s = 0.f;
  for (int c = lane; c < sq.n_chunks; c += 64) merge(m, s, p[c].x, p[c].y);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float mo = __shfl_xor(m, off), so = __shfl_xor(s, off);
    merge(m, s, mo, so);
  }
  if (lane == 0) bias[row] = (s > 0.f) ? m + log2f(s) : INFINITY;
}

// ---------------------------------------------------------------------------
// Pass 2: per key, sum over this group's query rows of exp2(x - b_r).
// ---------------------------------------------------------------------------
template <class T, int D, int NW>
__global__ __launch_bounds__(NW * kWave) void k_colsum(const SeqDev* __restrict__ seqs,
                                                       const TileDev* __restrict__ tiles,
                                                       const uint8_t* __restrict__ tags,
                                                       const T* __restrict__ q, int64_t q_hs,
                                                       const T* __restrict__ k, int64_t k_hs,
                                                       int n_rep, float scale_log2,
                                                       const float* __restrict__ bias,
                                                       float* __restrict__ colpart) {
  using G = TileGeom<T, D>;
  using M = Mma<T>;
  __shared__ __attribute__((aligned(16))) char lds[2][G::kTileBytes];
  __shared__ float red[2][NW][kKeyTile];

  const TileDev tl = tiles[blockIdx.x];
  const SeqDev sq = seqs[tl.seq];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int rows_g = n_rep * sq.q_len;
  const int rg_end = min(rows_g, (tl.rg + 1) * sq.rows_per_rg);
  const int row0 = tl.rg * sq.rows_per_rg + wave * 64;
  const bool active = row0 < rg_end;
  const int n_active = (rg_end - tl.rg * sq.rows_per_rg + 63) / 64;

  QFrags<T, D> qfr;
  auto& qf = qfr.v;
  float b[2][16];
  if (active) {
    load_q<T, D>(qfr, q, q_hs, sq, tl.g, n_rep, row0, lane);
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int rho = row0 + rb * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        float v = INFINITY;
        if (rho < rg_end) {
          int r;
          row_of(sq, tl.g, n_rep, rho, r);
          v = bias[sq.bias_off + r];
        }
        b[rb][e] = v;
      }
  }

  const int64_t key_begin = (int64_t)tl.chunk * sq.chunk;
  int64_t key_end = key_begin + sq.chunk;
  if (key_end > sq.n_tokens) key_end = sq.n_tokens;
  const int n_tiles = (int)((key_end - key_begin + kKeyTile - 1) / kKeyTile);
  const T* kbase = k + (int64_t)tl.g * k_hs + sq.tok_off * D;
  float* out = colpart + sq.colpart_off + (int64_t)(tl.g * sq.n_rg + tl.rg) * sq.n_tokens;

  KStage<T, D, NW> st;
  st.load(kbase, key_begin, key_end, tid);
  for (int it = 0; it < n_tiles; ++it) {
    const int buf = it & 1;
    const int64_t t0 = key_begin + (int64_t)it * kKeyTile;
    st.store(lds[buf], tid);
    __syncthreads();
    // Reduce the previous tile's per-wave sums (its buffer is now stable).
    if (it > 0 && tid < kKeyTile) {
      const int64_t key = t0 - kKeyTile + tid;
      float v = 0.f;
      for (int w = 0; w < n_active; ++w) v += red[buf ^ 1][w][tid];
      if (key < key_end) out[key] = v;
    }
    if (it + 1 < n_tiles) st.load(kbase, t0 + kKeyTile, key_end, tid);
    if (active) {
#pragma unroll
      for (int kb = 0; kb < kKeyTile / 32; ++kb) {
        f32x16 acc[2] = {f32x16{}, f32x16{}};
#pragma unroll
        for (int ks = 0; ks < G::kSteps; ++ks) {
          const auto kf = lds_frag<T, D>(lds[buf], kb * 32 + (lane & 31), ks, lane);
          acc[0] = M::mma(qf[0][ks], kf, acc[0]);
          acc[1] = M::mma(qf[1][ks], kf, acc[1]);
        }
        // acc[rb][e]: key column kb*32 + lane%32, query row 8*(e/4)+4*(lane/32)+e%4.
        float cs = 0.f;
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
#pragma unroll
          for (int e = 0; e < 16; ++e) cs += exp2f(fmaf(acc[rb][e], scale_log2, -b[rb][e]));
        cs += __shfl_xor(cs, 32);
        if (lane < 32) red[buf][wave][kb * 32 + lane] = cs;
      }
    }
  }
  __syncthreads();
  if (n_tiles > 0 && tid < kKeyTile) {
    const int buf = (n_tiles - 1) & 1;
    const int64_t key = key_begin + (int64_t)(n_tiles - 1) * kKeyTile + tid;
    float v = 0.f;
    for (int w = 0; w < n_active; ++w) v += red[buf][w][tid];
    if (key < key_end) out[key] = v;
  }
}

// ---------------------------------------------------------------------------
// I_j = (sum over groups, fixed order) / (Hq * T); 0 for non-candidates.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_finalize(const SeqDev* __restrict__ seqs, int n_seq,
                                                  int64_t total_tok, const uint8_t* __restrict__ tags,
                                                  const float* __restrict__ colpart, int hq, int hkv,
                                                  float* __restrict__ scores) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total_tok) return;
  int lo = 0, hi = n_seq - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (seqs[mid].tag_off <= i) lo = mid; else hi = mid - 1;
  }
  const SeqDev& sq = seqs[lo];
  const int64_t j = i - sq.tag_off;
  float v = 0.f;
  if (tags[i] != 0 && sq.n_cand > 0) {
    const float* p = colpart + sq.colpart_off + j;
    const int planes = hkv * sq.n_rg;
    for (int pl = 0; pl < planes; ++pl) v += p[(int64_t)pl * sq.n_tokens];
    v = v / (float)(hq * sq.q_len);
  }
  scores[sq.tok_off + j] = v;
}

// ---------------------------------------------------------------------------
// Block-wide inclusive scan of 32-bit values (blockDim = NT, multiple of 64).
// ---------------------------------------------------------------------------
template <int NT>
__device__ __forceinline__ uint32_t block_incl_scan(uint32_t v, uint32_t* sh_wave, uint32_t& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t o = __shfl_up(v, off);
    if (lane >= off) v += o;
  }
  if (lane == 63) sh_wave[wave] = v;
  __syncthreads();
  uint32_t base = 0;
  total = 0;
#pragma unroll
  for (int w = 0; w < NT / 64; ++w) {
    const uint32_t x = sh_wave[w];
    if (w < wave) base += x;
    total += x;
  }
  __syncthreads();
  return v + base;
}

// ---------------------------------------------------------------------------
// Radix select of the k-th largest score bits of (sequence, modality).
// ---------------------------------------------------------------------------
constexpr int kSelThreads = 1024;

__global__ __launch_bounds__(kSelThreads) void k_select(SeqDev* __restrict__ seqs,
                                                        const uint8_t* __restrict__ tags,
                                                        const float* __restrict__ scores) {
  const int s = blockIdx.x >> 1, mi = blockIdx.x & 1;
  SeqDev* sq = &seqs[s];
  if (!sq->select[mi]) return;
  const uint8_t mod = (uint8_t)(mi + 1);
  const uint8_t* tg = tags + sq->tag_off;
  const uint32_t* sb = reinterpret_cast<const uint32_t*>(scores + sq->tok_off);
  const int64_t n = sq->n_tokens;
  const int tid = threadIdx.x, lane = tid & 63;

  __shared__ uint32_t hist[256];
  __shared__ uint32_t sh_wave[kSelThreads / 64];
  __shared__ uint32_t sh_prefix, sh_kk, sh_eq;

  uint32_t prefix = 0, mask = 0, kk = (uint32_t)sq->k_sel[mi], n_eq = 0;
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    if (tid < 256) hist[tid] = 0;
    __syncthreads();
    for (int64_t base = 0; base < n; base += kSelThreads) {
      const int64_t i = base + tid;
      bool part = false;
      uint32_t digit = 0;
      if (i < n && tg[i] == mod) {
        const uint32_t bits = sb[i];
        if ((bits & mask) == prefix) {
          part = true;
          digit = (bits >> shift) & 0xFFu;
        }
      }
      // Wave-aggregated increments for the few most common digits, then
      // plain atomics for whatever is left.
      uint64_t act = __ballot(part);
      for (int round = 0; round < 4 && act; ++round) {
        const int leader = __ffsll((unsigned long long)act) - 1;
        const uint32_t ld = __shfl(digit, leader);
        const uint64_t same = __ballot(part && digit == ld);
        if (lane == leader) atomicAdd(&hist[ld], (uint32_t)__popcll(same));
        if (part && digit == ld) part = false;
        act &= ~same;
      }
      if (part) atomicAdd(&hist[digit], 1u);
    }
    __syncthreads();
    // Digit holding the kk-th largest: scan the histogram from digit 255 down.
    uint32_t v = 0;
    if (tid < 256) v = hist[255 - tid];
    uint32_t total;
    const uint32_t cum = block_incl_scan<kSelThreads>(tid < 256 ? v : 0u, sh_wave, total);
    if (tid < 256 && cum >= kk && cum - v < kk) {
      const uint32_t d = 255u - (uint32_t)tid;
      sh_prefix = prefix | (d << shift);
      sh_kk = kk - (cum - v);
      sh_eq = v;
    }
    __syncthreads();
    prefix = sh_prefix;
    kk = sh_kk;
    n_eq = sh_eq;
    mask |= 0xFFu << shift;
    __syncthreads();
  }
  if (tid == 0) {
    sq->thr[mi] = prefix;
    sq->need[mi] = (int32_t)kk;
    sq->all_eq[mi] = (kk == n_eq) ? 1 : 0;
  }
}

// ---------------------------------------------------------------------------
// Keep mask and ordered compaction of the kept rows of one sequence.
// ---------------------------------------------------------------------------
constexpr int kScanThreads = 1024;
constexpr int kScanPer = 4;

__global__ __launch_bounds__(kScanThreads) void k_scan(const SeqDev* __restrict__ seqs,
                                                       const uint8_t* __restrict__ tags,
                                                       const float* __restrict__ scores,
                                                       int32_t* __restrict__ kept) {
  const SeqDev& sq = seqs[blockIdx.x];
  const uint8_t* tg = tags + sq.tag_off;
  const uint32_t* sb = reinterpret_cast<const uint32_t*>(scores + sq.tok_off);
  const int64_t n = sq.n_tokens;
  const int tid = threadIdx.x;
  __shared__ uint32_t sh_wave[kScanThreads / 64];
  const uint32_t thr[2] = {sq.thr[0], sq.thr[1]};
  const uint32_t need[2] = {(uint32_t)sq.need[0], (uint32_t)sq.need[1]};
  const bool ranked = !(sq.all_eq[0] && sq.all_eq[1]);
  uint32_t carry_eq[2] = {0, 0};
  uint32_t carry_keep = 0;
  int32_t* out = kept + sq.out_off;

  for (int64_t base = 0; base < n; base += (int64_t)kScanThreads * kScanPer) {
    uint8_t mtag[kScanPer];
    uint32_t bits[kScanPer];
    uint32_t n_eq_a = 0, n_eq_v = 0;
#pragma unroll
    for (int u = 0; u < kScanPer; ++u) {
      const int64_t i = base + (int64_t)tid * kScanPer + u;
      mtag[u] = i < n ? tg[i] : 0xFF;
      bits[u] = i < n ? sb[i] : 0u;
      if (mtag[u] == 1 && bits[u] == thr[0]) ++n_eq_a;
      if (mtag[u] == 2 && bits[u] == thr[1]) ++n_eq_v;
    }
    uint32_t rank[2] = {0, 0};
    if (ranked) {
      uint32_t tot;
      const uint32_t packed = n_eq_a | (n_eq_v << 16);
      const uint32_t incl = block_incl_scan<kScanThreads>(packed, sh_wave, tot);
      const uint32_t excl = incl - packed;
      rank[0] = carry_eq[0] + (excl & 0xFFFFu);
      rank[1] = carry_eq[1] + (excl >> 16);
      carry_eq[0] += tot & 0xFFFFu;
      carry_eq[1] += tot >> 16;
    }
    bool keep[kScanPer];
    uint32_t n_keep = 0;
#pragma unroll
    for (int u = 0; u < kScanPer; ++u) {
      bool kp;
      const uint8_t m = mtag[u];
      if (m == 0xFF) kp = false;
      else if (m == 0) kp = true;
      else {
        const int mi = m - 1;
        if (bits[u] > thr[mi]) kp = true;
        else if (bits[u] == thr[mi]) kp = (rank[mi]++ < need[mi]);
        else kp = false;
      }
      keep[u] = kp;
      n_keep += kp;
    }
    uint32_t tot;
    const uint32_t incl = block_incl_scan<kScanThreads>(n_keep, sh_wave, tot);
    uint32_t pos = carry_keep + incl - n_keep;
#pragma unroll
    for (int u = 0; u < kScanPer; ++u)
      if (keep[u]) {
        if (pos < (uint64_t)sq.n_kept) out[pos] = (int32_t)(sq.tok_off + base + (int64_t)tid * kScanPer + u);
        ++pos;
      }
    carry_keep += tot;
  }
}

// ---------------------------------------------------------------------------
// Host launch sequence.
// ---------------------------------------------------------------------------
template <class T, int D, int NW>
apack_status launch_scores_t(const PrunePlan& pl, const DevPtrs& dp, const void* q, int64_t q_hs,
                             const void* k, int64_t k_hs, int n_rep, hipStream_t stream) {
  const float scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)D));
  const int nt = (int)pl.tiles.size();
  if (nt > 0) {
    hipLaunchKernelGGL((k_rowstats<T, D, NW>), dim3(nt), dim3(NW * kWave), 0, stream, dp.seqs, dp.tiles,
                       dp.tags, (const T*)q, q_hs, (const T*)k, k_hs, n_rep, scale_log2, dp.stats);
    APACK_CHECK(launch_status("k_rowstats") == APACK_OK, APACK_E_HIP, "%s", apack_last_error());
    const int64_t rows = pl.total_rows;
    hipLaunchKernelGGL(k_rowreduce, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, stream, dp.seqs,
                       (int)pl.seqs.size(), rows, dp.stats, dp.bias);
    APACK_CHECK(launch_status("k_rowreduce") == APACK_OK, APACK_E_HIP, "%s", apack_last_error());
    hipLaunchKernelGGL((k_colsum<T, D, NW>), dim3(nt), dim3(NW * kWave), 0, stream, dp.seqs, dp.tiles,
                       dp.tags, (const T*)q, q_hs, (const T*)k, k_hs, n_rep, scale_log2, dp.bias,
                       dp.colpart);
    APACK_CHECK(launch_status("k_colsum") == APACK_OK, APACK_E_HIP, "%s", apack_last_error());
  }
  return APACK_OK;
}

template <class T, int D>
apack_status launch_scores_d(const PrunePlan& pl, const DevPtrs& dp, const void* q, int64_t q_hs,
                             const void* k, int64_t k_hs, int n_rep, hipStream_t stream) {
  switch (pl.waves) {
    case 1: return launch_scores_t<T, D, 1>(pl, dp, q, q_hs, k, k_hs, n_rep, stream);
    case 2: return launch_scores_t<T, D, 2>(pl, dp, q, q_hs, k, k_hs, n_rep, stream);
    case 4: return launch_scores_t<T, D, 4>(pl, dp, q, q_hs, k, k_hs, n_rep, stream);
    default: return launch_scores_t<T, D, 8>(pl, dp, q, q_hs, k, k_hs, n_rep, stream);
  }
}

}  // namespace

apack_status launch_prune(const PrunePlan& pl, const DevPtrs& dp, apack_dtype dt, int d, int hq, int hkv,
                          const void* q, int64_t q_hs, const void* k, int64_t k_hs, float* scores,
                          int32_t* kept, hipStream_t stream) {
  const int n_rep = hq / hkv;
  apack_status st;
  if (dt == APACK_BF16)
    st = d == 64 ? launch_scores_d<bf16_t, 64>(pl, dp, q, q_hs, k, k_hs, n_rep, stream)
                 : launch_scores_d<bf16_t, 128>(pl, dp, q, q_hs, k, k_hs, n_rep, stream);
  else
    st = d == 64 ? launch_scores_d<float, 64>(pl, dp, q, q_hs, k, k_hs, n_rep, stream)
                 : launch_scores_d<float, 128>(pl, dp, q, q_hs, k, k_hs, n_rep, stream);
  if (st != APACK_OK) return st;
  const int n_seq = (int)pl.seqs.size();
  if (pl.total_tok > 0) {
    hipLaunchKernelGGL(k_finalize, dim3((unsigned)((pl.total_tok + 255) / 256)), dim3(256), 0, stream,
                       dp.seqs, n_seq, pl.total_tok, dp.tags, dp.colpart, hq, hkv, scores);
    if ((st = launch_status("k_finalize")) != APACK_OK) return st;
  }
  if (pl.any_select) {
    hipLaunchKernelGGL(k_select, dim3(2 * n_seq), dim3(kSelThreads), 0, stream, dp.seqs, dp.tags, scores);
    if ((st = launch_status("k_select")) != APACK_OK) return st;
  }
  if (pl.total_tok > 0) {
    hipLaunchKernelGGL(k_scan, dim3(n_seq), dim3(kScanThreads), 0, stream, dp.seqs, dp.tags, scores, kept);
    if ((st = launch_status("k_scan")) != APACK_OK) return st;
  }
  return APACK_OK;
}

}  // namespace apack
