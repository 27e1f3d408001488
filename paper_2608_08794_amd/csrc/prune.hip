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
// The per-group partials are summed into I_j, and the per-modality top-k and
// ordered kept list are formed, by the kernels of select.hip.
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

// Query fragments of the rows a wave owns (kRB blocks of 32), loaded once.
template <class T, int D>
struct QFrags {
  typename Mma<T>::frag v[kRB][TileGeom<T, D>::kSteps];
};

// Rows past the group's end read a clamped, valid row and are zeroed after
// the (unconditional) loads, so all loads of a lane are in flight together.
template <class T, int D>
__device__ __forceinline__ void load_q(QFrags<T, D>& qfr, const T* q, int64_t q_hs, const SeqDev& sq, int g,
                                       int n_rep, int row0, int lane) {
  using M = Mma<T>;
  auto& qf = qfr.v;
  const int rows = n_rep * sq.q_len;
#pragma unroll
  for (int rb = 0; rb < kRB; ++rb) {
    const int rho = row0 + rb * 32 + (lane & 31);
    const int rc = rho < rows ? rho : rows - 1;
    const int h = g * n_rep + rc / sq.q_len;
    const int t = rc % sq.q_len;
    const T* src = q + (int64_t)h * q_hs + (sq.q_off + t) * (int64_t)D + (lane >> 5) * M::lane_k;
#pragma unroll
    for (int ks = 0; ks < TileGeom<T, D>::kSteps; ++ks)
      qf[rb][ks] = *reinterpret_cast<const typename M::frag*>(src + ks * M::kstep);
    if (rho >= rows) {
#pragma unroll
      for (int ks = 0; ks < TileGeom<T, D>::kSteps; ++ks) qf[rb][ks] = M::zero();
    }
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

// K fragments of one block of 32 keys, read from LDS in one batch.
template <class T, int D>
struct KFrags {
  typename Mma<T>::frag v[TileGeom<T, D>::kSteps];
  __device__ __forceinline__ void load(const char* lds, int kb, int lane) {
#pragma unroll
    for (int ks = 0; ks < TileGeom<T, D>::kSteps; ++ks) v[ks] = lds_frag<T, D>(lds, kb * 32 + (lane & 31), ks, lane);
  }
};

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// ---------------------------------------------------------------------------
// Pass 1: per query row, online max and sum of exp2 over one key chunk.
// C = K Q^T: lane (l % 32) owns a query column and 16 key rows per block.
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
  constexpr int NKB = kKeyTile / 32;
  __shared__ __attribute__((aligned(16))) char lds[2][G::kTileBytes];
  __shared__ __attribute__((aligned(16))) float lmask[2][kKeyTile];
  __shared__ int lmasked[2];

  const TileDev tl = tiles[blockIdx.x];
  const SeqDev sq = seqs[tl.seq];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int rows_g = n_rep * sq.q_len;
  const int rg_end = min(rows_g, (tl.rg + 1) * sq.rows_per_rg);
  const int row0 = tl.rg * sq.rows_per_rg + wave * kRowsPerWave;
  const bool active = row0 < rg_end;

  QFrags<T, D> qfr;
  auto& qf = qfr.v;
  if (active) load_q<T, D>(qfr, q, q_hs, sq, tl.g, n_rep, row0, lane);

  const int64_t key_begin = (int64_t)tl.chunk * sq.chunk;
  int64_t key_end = key_begin + sq.chunk;
  if (key_end > sq.n_tokens) key_end = sq.n_tokens;
  const int n_tiles = (int)((key_end - key_begin + kKeyTile - 1) / kKeyTile);
  const T* kbase = k + (int64_t)tl.g * k_hs + sq.tok_off * D;
  const uint8_t* tg = tags + sq.tag_off;

  float m_run[kRB], s_run[kRB];
#pragma unroll
  for (int rb = 0; rb < kRB; ++rb) {
    m_run[rb] = -FLT_MAX;
    s_run[rb] = 0.f;
  }

  KStage<T, D, NW> st;
  st.load(kbase, key_begin, key_end, tid);
  for (int it = 0; it < n_tiles; ++it) {
    const int buf = it & 1;
    const int64_t t0 = key_begin + (int64_t)it * kKeyTile;
    st.store(lds[buf], tid);
    if (tid < kKeyTile) {
      const bool cand = (t0 + tid < key_end) && tg[t0 + tid] != 0;
      lmask[buf][tid] = cand ? 0.0f : -INFINITY;
      const uint64_t bal = __ballot(!cand);
      if (tid == 0) lmasked[buf] = bal != 0;
    }
    __syncthreads();
    if (it + 1 < n_tiles) st.load(kbase, t0 + kKeyTile, key_end, tid);
    if (active) {
      const bool masked = lmasked[buf] != 0;
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) {
        KFrags<T, D> kf;
        kf.load(lds[buf], kb, lane);
        f32x16 acc[kRB];
#pragma unroll
        for (int rb = 0; rb < kRB; ++rb) acc[rb] = f32x16{};
#pragma unroll
        for (int ks = 0; ks < G::kSteps; ++ks)
#pragma unroll
          for (int rb = 0; rb < kRB; ++rb) acc[rb] = M::mma(kf.v[ks], qf[rb][ks], acc[rb]);
        // acc[rb][e]: query column (lane % 32) of block rb, key row
        // kb*32 + 8*(e/4) + 4*(lane/32) + e%4.
        if (masked) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float4 mk = *reinterpret_cast<const float4*>(&lmask[buf][kb * 32 + 8 * i + 4 * (lane >> 5)]);
#pragma unroll
            for (int rb = 0; rb < kRB; ++rb) {
              acc[rb][4 * i + 0] += mk.x;
              acc[rb][4 * i + 1] += mk.y;
              acc[rb][4 * i + 2] += mk.z;
              acc[rb][4 * i + 3] += mk.w;
            }
          }
        }
#pragma unroll
        for (int rb = 0; rb < kRB; ++rb) {
          float lmax = acc[rb][0];
#pragma unroll
          for (int e = 1; e < 16; ++e) lmax = fmaxf(lmax, acc[rb][e]);
          const float m_new = fmaxf(m_run[rb], lmax * scale_log2);
          float s = 0.f;
#pragma unroll
          for (int e = 0; e < 16; ++e) s += fast_exp2(fmaf(acc[rb][e], scale_log2, -m_new));
          s_run[rb] = s_run[rb] * fast_exp2(m_run[rb] - m_new) + s;
          m_run[rb] = m_new;
        }
      }
    }
  }
  if (!active) return;
#pragma unroll
  for (int rb = 0; rb < kRB; ++rb) {
    const float mo = __shfl_xor(m_run[rb], 32);
    const float so = __shfl_xor(s_run[rb], 32);
    const float mm = fmaxf(m_run[rb], mo);
    const float ss = s_run[rb] * fast_exp2(m_run[rb] - mm) + so * fast_exp2(mo - mm);
    const int rho = row0 + rb * 32 + lane;
    if (lane < 32 && rho < rg_end)
      stats[sq.stats_off + ((int64_t)tl.g * sq.rows_pad + rho) * sq.n_chunks + tl.chunk] = make_float2(mm, ss);
  }
}

// ---------------------------------------------------------------------------
// Combine chunk partials of every (group, padded row): b = M + log2(Z);
// padding rows get +inf so they contribute exp2(-inf) = 0 in pass 2.
// One wave per row; lanes stride the chunks; fixed-order tree merge.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void merge(float& m, float& s, float mo, float so) {
  const float mm = fmaxf(m, mo);
  s = s * fast_exp2(m - mm) + so * fast_exp2(mo - mm);
  m = mm;
}

__global__ __launch_bounds__(256) void k_rowreduce(const SeqDev* __restrict__ seqs, int n_seq,
                                                   int64_t total_rows, int n_rep,
                                                   const float2* __restrict__ stats, float* __restrict__ bias) {
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= total_rows) return;
  int lo = 0, hi = n_seq - 1;
  while (lo < hi) {  // last sequence whose bias_off <= row
    const int mid = (lo + hi + 1) >> 1;
    if (seqs[mid].bias_off <= row) lo = mid; else hi = mid - 1;
  }
  const SeqDev& sq = seqs[lo];
  const int64_t r = row - sq.bias_off;            // g * rows_pad + rho
  const int rho = (int)(r % sq.rows_pad);
  float m = -FLT_MAX, s = 0.f;
  if (rho < n_rep * sq.q_len) {
    const float2* p = stats + sq.stats_off + r * sq.n_chunks;
    for (int c = lane; c < sq.n_chunks; c += 64) merge(m, s, p[c].x, p[c].y);
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float mo = __shfl_xor(m, off), so = __shfl_xor(s, off);
    merge(m, s, mo, so);
  }
  if (lane == 0) bias[row] = (s > 0.f) ? m + log2f(s) : INFINITY;
}

// ---------------------------------------------------------------------------
// Pass 2: per key, sum over this group's query rows of exp2(x - b_r).
// C = Q K^T: lane (l % 32) owns a key column and 16 query rows per block.
// The exponentials of one (key block, row block) run while the MFMAs of
// the next pair are in flight.
// ---------------------------------------------------------------------------
template <class T, int D, int NW>
__global__ __launch_bounds__(NW * kWave) void k_colsum(const SeqDev* __restrict__ seqs,
                                                       const TileDev* __restrict__ tiles,
                                                       const T* __restrict__ q, int64_t q_hs,
                                                       const T* __restrict__ k, int64_t k_hs,
                                                       int n_rep, float scale_log2,
                                                       const float* __restrict__ bias,
                                                       float* __restrict__ colpart) {
  using G = TileGeom<T, D>;
  using M = Mma<T>;
  constexpr int NKB = kKeyTile / 32;
  __shared__ __attribute__((aligned(16))) char lds[2][G::kTileBytes];
  __shared__ float red[2][NW][kKeyTile];

  const TileDev tl = tiles[blockIdx.x];
  const SeqDev sq = seqs[tl.seq];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int rows_g = n_rep * sq.q_len;
  const int rg_end = min(rows_g, (tl.rg + 1) * sq.rows_per_rg);
  const int row0 = tl.rg * sq.rows_per_rg + wave * kRowsPerWave;
  const bool active = row0 < rg_end;
  const int n_active = (rg_end - tl.rg * sq.rows_per_rg + kRowsPerWave - 1) / kRowsPerWave;

  QFrags<T, D> qfr;
  auto& qf = qfr.v;
  float b[kRB][16];
  if (active) {
    load_q<T, D>(qfr, q, q_hs, sq, tl.g, n_rep, row0, lane);
    const float* bb = bias + sq.bias_off + (int64_t)tl.g * sq.rows_pad + row0 + 4 * (lane >> 5);
#pragma unroll
    for (int rb = 0; rb < kRB; ++rb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float4 v = *reinterpret_cast<const float4*>(bb + rb * 32 + 8 * i);
        b[rb][4 * i + 0] = v.x;
        b[rb][4 * i + 1] = v.y;
        b[rb][4 * i + 2] = v.z;
        b[rb][4 * i + 3] = v.w;
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
      float cs[NKB];
      f32x16 prev;
      int prev_kb = -1, prev_rb = 0;
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) {
        KFrags<T, D> kf;
        kf.load(lds[buf], kb, lane);
        cs[kb] = 0.f;
#pragma unroll
        for (int rb = 0; rb < kRB; ++rb) {
          f32x16 acc = f32x16{};
#pragma unroll
          for (int ks = 0; ks < G::kSteps; ++ks) acc = M::mma(qf[rb][ks], kf.v[ks], acc);
          if (prev_kb >= 0) {
            // Epilogue of the previous (key block, row block) pair.
            float s = 0.f;
#pragma unroll
            for (int e = 0; e < 16; ++e) s += fast_exp2(fmaf(prev[e], scale_log2, -b[prev_rb][e]));
            cs[prev_kb] += s;
          }
          prev = acc;
          prev_kb = kb;
          prev_rb = rb;
        }
      }
      {
        float s = 0.f;
#pragma unroll
        for (int e = 0; e < 16; ++e) s += fast_exp2(fmaf(prev[e], scale_log2, -b[kRB - 1][e]));
        cs[NKB - 1] += s;
      }
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) {
        const float c = cs[kb] + __shfl_xor(cs[kb], 32);
        if (lane < 32) red[buf][wave][kb * 32 + lane] = c;
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
                       (int)pl.seqs.size(), rows, n_rep, dp.stats, dp.bias);
    APACK_CHECK(launch_status("k_rowreduce") == APACK_OK, APACK_E_HIP, "%s", apack_last_error());
    hipLaunchKernelGGL((k_colsum<T, D, NW>), dim3(nt), dim3(NW * kWave), 0, stream, dp.seqs, dp.tiles,
                       (const T*)q, q_hs, (const T*)k, k_hs, n_rep, scale_log2, dp.bias, dp.colpart);
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
    case 7: return launch_scores_t<T, D, 7>(pl, dp, q, q_hs, k, k_hs, n_rep, stream);
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
  if (pl.total_tok == 0) return APACK_OK;
  return launch_select(pl, dp, hq, hkv, scores, kept, stream);
}

}  // namespace apack
