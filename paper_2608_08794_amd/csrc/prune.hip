// In-LLM query-conditioned prune (Section 3.2, Eq. 5 and Eq. 6) on gfx950.
//
// Per sequence and prune layer:
//   I_j = 1/(Hq*T) * sum_{h,t} softmax_{j in S}( q[h,t] . k[h/(Hq/Hkv), j] / sqrt(D) )
// followed by a per-modality top-k with the lower row winning ties, and the
// ascending list of kept rows.
//
// Kernels (all on the caller's stream, no host synchronisation):
//   k_rowstats   pass 1: per query row, (reference, sum exp2) over a chunk
//                of keys: the online maximum until each lane has seen a
//                candidate key, then a fixed reference (see row_update_ref);
//                logits from MFMA with Q fragments resident in VGPRs and K
//                tiles staged through LDS; one (max, sum) partial per row
//                and chunk.
//   k_colsum     pass 2: each workgroup first combines its rows' chunk
//                partials (fixed order) into b_r = max_r + log2(Z_r), then
//                recomputes the logits with the roles of the MFMA operands
//                swapped so the per-key sum over query rows is lane-local,
//                then a fixed-order cross-wave sum through LDS.  The last
//                workgroup of each key chunk sums the per-group partials
//                into I_j and counts its first radix digit.
// The remaining radix digits, the per-modality top-k and the ordered kept
// list are formed by the kernels of select.hip.
#include <cfloat>
#include <cmath>
#include <type_traits>
#include <vector>

#include "common.hpp"
#include "prune_plan.hpp"
#include "radix.hpp"

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

// Key tiles live in LDS as unpadded rows whose 16-byte chunks are permuted
// by an XOR with the row index (chunk c of row r sits at c ^ (r & kSwz)), so
// the 32 rows one fragment read touches fall into distinct bank groups.
template <class T, int D>
struct TileGeom {
  static constexpr int kRowBytes = D * (int)sizeof(T);
  static constexpr int kChunks = kRowBytes / 16;     // 16-byte chunks per row
  static constexpr int kSwz = (kChunks < 16 ? kChunks : 16) - 1;
  static constexpr int kTileBytes = kKeyTile * kRowBytes;
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

typedef __attribute__((address_space(3))) void* lds_ptr_t;
typedef __attribute__((address_space(1))) void* glb_ptr_t;

// Global -> LDS copy of one key tile (kKeyTile rows of D elements) with
// 16-byte direct-to-LDS loads: wave-level load j fills LDS bytes
// [1024 j, 1024 (j+1)), lane t the 16 bytes at 1024 j + 16 t.  Rows past
// n_rows repeat row n_rows - 1 (valid memory; their results are masked or
// never written).  Completion is awaited with vmcnt before the barrier.
template <class T, int D, int NW>
struct KTileLoad {
  using G = TileGeom<T, D>;
  static constexpr int kLoads = G::kTileBytes / 1024;
  static constexpr int kPer = (kLoads + NW - 1) / NW;
  static_assert(G::kTileBytes % 1024 == 0, "tile must be a whole number of 1 KiB loads");
  // wave must be uniform (readfirstlane), so that the LDS addresses and the
  // tile's base are scalar and each load costs a clamp and a 32-bit offset.
  __device__ __forceinline__ static void issue(char* lds, const T* kbase, int64_t row0, int64_t n_rows, int wave,
                                               int lane) {
    const char* base = reinterpret_cast<const char*>(kbase + row0 * D);
    // Last row of the tile that exists (rows past it repeat it).
    const int64_t left = n_rows - 1 - row0;
    const int last = left < kKeyTile - 1 ? (int)left : kKeyTile - 1;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int j = wave + i * NW;
      if (j < kLoads) {
        const int byte = j * 1024 + lane * 16;
        const int r = byte / G::kRowBytes;
        const int c = ((byte % G::kRowBytes) >> 4) ^ (r & G::kSwz);
        const uint32_t off = (uint32_t)min(r, last) * G::kRowBytes + c * 16;
        __builtin_amdgcn_global_load_lds((glb_ptr_t)(base + off), (lds_ptr_t)(lds + j * 1024), 16, 0, 0);
      }
    }
  }
};

// Waits until the tile consumed next has landed while `ahead` later tiles
// (at most two) may still be in flight.  Each tile is kPer direct-to-LDS
// loads per wave, and loads complete in issue order, so at most
// ahead * kPer outstanding operations means the older tile is done (a
// younger store only makes the wait longer).
template <class T, int D, int NW>
__device__ __forceinline__ void wait_tile_loads(int ahead) {
  // The fewest loads any wave issues per tile (a wave that issues more
  // waits a little longer than it has to).
  constexpr int kPer = KTileLoad<T, D, NW>::kLoads / NW;
  if (ahead >= 2)
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * kPer) : "memory");
  else if (ahead == 1)
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(kPer) : "memory");
  else
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// LDS stages of the key tiles: four (three tiles in flight) where a few
// query rows leave each tile little work, so that the loads of one
// workgroup keep HBM busy; two otherwise.
// (Three stages for the seven- and eight-wave workgroups, whose tiles carry
// enough arithmetic to hide a load, measured slightly slower.)
template <class T, int D, int NW>
constexpr int key_stages() {
  return (NW == 4 && TileGeom<T, D>::kTileBytes <= 32768) ? 4 : 2;
}

template <class T, int D>
__device__ __forceinline__ typename Mma<T>::frag lds_frag(const char* lds, int key, int ks, int lane) {
  using M = Mma<T>;
  using G = TileGeom<T, D>;
  const int byte = (ks * M::kstep + (lane >> 5) * M::lane_k) * (int)sizeof(T);
  const char* p = lds + key * G::kRowBytes + ((((byte >> 4) ^ (key & G::kSwz)) << 4) | (byte & 15));
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

// v + (the value of the lane 32 away), added lower half first in every lane,
// through v_permlane32_swap: no LDS round trip, so no LDS wait that would
// also wait for the K-fragment reads in flight.
__device__ __forceinline__ float add_halves(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// ---------------------------------------------------------------------------
// Software pipeline of both passes.  Each wave issues the MFMAs of key
// block b while its VALU works on the logits of block b-1, so the matrix
// core and the vector ALU run together; the instruction groups below fix
// that interleave for the bf16 MFMA (the fp32 MFMA path keeps the
// compiler's order).
// ---------------------------------------------------------------------------
// Scheduling-group masks: VALU (which on gfx950 excludes the transcendental
// unit's instructions), MFMA, and TRANS (v_exp_f32 and the like).
enum : int { kSchedVALU = 0x002, kSchedMFMA = 0x008, kSchedTRANS = 0x400 };

// VALU and transcendental instructions placed after each MFMA of a block
// (0 VALU: no placement).  The exponentials must be placed too, or they
// pile up behind the first MFMAs and leave the last ones bare.
#ifndef APACK_RS_VALU_PER_MFMA
#define APACK_RS_VALU_PER_MFMA 8
#endif
#ifndef APACK_CS_VALU_PER_MFMA
#define APACK_CS_VALU_PER_MFMA 7
#endif
#ifndef APACK_RS_TRANS_PER_MFMA
#define APACK_RS_TRANS_PER_MFMA 2
#endif
#ifndef APACK_CS_TRANS_PER_MFMA
#define APACK_CS_TRANS_PER_MFMA 2
#endif

template <class T, int N_MFMA, int N_PER, int N_TRANS>
__device__ __forceinline__ void interleave_hint() {
  if constexpr (sizeof(T) == 2 && N_PER > 0) {
#pragma unroll
    for (int i = 0; i < N_MFMA; ++i) {
      __builtin_amdgcn_sched_group_barrier(kSchedMFMA, 1, 0);
      __builtin_amdgcn_sched_group_barrier(kSchedVALU, N_PER, 0);
      if constexpr (N_TRANS > 0) __builtin_amdgcn_sched_group_barrier(kSchedTRANS, N_TRANS, 0);
    }
  }
}

// The next block's K fragments are prefetched into registers for the bf16
// MFMA (32 VGPRs per block); the fp32 fragments of a block are too large.
template <class T>
constexpr bool kPrefetchFrags = sizeof(T) == 2;

__device__ __forceinline__ f32x16 neg_inf16() {
  f32x16 c;
#pragma unroll
  for (int e = 0; e < 16; ++e) c[e] = -INFINITY;
  return c;
}

// Accumulator start of one key block in C = K Q^T: 0 for candidate keys and
// -inf for the rest, so non-candidate logits leave the MFMA as -inf.
__device__ __forceinline__ f32x16 mask_init(const float* lm, int kb, int lane) {
  f32x16 c;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float4 v = *reinterpret_cast<const float4*>(lm + kb * 32 + 8 * i + 4 * (lane >> 5));
    c[4 * i + 0] = v.x;
    c[4 * i + 1] = v.y;
    c[4 * i + 2] = v.z;
    c[4 * i + 3] = v.w;
  }
  return c;
}

// Online (max, sum exp2) update of one query row with 16 of its logits.
// All -inf (masked keys, or the empty first pipeline stage) leaves m and s
// unchanged.
__device__ __forceinline__ void row_update(const f32x16& x, float scale, float& m_run, float& s_run) {
  float lmax = x[0];
#pragma unroll
  for (int e = 1; e < 16; ++e) lmax = fmaxf(lmax, x[e]);
  const float m_new = fmaxf(m_run, lmax * scale);
  // Four running sums, each started from its first term (no add to zero).
  float p[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) p[e] = fast_exp2(fmaf(x[e], scale, -m_new));
#pragma unroll
  for (int e = 4; e < 16; ++e) p[e & 3] += fast_exp2(fmaf(x[e], scale, -m_new));
  s_run = fmaf(s_run, fast_exp2(m_run - m_new), (p[0] + p[1]) + (p[2] + p[3]));
  m_run = m_new;
}

// Σ exp2 of one query row's 16 logits against a fixed reference m0 (no
// per-block maximum or rescale).  m0 is the row's running maximum when the
// wave switches to this form, plus 64: a term overflows only for a logit
// more than 191 above that maximum (the caller then redoes the chunk with
// row_update) and underflows only below 2^-62 of it, far under the fp32
// resolution of the sum.
__device__ __forceinline__ void row_update_ref(const f32x16& x, float scale, float m0, float& s_run) {
  float p[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) p[e] = fast_exp2(fmaf(x[e], scale, -m0));
#pragma unroll
  for (int e = 4; e < 16; ++e) p[e & 3] += fast_exp2(fmaf(x[e], scale, -m0));
  s_run += (p[0] + p[1]) + (p[2] + p[3]);
}

// Fixed-order combination of two (max, sum exp2) partials of one row.
__device__ __forceinline__ void merge(float& m, float& s, float mo, float so) {
  const float mm = fmaxf(m, mo);
  s = s * fast_exp2(m - mm) + so * fast_exp2(mo - mm);
  m = mm;
}

// ---------------------------------------------------------------------------
// Pass 1: per query row, online max and sum of exp2 over one key chunk.
// C = K Q^T: lane (l % 32) owns a query column and 16 key rows per block.
// ---------------------------------------------------------------------------
template <class T, int D, int NW, int S>
__global__ __launch_bounds__(NW * kWave) void k_rowstats(const SeqDev* __restrict__ seqs,
                                                         const TileDev* __restrict__ tiles,
                                                         const uint8_t* __restrict__ tags,
                                                         const T* __restrict__ q, int64_t q_hs,
                                                         const T* __restrict__ k, int64_t k_hs,
                                                         int n_rep, float scale_log2,
                                                         float2* __restrict__ stats, uint32_t* __restrict__ zero,
                                                         int64_t zero_n) {
  using G = TileGeom<T, D>;
  using M = Mma<T>;
  constexpr int NKB = kKeyTile / 32;
  __shared__ __attribute__((aligned(16))) char lds[S][G::kTileBytes];
  // Accumulator start (0 or -inf) of every key of the chunk, built once
  // before the loop so that no tile waits on a load of its tags.
  __shared__ __attribute__((aligned(16))) float lmask[kMaxChunk];

  const TileDev tl = tiles[blockIdx.x];
  const SeqDev sq = seqs[tl.seq];
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int rows_g = n_rep * sq.q_len;
  const int rg_end = min(rows_g, (tl.rg + 1) * sq.rows_per_rg);
  const int row0 = tl.rg * sq.rows_per_rg + wave * kRowsPerWave;
  const bool active = row0 < rg_end;

  const int64_t key_begin = (int64_t)tl.chunk * sq.chunk;
  int64_t key_end = key_begin + sq.chunk;
  if (key_end > sq.n_tokens) key_end = sq.n_tokens;
  const int n_tiles = (int)((key_end - key_begin + kKeyTile - 1) / kKeyTile);
  const T* kbase = k + (int64_t)tl.g * k_hs + sq.tok_off * D;
  // The first key tiles are requested before anything else, so their loads
  // run under the clearing, the query loads and the mask build.
  for (int p = 0; p < S - 1 && p < n_tiles; ++p)
    KTileLoad<T, D, NW>::issue(lds[p], kbase, key_begin + (int64_t)p * kKeyTile, key_end, wave, lane);

  // This workgroup's share of clearing the radix histograms used by the
  // score finalisation at the end of the pass-2 kernel.
  {
    const int64_t per = (zero_n + gridDim.x - 1) / gridDim.x;
    const int64_t z0 = (int64_t)blockIdx.x * per, z1 = min(zero_n, z0 + per);
    for (int64_t i = z0 + tid; i < z1; i += NW * kWave) zero[i] = 0;
  }

  QFrags<T, D> qfr;
  auto& qf = qfr.v;
  if (active) load_q<T, D>(qfr, q, q_hs, sq, tl.g, n_rep, row0, lane);
  const uint8_t* tg = tags + sq.tag_off;

  // Tags are read in batches of 8 per thread, all in flight together (the
  // index is clamped to a valid row; rows past the chunk get -inf).
  {
    constexpr int kB = 8;
    const int n_mask = n_tiles * kKeyTile;
    for (int b0 = 0; b0 < n_mask; b0 += kB * NW * kWave) {
      uint8_t t[kB];
#pragma unroll
      for (int j = 0; j < kB; ++j) {
        const int64_t r = key_begin + b0 + tid + j * NW * kWave;
        t[j] = tg[r < key_end ? r : key_end - 1];
      }
#pragma unroll
      for (int j = 0; j < kB; ++j) {
        const int i = b0 + tid + j * NW * kWave;
        if (i < n_mask) lmask[i] = (key_begin + i < key_end && t[j] != 0) ? 0.0f : -INFINITY;
      }
    }
  }
  // One pass over the chunk's key tiles: with exact = false each lane sums
  // against its fixed reference (row_update_ref), with exact = true it keeps
  // the online maximum (row_update).  The first is taken; the second redoes
  // the chunk only if some lane's sum overflowed.
  float m_run[kRB], s_run[kRB];
  auto run_chunk = [&](auto exact_tag) {
    constexpr bool kExactOnly = decltype(exact_tag)::value;
    f32x16 pend[kRB];  // logits of the block whose VALU work is still due
#pragma unroll
    for (int rb = 0; rb < kRB; ++rb) {
      m_run[rb] = -FLT_MAX;
      s_run[rb] = 0.f;
      pend[rb] = neg_inf16();
    }
    // A wave sums with the online maximum until every lane has seen a
    // candidate key (checked at each tile start), then against a fixed
    // reference per lane: m_run + 64, with the sum rescaled once.  (The fp32
    // inputs keep the online form: their larger fragments leave no registers
    // for a second loop body.)
    constexpr bool kUseRef = sizeof(T) == 2;
    bool ref = false;
    auto tile_body = [&](auto exact_body_tag, const char* tile, const float* lm) {
      constexpr bool kExact = decltype(exact_body_tag)::value;
      // K fragments and mask of block kb+1 are read from LDS while block kb
      // computes.
      constexpr int NB = kPrefetchFrags<T> ? 2 : 1;
      KFrags<T, D> kf[NB];
      f32x16 init[NB];
      kf[0].load(tile, 0, lane);
      init[0] = mask_init(lm, 0, lane);
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) {
        const int c = kb % NB;
        if (NB == 1 && kb > 0) {
          kf[0].load(tile, kb, lane);
          init[0] = mask_init(lm, kb, lane);
        }
        if (NB == 2 && kb + 1 < NKB) {
          kf[(kb + 1) % NB].load(tile, kb + 1, lane);
          init[(kb + 1) % NB] = mask_init(lm, kb + 1, lane);
        }
        f32x16 cur[kRB];
#pragma unroll
        for (int rb = 0; rb < kRB; ++rb) cur[rb] = init[c];
#pragma unroll
        for (int ks = 0; ks < G::kSteps; ++ks)
#pragma unroll
          for (int rb = 0; rb < kRB; ++rb) cur[rb] = M::mma(kf[c].v[ks], qf[rb][ks], cur[rb]);
        // cur[rb][e]: query column (lane % 32) of block rb, key row
        // kb*32 + 8*(e/4) + 4*(lane/32) + e%4.
#pragma unroll
        for (int rb = 0; rb < kRB; ++rb) {
          if constexpr (kExact)
            row_update(pend[rb], scale_log2, m_run[rb], s_run[rb]);
          else
            row_update_ref(pend[rb], scale_log2, m_run[rb], s_run[rb]);
        }
        // The first block's fragments are read at the tile start; the
        // grouping hint there made the compiler issue one row block's MFMA
        // chain back to back, so that block is left to the default schedule
        // (which alternates the two chains with the VALU work).
        if (kb > 0) interleave_hint<T, kRB * G::kSteps, APACK_RS_VALU_PER_MFMA, APACK_RS_TRANS_PER_MFMA>();
#pragma unroll
        for (int rb = 0; rb < kRB; ++rb) pend[rb] = cur[rb];
        __builtin_amdgcn_sched_barrier(0);  // keep later blocks' LDS reads out of this one
      }
    };
    for (int it = 0; it < n_tiles; ++it) {
      const int buf = it % S;
      const int64_t t0 = key_begin + (int64_t)it * kKeyTile;
      const float* lm = lmask + it * kKeyTile;
      wait_tile_loads<T, D, NW>(min(S - 2, n_tiles - 1 - it));
      __syncthreads();
      if (it + S - 1 < n_tiles)
        KTileLoad<T, D, NW>::issue(lds[(it + S - 1) % S], kbase, t0 + (int64_t)(S - 1) * kKeyTile, key_end, wave,
                                   lane);
      if (active) {
        if (kUseRef && !kExactOnly && !ref) {
          bool unset = false;
#pragma unroll
          for (int rb = 0; rb < kRB; ++rb) unset |= m_run[rb] == -FLT_MAX;
          if (__ballot(unset) == 0) {
            ref = true;
#pragma unroll
            for (int rb = 0; rb < kRB; ++rb) {
              m_run[rb] += 64.f;
              s_run[rb] *= 0x1p-64f;
            }
          }
        }
        if (ref)
          tile_body(std::false_type{}, lds[buf], lm);
        else
          tile_body(std::true_type{}, lds[buf], lm);
      }
    }
    if (active) {
#pragma unroll
      for (int rb = 0; rb < kRB; ++rb) {
        if (ref)
          row_update_ref(pend[rb], scale_log2, m_run[rb], s_run[rb]);
        else
          row_update(pend[rb], scale_log2, m_run[rb], s_run[rb]);
      }
    }
  };
  run_chunk(std::false_type{});
  bool overflow = false;
  if (active) {
#pragma unroll
    for (int rb = 0; rb < kRB; ++rb) overflow |= !(s_run[rb] < INFINITY);
  }
  if (sizeof(T) == 2 && __syncthreads_or(overflow)) {
    // A logit far above its lane's reference: the whole workgroup streams the
    // chunk again with the online maximum (the tile buffers are free).
    for (int p = 0; p < S - 1 && p < n_tiles; ++p)
      KTileLoad<T, D, NW>::issue(lds[p], kbase, key_begin + (int64_t)p * kKeyTile, key_end, wave, lane);
    run_chunk(std::true_type{});
  }
  // The chunk's (max, sum) of each row, combined over the two lane halves;
  // pass 2 merges the chunks of its rows.
  if (active) {
#pragma unroll
    for (int rb = 0; rb < kRB; ++rb) {
      const float mo = __shfl_xor(m_run[rb], 32);
      const float so = __shfl_xor(s_run[rb], 32);
      const float mm = fmaxf(m_run[rb], mo);
      const float ss = s_run[rb] * fast_exp2(m_run[rb] - mm) + so * fast_exp2(mo - mm);
      const int rho = row0 + rb * 32 + lane;
      if (lane < 32 && rho < rg_end)
        stats[sq.stats_off + ((int64_t)tl.g * sq.n_chunks + tl.chunk) * sq.rows_pad + rho] = make_float2(mm, ss);
    }
  }
}

// ---------------------------------------------------------------------------
// Pass 2: per key, sum over this group's query rows of exp2(x - b_r).
// C = Q K^T: lane (l % 32) owns a key column and 16 query rows per block.
// Per-wave column sums of a tile go to one of three LDS slots; the sum over
// waves of tile t (fixed wave order) is formed at the start of tile t+2,
// when every wave has finished it, and after the loop for the last two.
// ---------------------------------------------------------------------------
template <int NKB, int NW>
__device__ __forceinline__ void col_flush(float (&red)[3][NW][NKB * 32], int slot, int n_active, int64_t tile0,
                                          int64_t key_end, float* out, int tid) {
  for (int i = tid; i < NKB * 32; i += NW * kWave) {
    // All NW reads are issued before the fixed-order sum.
    float r[NW];
#pragma unroll
    for (int w = 0; w < NW; ++w) r[w] = w < n_active ? red[slot][w][i] : 0.f;
    float v = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w)
      if (w < n_active) v += r[w];
    if (tile0 + i < key_end) st_agent(&out[tile0 + i], v);
  }
}

template <class T, int D, int NW, int S>
__global__ __launch_bounds__(NW * kWave) void k_colsum(SeqDev* __restrict__ seqs,
                                                       const TileDev* __restrict__ tiles,
                                                       const uint8_t* __restrict__ tags,
                                                       const T* __restrict__ q, int64_t q_hs,
                                                       const T* __restrict__ k, int64_t k_hs,
                                                       int n_rep, int hkv, float scale_log2,
                                                       const float2* __restrict__ stats,
                                                       float* __restrict__ colpart, float* __restrict__ scores,
                                                       uint32_t* __restrict__ hist, uint32_t* __restrict__ ctr) {
  using G = TileGeom<T, D>;
  using M = Mma<T>;
  constexpr int NKB = kKeyTile / 32;
  __shared__ __attribute__((aligned(16))) char lds[S][G::kTileBytes];
  __shared__ float red[3][NW][kKeyTile];

  const TileDev tl = tiles[blockIdx.x];
  const SeqDev sq = seqs[tl.seq];
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int rows_g = n_rep * sq.q_len;
  const int rg_end = min(rows_g, (tl.rg + 1) * sq.rows_per_rg);
  const int row0 = tl.rg * sq.rows_per_rg + wave * kRowsPerWave;
  const bool active = row0 < rg_end;
  const int n_active = (rg_end - tl.rg * sq.rows_per_rg + kRowsPerWave - 1) / kRowsPerWave;

  const int64_t key_begin = (int64_t)tl.chunk * sq.chunk;
  int64_t key_end = key_begin + sq.chunk;
  if (key_end > sq.n_tokens) key_end = sq.n_tokens;
  const int n_tiles = (int)((key_end - key_begin + kKeyTile - 1) / kKeyTile);
  const T* kbase = k + (int64_t)tl.g * k_hs + sq.tok_off * D;
  // The first key tiles are requested before the query loads and the row-partial merge.
  for (int p = 0; p < S - 1 && p < n_tiles; ++p)
    KTileLoad<T, D, NW>::issue(lds[p], kbase, key_begin + (int64_t)p * kKeyTile, key_end, wave, lane);

  QFrags<T, D> qfr;
  auto& qf = qfr.v;
  if (active) load_q<T, D>(qfr, q, q_hs, sq, tl.g, n_rep, row0, lane);
  // b_r = M_r + log2(Z_r) of the row group's rows, combined from pass 1's
  // chunk partials in chunk order (padding rows get +inf, so they add
  // exp2(-inf) = 0).  With fewer rows than threads, ng threads share a row,
  // each merging a contiguous run of chunks, and the runs are combined in
  // order.  The column-sum slots hold the values until the loop starts.
  float b[kRB][16];
  {
    const int R = sq.rows_per_rg, nthr = NW * kWave, r_lo = tl.rg * sq.rows_per_rg;
    const int ng = R <= nthr / 4 ? 4 : R <= nthr / 2 ? 2 : 1;
    float* lb = &red[0][0][0];
    float2* part = reinterpret_cast<float2*>(lb + R);
    const float2* p0 = stats + sq.stats_off + (int64_t)tl.g * sq.n_chunks * sq.rows_pad;
    const int cpg = (sq.n_chunks + ng - 1) / ng;
    if (tid < ng * R) {
      const int grp = tid / R, r = tid - grp * R, rho = r_lo + r;
      float m = -FLT_MAX, s = 0.f;
      if (rho < rows_g) {
        const int c_lo = grp * cpg, c_hi = min(sq.n_chunks, (grp + 1) * cpg);
        constexpr int CB = 16;
        for (int c0 = c_lo; c0 < c_hi; c0 += CB) {
          float2 v[CB];
#pragma unroll
          for (int i = 0; i < CB; ++i) v[i] = p0[(int64_t)min(c0 + i, c_hi - 1) * sq.rows_pad + rho];
#pragma unroll
          for (int i = 0; i < CB; ++i)
            if (c0 + i < c_hi) merge(m, s, v[i].x, v[i].y);
        }
      }
      part[grp * R + r] = make_float2(m, s);
    }
    __syncthreads();
    for (int r = tid; r < R; r += nthr) {
      float mm = part[r].x, ss = part[r].y;
      for (int g2 = 1; g2 < ng; ++g2) merge(mm, ss, part[g2 * R + r].x, part[g2 * R + r].y);
      lb[r] = (ss > 0.f) ? mm + log2f(ss) : INFINITY;
    }
    __syncthreads();
    if (active) {
      const float* bb = lb + (row0 - r_lo) + 4 * (lane >> 5);
#pragma unroll
      for (int rb = 0; rb < kRB; ++rb)
#pragma unroll
        for (int e = 0; e < 16; ++e) b[rb][e] = bb[rb * 32 + 8 * (e >> 2) + (e & 3)];
    }
  }

  float* out = colpart + sq.colpart_off + (int64_t)(tl.g * sq.n_rg + tl.rg) * sq.n_tokens;

  // The pipeline unit is one (key block, row block) pair: its MFMAs run
  // while the VALU sums the exponentials of the previous unit into cs, the
  // running column sum of that unit's key block.
  f32x16 pend = neg_inf16();
  float cs = 0.f;
  auto add_pend = [&](int rb) {
    float p[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) p[e] = fast_exp2(fmaf(pend[e], scale_log2, -b[rb][e]));
#pragma unroll
    for (int e = 4; e < 16; ++e) p[e & 3] += fast_exp2(fmaf(pend[e], scale_log2, -b[rb][e]));
    // The first row block of a key block starts its column sum.
    const float t = (p[0] + p[1]) + (p[2] + p[3]);
    cs = rb == 0 ? t : cs + t;
  };
  // Column sums of a finished key block into its tile's slot (lanes < 32).
  auto flush_block = [&](int slot, int blk) {
    const float c = add_halves(cs);
    if (lane < 32) red[slot][wave][blk * 32 + lane] = c;
    cs = 0.f;
  };

  for (int it = 0; it < n_tiles; ++it) {
    const int buf = it % S;
    const int64_t t0 = key_begin + (int64_t)it * kKeyTile;
    wait_tile_loads<T, D, NW>(min(S - 2, n_tiles - 1 - it));
    __syncthreads();
    if (it >= 2) col_flush<NKB, NW>(red, (it - 2) % 3, n_active, t0 - 2 * kKeyTile, key_end, out, tid);
    if (it + S - 1 < n_tiles)
      KTileLoad<T, D, NW>::issue(lds[(it + S - 1) % S], kbase, t0 + (int64_t)(S - 1) * kKeyTile, key_end, wave,
                                 lane);
    if (active) {
      const int slot = it % 3, prev_slot = (it + 2) % 3;
      // K fragments of block kb+1 are read from LDS while block kb computes.
      constexpr int NB = kPrefetchFrags<T> ? 2 : 1;
      KFrags<T, D> kf[NB];
      kf[0].load(lds[buf], 0, lane);
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) {
        const int c = kb % NB;
        if (NB == 1 && kb > 0) kf[0].load(lds[buf], kb, lane);
        if (NB == 2 && kb + 1 < NKB) kf[(kb + 1) % NB].load(lds[buf], kb + 1, lane);
#pragma unroll
        for (int rb = 0; rb < kRB; ++rb) {
          f32x16 cur = f32x16{};
#pragma unroll
          for (int ks = 0; ks < G::kSteps; ++ks) cur = M::mma(qf[rb][ks], kf[c].v[ks], cur);
          // cur[e]: key column kb*32 + (lane % 32), query row
          // rb*32 + 8*(e/4) + 4*(lane/32) + e%4 of this wave.
          // The pending unit is the previous one; for the first unit of the
          // first tile it is all -inf and writes zeros to a slot no tile has
          // used yet.
          add_pend(rb == 0 ? kRB - 1 : rb - 1);
          if (rb == 0) flush_block(kb == 0 ? prev_slot : slot, kb == 0 ? NKB - 1 : kb - 1);
          interleave_hint<T, G::kSteps, APACK_CS_VALU_PER_MFMA, APACK_CS_TRANS_PER_MFMA>();
          pend = cur;
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
  }
  if (active && n_tiles > 0) {
    add_pend(kRB - 1);
    flush_block((n_tiles - 1) % 3, NKB - 1);
  }
  __syncthreads();
  const int64_t last0 = key_begin + (int64_t)(n_tiles - 1) * kKeyTile;
  if (n_tiles >= 2) col_flush<NKB, NW>(red, (n_tiles - 2) % 3, n_active, last0 - kKeyTile, key_end, out, tid);
  if (n_tiles >= 1) col_flush<NKB, NW>(red, (n_tiles - 1) % 3, n_active, last0, key_end, out, tid);

  // The last workgroup of this key chunk (over groups and row groups) forms
  // I_j = (sum of the per-group partials, fixed order) / (Hq * T), 0 for
  // non-candidates, and counts the first radix digit; the last chunk of the
  // sequence picks the digit's bin.  The descriptor is read again here
  // rather than kept live across the main loop.
  SeqDev* sr = &seqs[tl.seq];
  const int planes = hkv * sr->n_rg;
  if (!arrive_last<NW * kWave>(ctr + sr->ctr_off + tl.chunk, (uint32_t)planes)) return;
  const bool sel = sr->select[0] || sr->select[1];
  uint32_t* lh = reinterpret_cast<uint32_t*>(&lds[0][0]);  // 2 x 2048 bins; the key tiles are done
  if (sel) {
    for (int b = tid; b < 2 * kRadixBins; b += NW * kWave) lh[b] = 0;
    __syncthreads();
  }
  const uint8_t* tg = tags + sr->tag_off;
  const float denom = (float)(n_rep * hkv * sr->q_len);
  const float* cp = colpart + sr->colpart_off;
  const int64_t n_tok = sr->n_tokens;
  float* sc = scores + sr->tok_off;
  const int32_t sel_m[2] = {sr->select[0], sr->select[1]};
  // KB keys per thread and PB planes at a time are loaded together, then
  // summed in plane order.
  constexpr int KB = 4, PB = 8;
  for (int64_t j0 = key_begin + tid; j0 < key_end; j0 += (int64_t)KB * NW * kWave) {
    uint8_t mt[KB];
    float acc[KB];
#pragma unroll
    for (int b = 0; b < KB; ++b) {
      const int64_t j = j0 + (int64_t)b * NW * kWave;
      mt[b] = j < key_end ? tg[j] : (uint8_t)0;
      acc[b] = 0.f;
    }
    for (int p0 = 0; p0 < planes; p0 += PB) {
      float v[KB][PB];
#pragma unroll
      for (int b = 0; b < KB; ++b)
#pragma unroll
        for (int i = 0; i < PB; ++i) {
          const int64_t j = j0 + (int64_t)b * NW * kWave;
          v[b][i] = (j < key_end && mt[b] != 0 && p0 + i < planes) ? ld_agent(cp + (int64_t)(p0 + i) * n_tok + j)
                                                                   : 0.f;
        }
#pragma unroll
      for (int b = 0; b < KB; ++b)
#pragma unroll
        for (int i = 0; i < PB; ++i)
          if (p0 + i < planes) acc[b] += v[b][i];
    }
#pragma unroll
    for (int b = 0; b < KB; ++b) {
      const int64_t j = j0 + (int64_t)b * NW * kWave;
      if (j >= key_end) continue;
      const uint8_t m = mt[b];
      float v = 0.f;
      if (m != 0) {
        v = acc[b] / denom;
        if ((m == 1 || m == 2) && sel_m[m - 1]) atomicAdd(&lh[(m - 1) * kRadixBins + (clamp_bits(v) >> 20)], 1u);
      }
      sc[j] = v;
    }
  }
  if (!sel) return;
  __syncthreads();
  uint32_t* gh = hist + (int64_t)tl.seq * 2 * kRadixBins;
  merge_hist<NW * kWave>(lh, gh);
  if (arrive_last<NW * kWave>(ctr + sr->ctr_off + sr->n_chunks, (uint32_t)sr->n_chunks))
    pick_bins<NW * kWave>(sr, gh, 0);
}

// ---------------------------------------------------------------------------
// Host launch sequence.
// ---------------------------------------------------------------------------
template <class T, int D, int NW, int S = key_stages<T, D, NW>()>
apack_status launch_scores_t(const PrunePlan& pl, const DevPtrs& dp, const void* q, int64_t q_hs,
                             const void* k, int64_t k_hs, int n_rep, int hkv, float* scores, hipStream_t stream) {
  const float scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)D));
  const int nt = (int)pl.tiles.size();
  if (nt > 0) {
    hipLaunchKernelGGL((k_rowstats<T, D, NW, S>), dim3(nt), dim3(NW * kWave), 0, stream, dp.seqs, dp.tiles,
                       dp.tags, (const T*)q, q_hs, (const T*)k, k_hs, n_rep, scale_log2, dp.stats, dp.hist,
                       pl.any_select ? select_hist_words((int64_t)pl.seqs.size()) : (int64_t)0);
    APACK_CHECK(launch_status("k_rowstats") == APACK_OK, APACK_E_HIP, "%s", apack_last_error());
    hipLaunchKernelGGL((k_colsum<T, D, NW, S>), dim3(nt), dim3(NW * kWave), 0, stream, dp.seqs, dp.tiles, dp.tags,
                       (const T*)q, q_hs, (const T*)k, k_hs, n_rep, hkv, scale_log2, dp.stats, dp.colpart, scores,
                       dp.hist, dp.ctr);
    APACK_CHECK(launch_status("k_colsum") == APACK_OK, APACK_E_HIP, "%s", apack_last_error());
  }
  return APACK_OK;
}

template <class T, int D>
apack_status launch_scores_d(const PrunePlan& pl, const DevPtrs& dp, const void* q, int64_t q_hs,
                             const void* k, int64_t k_hs, int n_rep, int hkv, float* scores, hipStream_t stream) {
  // Up to four waves of query rows run as four-wave workgroups: with one or
  // two row waves the others only share the tile loads and the chunk's
  // closing sums, and the tiles stream through four LDS stages.
  switch (pl.waves) {
    case 1:
    case 2:
    case 4: return launch_scores_t<T, D, 4>(pl, dp, q, q_hs, k, k_hs, n_rep, hkv, scores, stream);
    case 7: return launch_scores_t<T, D, 7>(pl, dp, q, q_hs, k, k_hs, n_rep, hkv, scores, stream);
    default: return launch_scores_t<T, D, 8>(pl, dp, q, q_hs, k, k_hs, n_rep, hkv, scores, stream);
  }
}

}  // namespace

apack_status launch_prune(const PrunePlan& pl, const DevPtrs& dp, apack_dtype dt, int d, int hq, int hkv,
                          const void* q, int64_t q_hs, const void* k, int64_t k_hs, float* scores,
                          int32_t* kept, hipStream_t stream) {
  const int n_rep = hq / hkv;
  apack_status st;
  if (dt == APACK_BF16)
    st = d == 64 ? launch_scores_d<bf16_t, 64>(pl, dp, q, q_hs, k, k_hs, n_rep, hkv, scores, stream)
                 : launch_scores_d<bf16_t, 128>(pl, dp, q, q_hs, k, k_hs, n_rep, hkv, scores, stream);
  else
    st = d == 64 ? launch_scores_d<float, 64>(pl, dp, q, q_hs, k, k_hs, n_rep, hkv, scores, stream)
                 : launch_scores_d<float, 128>(pl, dp, q, q_hs, k, k_hs, n_rep, hkv, scores, stream);
  if (st != APACK_OK) return st;
  if (pl.total_tok == 0) return APACK_OK;
  return launch_select(pl, dp, scores, kept, stream);
}

}  // namespace apack
