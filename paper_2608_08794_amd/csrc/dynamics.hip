// Pre-LLM local audio-visual dynamics scorer (Section 3.1, Eq. 1-4; the
// first loop of Algorithm 1) on gfx950.
//
//   k_pool       coarse pass: frame means v_f, audio-bin means a_f (adaptive
//                pooling onto the frame axis) and the query mean, in fp64;
//                the same read leaves per-slice row sums of squares
//   k_band       band Gram v_f.v_{f+d}, a_f.a_{f+d} (d < w), v_f.q, q.q
//   k_cka        Eq. 1 per frame from the centred w x w window Grams, the
//                clip mean and the gate of Eq. 2
//   k_norms      squared norms of every visual and audio token of the clips
//                (fp64), from k_pool's per-slice sums, and 1/|x| of the
//                visual tokens
//   k_gate_gemm  only where the gate fired: X_A . X_V^T on bf16 MFMA, scaled
//                by 1/|a_j|, max over audio tokens in-lane, merged across
//                tiles by atomicMax on order-preserving uint keys
//   k_plan       one 1024-thread workgroup per clip, arrays in LDS:
//                direct distance, Eq. 2 blend,
//                continuity smoothing and cuts, Eq. 3 segment scores, frame
//                scores, Eq. 4 segment budgets and frame budgets (capped
//                largest remainder), anchors and output offsets
//   k_gram       fp64 Gram of the tokens of every anchor frame (fp64 MFMA)
//   k_dafps      per anchor frame: cosines from the Gram and its diagonal,
//                then density-aware farthest-point sampling in one wave
//   k_dedup_sim, k_dedup_pick  one wave per token, then one workgroup per
//                non-anchor frame: keep the positions least
//                similar to the anchor
//
// Every discrete decision (gate, cuts, budgets, DA-FPS argmax, dedup ranks)
// is taken in fp64, as in the oracle.  The gate GEMM accumulates in fp32.
#include <algorithm>
#include <cfloat>
#include <cmath>
#include <type_traits>

#include "common.hpp"
#include "dynamics_plan.hpp"

namespace apack {
namespace {

typedef unsigned short bf16_t;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kBlk = 256;

// 8 consecutive elements as doubles (16- or 32-byte aligned loads).
__device__ __forceinline__ void load8(const bf16_t* p, double (&o)[8]) {
  const uint4 u = *reinterpret_cast<const uint4*>(p);
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    o[2 * i] = (double)__uint_as_float(w[i] << 16);
    o[2 * i + 1] = (double)__uint_as_float(w[i] & 0xFFFF0000u);
  }
}
__device__ __forceinline__ void load8(const float* p, double (&o)[8]) {
  const float4 a = reinterpret_cast<const float4*>(p)[0];
  const float4 b = reinterpret_cast<const float4*>(p)[1];
  o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w;
  o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
}

// Cross-lane reductions of a double over the 64 lanes of a wave, in every
// lane, without the LDS crossbar: DPP within 16-lane rows, then
// v_permlane16_swap (rows 0<->1, 2<->3) and v_permlane32_swap (halves).
// All 64 lanes must be active.
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
  const uint64_t b = (uint64_t)__double_as_longlong(v);
  const int lo = __builtin_amdgcn_update_dpp((int)(uint32_t)b, (int)(uint32_t)b, CTRL, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp((int)(uint32_t)(b >> 32), (int)(uint32_t)(b >> 32), CTRL, 0xF, 0xF, false);
  return __longlong_as_double((long long)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo));
}
// The two values of a swap pair (rows 2k and 2k+1, or the two halves), the
// lower one first, the same in both lanes of the pair.
template <bool ROWS16>
__device__ __forceinline__ void swap_pair_f64(double v, double& x, double& y) {
  const uint64_t b = (uint64_t)__double_as_longlong(v);
  const uint32_t lo = (uint32_t)b, hi = (uint32_t)(b >> 32);
  uint32_t l0, l1, h0, h1;
  if constexpr (ROWS16) {
    const auto l = __builtin_amdgcn_permlane16_swap(lo, lo, false, false);
    const auto h = __builtin_amdgcn_permlane16_swap(hi, hi, false, false);
    l0 = l[0]; l1 = l[1]; h0 = h[0]; h1 = h[1];
  } else {
    const auto l = __builtin_amdgcn_permlane32_swap(lo, lo, false, false);
    const auto h = __builtin_amdgcn_permlane32_swap(hi, hi, false, false);
    l0 = l[0]; l1 = l[1]; h0 = h[0]; h1 = h[1];
  }
  x = __longlong_as_double((long long)(((uint64_t)h0 << 32) | l0));
  y = __longlong_as_double((long long)(((uint64_t)h1 << 32) | l1));
}
// Sum: every step pairs lanes symmetrically (quad xor 1, quad xor 2,
// half-row mirror, row mirror, then the swaps), so both lanes of a pair add
// the same two values and every lane ends with the same bits.
__device__ __forceinline__ double wave_sum(double v) {
  v += dpp_f64<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp_f64<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp_f64<0x141>(v);  // row_half_mirror
  v += dpp_f64<0x140>(v);  // row_mirror
  double x, y;
  swap_pair_f64<true>(v, x, y);
  swap_pair_f64<false>(x + y, x, y);
  return x + y;
}
__device__ __forceinline__ double wave_max_f64(double v) {
  v = fmax(v, dpp_f64<0xB1>(v));
  v = fmax(v, dpp_f64<0x4E>(v));
  v = fmax(v, dpp_f64<0x141>(v));
  v = fmax(v, dpp_f64<0x140>(v));
  double x, y;
  swap_pair_f64<true>(v, x, y);
  swap_pair_f64<false>(fmax(x, y), x, y);
  return fmax(x, y);
}

// Four sums at once, each over the 64 lanes: lane j (< 4) returns the sum
// of v[j].  Lanes 2k and 2k+1 swap halves (the even lane keeps v[0] and
// v[2], the odd one v[1] and v[3]), then lanes 4k..4k+3 do the same with
// what they kept, so lane i holds a four-lane sum of v[i % 4]; rotations
// by 4 and 8 lanes and the 16- and 32-lane swaps add the lanes with the
// same i % 4.  The other lanes return partial sums.  All 64 lanes must be
// active.
__device__ __forceinline__ double wave_sum4(const double (&v)[4]) {
  const int lane = threadIdx.x & 63;
  const bool odd = lane & 1, hi2 = lane & 2;
  const double x = (odd ? v[1] : v[0]) + dpp_f64<0xB1>(odd ? v[0] : v[1]);
  const double y = (odd ? v[3] : v[2]) + dpp_f64<0xB1>(odd ? v[2] : v[3]);
  double t = (hi2 ? y : x) + dpp_f64<0x4E>(hi2 ? x : y);
  t += dpp_f64<0x124>(t);  // row_ror:4
  t += dpp_f64<0x128>(t);  // row_ror:8
  double a, b;
  swap_pair_f64<true>(t, a, b);
  swap_pair_f64<false>(a + b, a, b);
  return a + b;
}

// Block-wide reductions over NT threads (sh holds NT / 64 words); every
// thread gets the result.
template <int NT = kBlk>
__device__ double block_sum(double v, double* sh) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) sh[wave] = v;
  __syncthreads();
  double t = 0.0;
  for (int w = 0; w < NT / 64; ++w) t += sh[w];
  __syncthreads();
  return t;
}
template <int NT = kBlk>
__device__ double block_max(double v, double* sh) {
  v = wave_max_f64(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) sh[wave] = v;
  __syncthreads();
  double t = sh[0];
  for (int w = 1; w < NT / 64; ++w) t = fmax(t, sh[w]);
  __syncthreads();
  return t;
}
template <int NT = kBlk>
__device__ double block_min(double v, double* sh) { return -block_max<NT>(-v, sh); }

// Eight consecutive elements of a row as raw bits, widened to doubles when
// used (so that many rows' loads can be in flight in few registers).
template <class T>
struct Raw8;
template <>
struct Raw8<bf16_t> {
  uint4 u;
  // Always loads (from the row's last 8 elements when k is past dim - 8), so
  // the loads carry no branch; get() zeroes a step past the limit.
  __device__ __forceinline__ void load(const bf16_t* row, int k, int dim) {
    u = *reinterpret_cast<const uint4*>(row + min(k, dim - 8));
  }
  __device__ __forceinline__ void get(double (&o)[8], bool valid) const {
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      o[2 * i] = valid ? (double)__uint_as_float(w[i] << 16) : 0.0;
      o[2 * i + 1] = valid ? (double)__uint_as_float(w[i] & 0xFFFF0000u) : 0.0;
    }
  }
};
template <>
struct Raw8<float> {
  float4 a, b;
  __device__ __forceinline__ void load(const float* row, int k, int dim) {
    const float4* p = reinterpret_cast<const float4*>(row + min(k, dim - 8));
    a = p[0];
    b = p[1];
  }
  __device__ __forceinline__ void get(double (&o)[8], bool valid) const {
    const float v[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = valid ? (double)v[e] : 0.0;
  }
};

// ---------------------------------------------------------------------------
// Coarse pass (Section 3.1): v_f, a_f and the query mean.
// One block per (item, 512-element slice of the embedding, 8 per lane); the
// items are every frame of every clip, then one per clip for the query.
// The slices of an item are consecutive block indices, so the blocks that
// read the same rows run together and each DRAM page is opened once.
// The block's four waves take every fourth row of the frame's visual tokens,
// of its audio bin (or of the clip's query span); their fp64 partial sums
// meet in LDS and are added in wave order.  A wave loads eight of its rows
// (four of the audio bin's) together as raw bits before widening any, so
// that enough bytes are in flight for HBM.  The same pass leaves
// each visual and audio row's sum of squares over the slice in
// sqp[slice][row] (audio rows after the n_vis visual rows), so the token
// norms need no second read of X_V and X_A.
// ---------------------------------------------------------------------------
constexpr int kPoolWaves = kBlk / 64;      // row groups per block

template <class T>
__global__ __launch_bounds__(kBlk) void k_pool(const ClipDev* __restrict__ clips, const FrameDev* __restrict__ frames,
                                               int64_t total_frames, int dim, int slices, const T* __restrict__ xv,
                                               const T* __restrict__ xa, const T* __restrict__ xq,
                                               double* __restrict__ v, double* __restrict__ a,
                                               double* __restrict__ q, int64_t n_vis, int64_t sq_stride,
                                               double* __restrict__ sqp) {
  __shared__ double part[2][kPoolWaves - 1][kPoolSlice];
  const int lane = threadIdx.x & 63, rg = threadIdx.x >> 6;
  const int64_t item = blockIdx.x / slices;
  const int slice = (int)(blockIdx.x - item * slices);
  const int d0 = slice * kPoolSlice + lane * 8;
  // Lanes past dim read nothing and add zeros: every lane of a wave takes
  // part in the row norms' cross-lane sums, and the block meets at a barrier.
  const bool live = d0 < dim;
  auto row8 = [&](const T* p, double (&o)[8]) {
    if (live) {
      load8(p, o);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = 0.0;
    }
  };
  double* sq = sqp + (int64_t)slice * sq_stride;
  double av[8], aa[8], o[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) av[e] = aa[e] = 0.0;
  const bool is_frame = item < total_frames;
  int64_t frame = 0, lo = 0, hi = 0, rows_v = 1;
  int ci = 0;
  if (is_frame) {
    const FrameDev fr = frames[item];
    const ClipDev c = clips[fr.clip];
    frame = c.frame_off + fr.f;
    rows_v = c.per_frame;
    // Adaptive average-pool bin of the audio rows for this frame.
    lo = ((int64_t)fr.f * c.n_audio) / c.n_frames;
    hi = (((int64_t)fr.f + 1) * c.n_audio + c.n_frames - 1) / c.n_frames;
    const int64_t row0 = c.vis_off + (int64_t)fr.f * c.per_frame;
    // Lanes past dim load the row's last eight elements (Raw8 clamps) and
    // widen them to zeros.
    const T* vrow = xv + row0 * dim;
    // The wave's rows rg, rg + 4, ... eight at a time: the eight loads are
    // issued together as raw bits (a row past the frame re-reads its last
    // row and adds nothing), then widened and added in row order; the sums
    // of squares are reduced four rows at a time.
    const int P = c.per_frame;
    for (int p0 = rg; p0 < P; p0 += 8 * kPoolWaves) {
      Raw8<T> raw[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) raw[j].load(vrow + (int64_t)min(p0 + j * kPoolWaves, P - 1) * dim, d0, dim);
      double s2[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        s2[j] = 0.0;
        if (p0 + j * kPoolWaves < P) {
          double o8[8];
          raw[j].get(o8, live);
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            av[e] += o8[e];
            s2[j] = fma(o8[e], o8[e], s2[j]);
          }
        }
      }
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const double t = wave_sum4(*reinterpret_cast<const double(*)[4]>(&s2[4 * h]));
        const int p = p0 + (4 * h + lane) * kPoolWaves;
        if (lane < 4 && p < P) sq[row0 + p] = t;
      }
    }
    // The audio bin's rows rg, rg + 4, ... four at a time, the same way.
    // A row shared by two bins gets the same value from both.
    const T* arow = xa + c.aud_off * dim;
    for (int64_t r0 = lo + rg; r0 < hi; r0 += 4 * kPoolWaves) {
      Raw8<T> raw[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) raw[j].load(arow + min(r0 + j * kPoolWaves, hi - 1) * dim, d0, dim);
      double s2[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        s2[j] = 0.0;
        if (r0 + j * kPoolWaves < hi) {
          double o8[8];
          raw[j].get(o8, live);
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            aa[e] += o8[e];
            s2[j] = fma(o8[e], o8[e], s2[j]);
          }
        }
      }
      const double t = wave_sum4(s2);
      const int64_t r = r0 + lane * kPoolWaves;
      if (lane < 4 && r < hi) sq[n_vis + c.aud_off + r] = t;
    }
  } else {
    ci = (int)(item - total_frames);
    const ClipDev c = clips[ci];
    rows_v = c.n_query;
#pragma unroll 4
    for (int64_t r = rg; r < c.n_query; r += kPoolWaves) {
      row8(xq + (c.qry_off + r) * dim + d0, o);
#pragma unroll
      for (int e = 0; e < 8; ++e) av[e] += o[e];
    }
  }
  if (rg > 0) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      part[0][rg - 1][lane * 8 + e] = av[e];
      part[1][rg - 1][lane * 8 + e] = aa[e];
    }
  }
  __syncthreads();
  if (rg != 0 || !live) return;
  for (int w = 0; w < kPoolWaves - 1; ++w)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      av[e] += part[0][w][lane * 8 + e];
      aa[e] += part[1][w][lane * 8 + e];
    }
  if (is_frame) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      v[frame * dim + d0 + e] = av[e] / (double)rows_v;
      a[frame * dim + d0 + e] = hi > lo ? aa[e] / (double)(hi - lo) : 0.0;
    }
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) q[(int64_t)ci * dim + d0 + e] = av[e] / (double)rows_v;
  }
}

// ---------------------------------------------------------------------------
// Band Gram entries of one frame: v_f.v_{f+d}, a_f.a_{f+d} for d < w, v_f.q
// (and q.q for the first frame of the clip).  W bounds the partners a frame
// needs (w, and 2 for the continuity cosine), so only 2W + 2 sums are formed
// and reduced; entries are stored kMaxWindow apart.  NT threads per frame:
// 1024 when a launch has few frames (each frame's loads then spread over
// four times the waves), 256 otherwise.
// ---------------------------------------------------------------------------
constexpr int kBandWideFrames = 1024;  // below this many frames, 1024 threads per frame
template <int W, int NT>
__global__ __launch_bounds__(NT) void k_band(const ClipDev* __restrict__ clips, const FrameDev* __restrict__ frames,
                                               int dim, int w, const double* __restrict__ v,
                                               const double* __restrict__ a, const double* __restrict__ q,
                                               double* __restrict__ band_v, double* __restrict__ band_a,
                                               double* __restrict__ vq, double* __restrict__ qq) {
  constexpr int NA = 2 * W + 2;
  __shared__ double sh[NT / 64][NA];
  const FrameDev fr = frames[blockIdx.x];
  const ClipDev c = clips[fr.clip];
  const int64_t f0 = c.frame_off + fr.f;
  const int nd = min(max(w, 2), c.n_frames - fr.f);  // partners f .. f+nd-1 (f+1 for continuity)
  const double* qv = q + (int64_t)fr.clip * dim;
  double acc[NA];
#pragma unroll
  for (int i = 0; i < NA; ++i) acc[i] = 0.0;
  for (int d = threadIdx.x; d < dim; d += NT) {
    const double vf = v[f0 * dim + d], af = a[f0 * dim + d], qd = qv[d];
#pragma unroll
    for (int dd = 0; dd < W; ++dd) {
      if (dd < nd) {
        acc[dd] += vf * v[(f0 + dd) * dim + d];
        acc[W + dd] += af * a[(f0 + dd) * dim + d];
      }
    }
    acc[2 * W] += vf * qd;
    acc[2 * W + 1] += qd * qd;
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int i = 0; i < NA; ++i) {
    const double s = wave_sum(acc[i]);
    if (lane == 0) sh[wave][i] = s;
  }
  __syncthreads();
  const int i = threadIdx.x;
  if (i < NA) {
    double s = 0.0;
    for (int ww = 0; ww < NT / 64; ++ww) s += sh[ww][i];
    if (i < W) {
      if (i < nd) band_v[f0 * kMaxWindow + i] = s;
    } else if (i < 2 * W) {
      if (i - W < nd) band_a[f0 * kMaxWindow + (i - W)] = s;
    } else if (i == 2 * W) {
      vq[f0] = s;
    } else if (fr.f == 0) {
      qq[fr.clip] = s;
    }
  }
}

// Gram entry (i, j) of frames i, j of a clip from the band (|i - j| < w).
__device__ __forceinline__ double band_at(const double* band, int64_t f0, int i, int j) {
  return i <= j ? band[(f0 + i) * kMaxWindow + (j - i)] : band[(f0 + j) * kMaxWindow + (i - j)];
}

// ---------------------------------------------------------------------------
// Eq. 1 per frame over its clamped window, the clip mean and the gate.
// W >= w bounds the window, so the loops unroll and the row means stay in
// registers; the Gram entries are read from the band where they are used.
// ---------------------------------------------------------------------------
template <int W>
__global__ __launch_bounds__(kBlk) void k_cka(ClipDev* __restrict__ clips, int w, double tau, int alignment,
                                              const double* __restrict__ band_v, const double* __restrict__ band_a,
                                              double* __restrict__ cka, float* __restrict__ frame_cka,
                                              uint8_t* __restrict__ gate_out) {
  __shared__ double sh[kBlk / 64];
  ClipDev* c = &clips[blockIdx.x];
  const int F = c->n_frames;
  const int64_t f0 = c->frame_off;
  const int ww = F <= w ? F : w;
  double sum = 0.0;
  for (int f = threadIdx.x; f < F; f += kBlk) {
    if (alignment == APACK_ALIGN_SPATIAL_CKA) {  // c_f already written by k_spatial_reduce
      const double cf = cka[f0 + f];
      if (frame_cka) frame_cka[f0 + f] = (float)cf;
      sum += cf;
      continue;
    }
    int lo = 0;
    if (F > w) lo = min(max(f - w / 2, 0), F - w);
    // Centred Grams K = H G H of the window rows lo .. lo+ww-1, and the
    // traces of the raw Grams G.
    double ra[W], rv[W], ta = 0.0, tv = 0.0, tra = 0.0, trv = 0.0;
#pragma unroll
    for (int i = 0; i < W; ++i) {
      ra[i] = rv[i] = 0.0;
      if (i < ww) {
#pragma unroll
        for (int j = 0; j < W; ++j) {
          if (j < ww) {
            ra[i] += band_at(band_a, f0, lo + i, lo + j);
            rv[i] += band_at(band_v, f0, lo + i, lo + j);
          }
        }
        ra[i] /= ww;
        rv[i] /= ww;
        ta += ra[i];
        tv += rv[i];
        tra += band_at(band_a, f0, lo + i, lo + i);
        trv += band_at(band_v, f0, lo + i, lo + i);
      }
    }
    ta /= ww;
    tv /= ww;
    double num = 0.0, na = 0.0, nv = 0.0;
#pragma unroll
    for (int i = 0; i < W; ++i) {
      if (i >= ww) continue;
#pragma unroll
      for (int j = 0; j < W; ++j) {
        if (j >= ww) continue;
        const double ka = band_at(band_a, f0, lo + i, lo + j) - ra[i] - ra[j] + ta;
        const double kv = band_at(band_v, f0, lo + i, lo + j) - rv[i] - rv[j] + tv;
        num += ka * kv;
        na += ka * ka;
        nv += kv * kv;
      }
    }
    // A degenerate side (no variation the Gram resolves) gives 0.
    const double sa = sqrt(na), sv = sqrt(nv);
    const double cf = (sa <= kCkaDegenerate * tra || sv <= kCkaDegenerate * trv) ? 0.0 : num / (sa * sv);
    cka[f0 + f] = cf;
    if (frame_cka) frame_cka[f0 + f] = (float)cf;
    sum += cf;
  }
  sum = block_sum(sum, sh);
  if (threadIdx.x == 0) {
    // The window (or spatial) CKA gate of Eq. 2; CKA alone never fires it,
    // AV cosine always does.
    int fired = (F > 0 && sum / F < tau) ? 1 : 0;
    if (alignment == APACK_ALIGN_CKA) fired = 0;
    if (alignment == APACK_ALIGN_AV_COSINE) fired = F > 0 ? 1 : 0;
    c->gate = fired;
    if (gate_out) gate_out[blockIdx.x] = (uint8_t)fired;
  }
}

// ---------------------------------------------------------------------------
// Squared norms of the visual rows [0, n_vis) and audio rows [0, n_aud) of
// the clips, from k_pool's per-slice partials added in slice order; the
// visual max-cosine keys start at 0 (below every real key).  Rows in no
// clip get whatever their slots held and are never read.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlk) void k_norms(int64_t n_vis, int64_t n_aud, int slices,
                                                const double* __restrict__ sqp, double* __restrict__ nv,
                                                double* __restrict__ rv, double* __restrict__ na,
                                                uint32_t* __restrict__ maxkey) {
  const int64_t stride = n_vis + n_aud;
  const int64_t row = (int64_t)blockIdx.x * kBlk + threadIdx.x;
  if (row >= stride) return;
  double s = 0.0;
  for (int k = 0; k < slices; ++k) s += sqp[(int64_t)k * stride + row];
  if (row < n_vis) {
    nv[row] = s;
    rv[row] = s > 0.0 ? 1.0 / sqrt(s) : 0.0;   // 1/|x| for the direct distance, 0 for a zero token
    maxkey[row] = 0u;
  } else {
    na[row - n_vis] = s;
  }
}

// ---------------------------------------------------------------------------
// Gate GEMM: for every visual token i, max_j (x_A[j] . x_V[i]) / |x_A[j]|.
// C = X_A X_V^T in 128 x 128 tiles (4 waves, 64 x 64 each), K through
// padded, double-buffered LDS in steps of 64 elements.
// ---------------------------------------------------------------------------
template <class T> struct GMma;
template <> struct GMma<bf16_t> {
  using frag = bf16x8;
  static constexpr int kstep = 16, lane_k = 8;
  static __device__ __forceinline__ f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};
template <> struct GMma<float> {
  using frag = float;
  static constexpr int kstep = 2, lane_k = 1;
  static __device__ __forceinline__ f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
};

constexpr int kGB = 128;   // tile rows and columns
constexpr int kGK = 64;    // K elements per LDS stage

template <class T>
__global__ __launch_bounds__(kBlk) void k_gate_gemm(const ClipDev* __restrict__ clips,
                                                    const GemmTileDev* __restrict__ tiles, int dim,
                                                    const T* __restrict__ xv, const T* __restrict__ xa,
                                                    const double* __restrict__ na, uint32_t* __restrict__ maxkey) {
  using M = GMma<T>;
  constexpr int kRowBytes = kGK * (int)sizeof(T);
  constexpr int kPitch = kRowBytes + 16;
  constexpr int kUnits = kRowBytes / 16;          // 16-byte units per tile row
  constexpr int kPer = kGB * kUnits / kBlk;       // units per thread per tile
  constexpr int kEl = 16 / (int)sizeof(T);        // elements per unit
  __shared__ __attribute__((aligned(16))) char lds_a[2][kGB * kPitch];
  __shared__ __attribute__((aligned(16))) char lds_b[2][kGB * kPitch];

  const GemmTileDev tl = tiles[blockIdx.x];
  const ClipDev c = clips[tl.clip];
  if (!c.gate) return;
  const int64_t n_a = c.n_audio, n_v = (int64_t)c.n_frames * c.per_frame;
  const T* A = xa + c.aud_off * dim;
  const T* B = xv + c.vis_off * dim;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave >> 1, wc = wave & 1;

  uint4 ra[kPer], rb[kPer];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int u = tid + i * kBlk;
      const int row = u / kUnits, col = u % kUnits;
      const int kk = k0 + col * kEl;
      uint4 x = make_uint4(0, 0, 0, 0), y = make_uint4(0, 0, 0, 0);
      if (tl.m0 + row < n_a && kk < dim) x = *reinterpret_cast<const uint4*>(A + (tl.m0 + row) * (int64_t)dim + kk);
      if (tl.n0 + row < n_v && kk < dim) y = *reinterpret_cast<const uint4*>(B + (tl.n0 + row) * (int64_t)dim + kk);
      ra[i] = x;
      rb[i] = y;
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int u = tid + i * kBlk;
      const int row = u / kUnits, col = u % kUnits;
      *reinterpret_cast<uint4*>(lds_a[buf] + row * kPitch + col * 16) = ra[i];
      *reinterpret_cast<uint4*>(lds_b[buf] + row * kPitch + col * 16) = rb[i];
    }
  };
  auto frag = [&](const char* lds, int row, int ks) {
    const char* p = lds + row * kPitch + (ks * M::kstep + (lane >> 5) * M::lane_k) * (int)sizeof(T);
    return *reinterpret_cast<const typename M::frag*>(p);
  };

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};
  const int n_k = (dim + kGK - 1) / kGK;
  gload(0);
  for (int it = 0; it < n_k; ++it) {
    const int buf = it & 1;
    lstore(buf);
    __syncthreads();
    if (it + 1 < n_k) gload((it + 1) * kGK);
#pragma unroll
    for (int ks = 0; ks < kGK / M::kstep; ++ks) {
      typename M::frag fa[2], fb[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        fa[i] = frag(lds_a[buf], wr * 64 + i * 32 + (lane & 31), ks);
        fb[i] = frag(lds_b[buf], wc * 64 + i * 32 + (lane & 31), ks);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = M::mma(fa[i], fb[j], acc[i][j]);
    }
  }
  // Epilogue: acc[i][j][e] is audio row wr*64 + i*32 + 8*(e/4) + 4*(lane/32) + e%4,
  // visual column wc*64 + j*32 + lane%32.
  float inv[2][16];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int64_t r = tl.m0 + wr * 64 + i * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
      float s = -INFINITY;  // rows past the clip's audio never win the max
      if (r < n_a) {
        const double nn = na[c.aud_off + r];
        s = nn > 0.0 ? (float)(1.0 / sqrt(nn)) : 0.0f;
      }
      inv[i][e] = s;
    }
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    float m = -INFINITY;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float x = inv[i][e] == -INFINITY ? -INFINITY : acc[i][j][e] * inv[i][e];
        m = fmaxf(m, x);
      }
    m = fmaxf(m, __shfl_xor(m, 32));
    const int64_t col = tl.n0 + wc * 64 + j * 32 + (lane & 31);
    if (lane < 32 && col < n_v && m > -INFINITY) atomicMax(&maxkey[c.vis_off + col], order_key(m));
  }
}

// ---------------------------------------------------------------------------
// Capped largest-remainder apportionment of `total` over items [0, n) with
// weights w[i] and caps cap[i], run by one wave: lane l owns items l, l + 64,
// ... and alone writes their fixed, quota and alloc entries.  Water-filling
// first (items whose quota exceeds their cap are fixed at the cap, the rest
// re-shared), then floors and the leftover units to the largest fractional
// parts, lower index first on ties.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "workgroup");
  __builtin_amdgcn_wave_barrier();
}

__device__ void apportion_wave(int64_t total, int n, const double* w, const int64_t* cap, int32_t* fixed,
                               double* quota, int64_t* alloc) {
  const int lane = threadIdx.x & 63;
  for (int i = lane; i < n; i += 64) fixed[i] = 0;
  for (int round = 0; round <= n; ++round) {
    double fixed_caps = 0.0, sw = 0.0, nfree = 0.0;
    for (int i = lane; i < n; i += 64) {
      if (fixed[i]) fixed_caps += (double)cap[i];
      else {
        sw += w[i];
        nfree += 1.0;
      }
    }
    fixed_caps = wave_sum(fixed_caps);
    sw = wave_sum(sw);
    nfree = wave_sum(nfree);
    const double remaining = (double)total - fixed_caps;
    bool over = false;
    for (int i = lane; i < n; i += 64) {
      if (fixed[i]) continue;
      const double qv = sw > 0.0 ? remaining * w[i] / sw : remaining / nfree;
      quota[i] = qv;
      if (qv > (double)cap[i]) {  // fixed at its cap from the next round on
        fixed[i] = 1;
        over = true;
      }
    }
    if (__ballot(over) == 0) break;
  }
  double used = 0.0;
  for (int i = lane; i < n; i += 64) {
    const double fl = floor(quota[i]);
    const int64_t a = fixed[i] ? cap[i] : (int64_t)fl;
    alloc[i] = a;
    used += (double)a;
    quota[i] = fixed[i] ? -1.0 : quota[i] - fl;  // fractional part; fixed items take no leftover unit
  }
  used = wave_sum(used);
  const int64_t left = total - (int64_t)used;
  if (left <= 0) return;
  wave_sync();
  for (int i = lane; i < n; i += 64) {
    const double fi = quota[i];
    if (fi < 0.0) continue;
    int64_t rank = 0;
    for (int j = 0; j < n; ++j) {
      const double fj = quota[j];
      rank += (fj > fi || (fj == fi && j < i)) ? 1 : 0;
    }
    if (rank < left) alloc[i] += 1;
  }
}

// Inclusive scan of one value per thread over a block of NT threads; sh
// holds NT / 64 words and `total` receives the block's sum.
template <int NT>
__device__ __forceinline__ uint32_t block_scan_u32(uint32_t v, uint32_t* sh, uint32_t& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t o = __shfl_up(v, off);
    if (lane >= off) v += o;
  }
  if (lane == 63) sh[wave] = v;
  __syncthreads();
  uint32_t base = 0;
  total = 0;
#pragma unroll
  for (int w = 0; w < NT / 64; ++w) {
    const uint32_t x = sh[w];
    if (w < wave) base += x;
    total += x;
  }
  __syncthreads();
  return v + base;
}

// ---------------------------------------------------------------------------
// Per-clip plan: scores, segments and budgets, one 1024-thread workgroup per
// clip.  Its per-frame arrays (F + 1 entries each) sit in LDS for clips of
// fewer than kPlanLds frames; longer clips use the global scratch, which
// holds (sum F + n_clips) entries per array, clip c at frame_off + c.  The
// code reaches both through the same generic pointers.
// ---------------------------------------------------------------------------
constexpr int kPlanBlk = 1024;
constexpr int kPlanLds = 1024;

struct PlanScratch {
  double *d, *alpha, *cont, *smooth, *rel, *score, *g, *quota, *fquota;
  int64_t *cap, *alloc, *fcap, *falloc;
  int32_t *fixed, *ffixed, *start;
};

// Nine fp64, four int64 and three int32 arrays of n entries each, in that
// order, starting `o` entries into each.
__device__ __forceinline__ PlanScratch carve_plan(double* b, int64_t n, int64_t o) {
  int64_t* ib = reinterpret_cast<int64_t*>(b + 9 * n);
  int32_t* jb = reinterpret_cast<int32_t*>(ib + 4 * n);
  PlanScratch s;
  s.d = b + o; s.alpha = b + n + o; s.cont = b + 2 * n + o; s.smooth = b + 3 * n + o; s.rel = b + 4 * n + o;
  s.score = b + 5 * n + o; s.g = b + 6 * n + o; s.quota = b + 7 * n + o; s.fquota = b + 8 * n + o;
  s.cap = ib + o; s.alloc = ib + n + o; s.fcap = ib + 2 * n + o; s.falloc = ib + 3 * n + o;
  s.fixed = jb + o; s.ffixed = jb + n + o; s.start = jb + 2 * n + o;
  return s;
}
constexpr int kPlanLdsBytes = kPlanLds * (9 * 8 + 4 * 8 + 3 * 4);

__global__ __launch_bounds__(kPlanBlk) void k_plan(ClipDev* __restrict__ clips, DynParamsDev prm,
                                                   const double* __restrict__ cka, const double* __restrict__ band_v,
                                                   const double* __restrict__ vq, const double* __restrict__ qq,
                                                   const double* __restrict__ rv, const uint32_t* __restrict__ maxkey,
                                                   FramePlanDev* __restrict__ plan, int32_t* __restrict__ anchors,
                                                   double* scratch, int64_t scratch_n,
                                                   float* __restrict__ frame_score,
                                                   int32_t* __restrict__ frame_budget,
                                                   int32_t* __restrict__ segment_id) {
  __shared__ double sh[kPlanBlk / 64];
  __shared__ uint32_t shu[kPlanBlk / 64];
  __shared__ __align__(16) double lds[kPlanLdsBytes / 8];
  ClipDev* cp = &clips[blockIdx.x];
  const ClipDev c = *cp;
  const int F = c.n_frames, P = c.per_frame;
  if (F == 0) return;
  const int64_t f0 = c.frame_off;
  const int tid = threadIdx.x;
  const PlanScratch w = F + 1 <= kPlanLds ? carve_plan(lds, kPlanLds, 0)
                                          : carve_plan(scratch, scratch_n, f0 + blockIdx.x);
  double *d = w.d, *alpha = w.alpha, *cont = w.cont, *smooth = w.smooth, *rel = w.rel, *score = w.score;
  double *g = w.g, *quota = w.quota, *fquota = w.fquota;
  int64_t *cap = w.cap, *alloc = w.alloc, *fcap = w.fcap, *falloc = w.falloc;
  int32_t *fixed = w.fixed, *ffixed = w.ffixed, *start = w.start;

  // Direct distance (eight threads per frame) and the Eq. 2 blend.
  if (c.gate) {
    const int sub = tid & 7;
    for (int f = tid >> 3; f < F; f += kPlanBlk / 8) {  // the eight threads of a frame share the trip count
      const int64_t row0 = c.vis_off + (int64_t)f * P;
      double sm = 0.0;
      // Six rows per thread per batch, all twelve loads issued before the
      // first is used: a zero-norm row has r == 0 and adds 0, a slot no
      // audio column reached (key 0) reads as 0, and a row past the frame
      // re-reads the frame's last row and is then zeroed, so nothing
      // branches on a loaded value. The sum keeps the order of p.
      constexpr int kU = 6;
      for (int p0 = sub; p0 < P; p0 += 8 * kU) {
        double r[kU];
        uint32_t mk[kU];
#pragma unroll
        for (int u = 0; u < kU; ++u) {
          const int p = min(p0 + 8 * u, P - 1);
          r[u] = rv[row0 + p];
          mk[u] = maxkey[row0 + p];
        }
#pragma unroll
        for (int u = 0; u < kU; ++u) {
          const float kv = mk[u] != 0u ? key_value(mk[u]) : 0.0f;
          const double t = (double)kv * r[u];
          sm += p0 + 8 * u < P ? t : 0.0;
        }
      }
      sm += __shfl_xor(sm, 1);
      sm += __shfl_xor(sm, 2);
      sm += __shfl_xor(sm, 4);
      if (sub == 0) {
        const double df = 1.0 - sm / P;
        d[f] = df;
        plan[f0 + f].dist = df;
      }
    }
    __syncthreads();
    double lo = INFINITY, hi = -INFINITY;
    for (int f = tid; f < F; f += kPlanBlk) {
      lo = fmin(lo, d[f]);
      hi = fmax(hi, d[f]);
    }
    lo = block_min<kPlanBlk>(lo, sh);
    hi = block_max<kPlanBlk>(hi, sh);
    for (int f = tid; f < F; f += kPlanBlk) {
      const double dh = hi == lo ? 0.0 : (d[f] - lo) / (hi - lo);
      alpha[f] = (1.0 - prm.beta) * cka[f0 + f] + prm.beta * (1.0 - dh);
    }
  } else {
    for (int f = tid; f < F; f += kPlanBlk) {
      alpha[f] = cka[f0 + f];
      plan[f0 + f].dist = 0.0;
    }
  }
  // Continuity cs_f = cos(v_f, v_{f+1}), its Gaussian smoothing (half-sample
  // symmetric ends, truncated at 4 sigma) and the relevance r_f.
  const double qn = qq[blockIdx.x];
  for (int f = tid; f < F; f += kPlanBlk) {
    const double nx = band_v[(f0 + f) * kMaxWindow];
    if (f + 1 < F) cont[f] = cos_from(band_v[(f0 + f) * kMaxWindow + 1], nx, band_v[(f0 + f + 1) * kMaxWindow]);
    rel[f] = (1.0 + cos_from(vq[f0 + f], nx, qn)) / 2.0;
  }
  __syncthreads();
  const int n = F - 1;
  const int radius = (int)(4.0 * prm.sigma + 0.5);
  for (int i = tid; i < n; i += kPlanBlk) {
    double wsum = 0.0;
    for (int k = -radius; k <= radius; ++k) wsum += exp(-0.5 * ((k / prm.sigma) * (k / prm.sigma)));
    double acc = 0.0;
    for (int k = -radius; k <= radius; ++k) {
      const double wt = exp(-0.5 * ((k / prm.sigma) * (k / prm.sigma))) / wsum;
      int j = (i + k) % (2 * n);
      if (j < 0) j += 2 * n;
      if (j >= n) j = 2 * n - 1 - j;
      acc += wt * cont[j];
    }
    smooth[i] = acc;
  }
  __syncthreads();
  // Cuts: one per maximal run of the smoothed continuity below tau_sim,
  // after the run's first minimum.  The thread at a run's first frame walks
  // the run; a block scan places the cuts in frame order.
  int n_seg = 1;
  for (int c0 = 0; c0 < n; c0 += kPlanBlk) {
    const int f = c0 + tid;
    const bool run_start = f < n && smooth[f] < prm.tau_sim && (f == 0 || !(smooth[f - 1] < prm.tau_sim));
    int cut = 0;
    if (run_start) {
      int e = f, best = f;
      while (e + 1 < n && smooth[e + 1] < prm.tau_sim) {
        ++e;
        if (smooth[e] < smooth[best]) best = e;
      }
      cut = best + 1;
    }
    uint32_t total;
    const uint32_t incl = block_scan_u32<kPlanBlk>(run_start ? 1u : 0u, shu, total);
    if (run_start) start[n_seg + (int)incl - 1] = cut;
    n_seg += (int)total;
  }
  if (tid == 0) {
    start[0] = 0;
    start[n_seg] = F;
    cp->n_seg = n_seg;
  }
  __syncthreads();
  for (int m = tid; m < n_seg; m += kPlanBlk) anchors[f0 + m] = start[m];
  // Segment scores g_m (Eq. 3) and caps |G_m| P.
  for (int m = tid; m < n_seg; m += kPlanBlk) {
    const int b = start[m], e = start[m + 1];
    double mx = -INFINITY, sm = 0.0;
    for (int f = b; f < e; ++f) {
      mx = fmax(mx, rel[f]);
      sm += rel[f];
    }
    const int len = e - b;
    g[m] = sqrt((double)len) * (prm.lambda_seg * mx + (1.0 - prm.lambda_seg) * (sm / len));
    cap[m] = (int64_t)len * P;
  }
  __syncthreads();
  double gmax = -INFINITY;
  for (int m = tid; m < n_seg; m += kPlanBlk) gmax = fmax(gmax, g[m]);
  gmax = block_max<kPlanBlk>(gmax, sh);
  // Frame scores s_f = gamma u_f + (1 - gamma) alpha_f with u_f = g_m / max g;
  // frame f lies in the last segment m with start[m] <= f.
  for (int f = tid; f < F; f += kPlanBlk) {
    int lo = 0, hi = n_seg - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (start[mid] <= f) lo = mid;
      else hi = mid - 1;
    }
    const int m = lo, b = start[m];
    const double sv = prm.gamma * (g[m] / gmax) + (1.0 - prm.gamma) * alpha[f];
    score[f] = sv;
    plan[f0 + f].score = sv;
    plan[f0 + f].seg = m;
    plan[f0 + f].anchor = b;
    plan[f0 + f].is_anchor = f == b ? 1 : 0;
    if (frame_score) frame_score[f0 + f] = (float)sv;
    if (segment_id) segment_id[f0 + f] = m;
  }
  // Segment budgets (Eq. 4), capped at |G_m| P, by wave 0; then frame
  // budgets within each segment by s_f, capped at P, one wave per segment
  // (a segment's entries of the per-frame arrays are its own frames').
  if (tid < 64) apportion_wave(c.budget, n_seg, g, cap, fixed, quota, alloc);
  __syncthreads();
  const int wave = tid >> 6, lane = tid & 63;
  for (int m = wave; m < n_seg; m += kPlanBlk / 64) {
    const int b = start[m], e = start[m + 1];
    for (int i = lane; i < e - b; i += 64) fcap[b + i] = P;
    apportion_wave(alloc[m], e - b, score + b, fcap + b, ffixed + b, fquota + b, falloc + b);
    for (int i = lane; i < e - b; i += 64) plan[f0 + b + i].budget = (int32_t)falloc[b + i];
  }
  __syncthreads();
  // Output offsets: exclusive prefix of k_f over the clip's frames.
  int64_t base = c.kept_off;
  for (int c0 = 0; c0 < F; c0 += kPlanBlk) {
    const int f = c0 + tid;
    const uint32_t k = f < F ? (uint32_t)falloc[f] : 0u;
    uint32_t total;
    const uint32_t incl = block_scan_u32<kPlanBlk>(k, shu, total);
    if (f < F) {
      plan[f0 + f].out_off = base + (int64_t)(incl - k);
      if (frame_budget) frame_budget[f0 + f] = (int32_t)k;
    }
    base += total;
  }
}

// ---------------------------------------------------------------------------
// Gram of an anchor frame's P tokens in fp64 on the matrix cores
// (v_mfma_f64_16x16x4f64).  One workgroup per 16 x 16 tile of the upper
// triangle of an anchor frame, looping over the batch's (anchor, tile)
// items; its kGramSplit waves take contiguous slices of the embedding and
// add their partial tiles in wave order through LDS.  Each tile is written
// twice, (i, j) and (j, i), so S is exactly symmetric.
// MFMA operands: lane l supplies A[l % 16][k = l / 16] and B[k = l / 16][l % 16];
// accumulator element e of lane l is D[4e + l / 16][l % 16].  Each lane
// loads 8 consecutive elements of its row and feeds them to 8 MFMAs, lane
// group g = l / 16 covering elements [k0 + 8g, k0 + 8g + 8) of a 32-element
// step; A and B use the same assignment, so every product enters once.
// ---------------------------------------------------------------------------
typedef double f64x4 __attribute__((ext_vector_type(4)));
constexpr int kGramTile = 16;
constexpr int kGramWaves = 4;  // tiles per workgroup of the spatial Gram
constexpr int kGramSplit = 8;  // K slices (waves) per workgroup of the anchor Gram
constexpr int kGramBlocks = 512;  // workgroups of the anchor Gram at most: two per CU
constexpr int kGramAhead = 4;  // K steps in flight per wave

// Eight consecutive input elements held as loaded, widened to fp64 on use.
template <class T>
__global__ __launch_bounds__(kGramSplit * 64) void k_gram(const ClipDev* __restrict__ clips, int n_clips,
                                                          const int32_t* __restrict__ anchors,
                                                          const FramePlanDev* __restrict__ plan, int dim,
                                                          const T* __restrict__ xv, double* __restrict__ gram) {
  __shared__ double red[kGramSplit - 1][4 * 64];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, g = lane >> 4, r16 = lane & 15;
  // This wave's K slice, in 32-element steps.
  const int nsteps = (dim + 31) / 32;
  const int per = (nsteps + kGramSplit - 1) / kGramSplit;
  const int s_begin = min(nsteps, wave * per), s_end = min(nsteps, s_begin + per);
  const int lim = min(dim, 32 * s_end);
  // Anchors go to XCDs round-robin (workgroup b runs on XCD b % 8), so an
  // anchor's rows are fetched into one L2; the XCD's slots share its
  // anchors' tiles in turn.  Every workgroup walks the same anchor sequence.
  const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3, nslot = gridDim.x >> 3;
  int c = 0;
  int64_t seg_before = 0;  // anchors of clips [0, c)
  int64_t jbase = 0;       // tiles of this XCD's earlier anchors
  for (int64_t an = xcd;; an += 8) {
    while (c < n_clips) {
      const int64_t ns = clips[c].n_frames > 0 ? clips[c].n_seg : 0;
      if (an < seg_before + ns) break;
      seg_before += ns;
      ++c;
    }
    if (c >= n_clips) return;
    const ClipDev cc = clips[c];
    const int P = cc.per_frame, nt = (P + kGramTile - 1) / kGramTile, tiles = nt * (nt + 1) / 2;
    const int f = anchors[cc.frame_off + (an - seg_before)];
    const int64_t j0 = jbase + ((slot - jbase % nslot) % nslot + nslot) % nslot;
    const int64_t jend = jbase + tiles;
    jbase = jend;
    if (plan[cc.frame_off + f].budget == 0) continue;  // the same for the whole workgroup
    for (int64_t jj = j0; jj < jend; jj += nslot) {
      int t = (int)(jj - (jend - tiles)), ti = 0;
      while (t >= nt - ti) {  // row-major upper triangle: tile (ti, tj), tj >= ti
        t -= nt - ti;
        ++ti;
      }
      const int tj = ti + t;
      const int64_t row0 = cc.vis_off + (int64_t)f * P;
      const int ra = min(ti * kGramTile + r16, P - 1), rb = min(tj * kGramTile + r16, P - 1);
      const T* xa = xv + (row0 + ra) * dim;
      const T* xb = xv + (row0 + rb) * dim;
      // kGramAhead steps loaded ahead of the MFMAs (the next group's loads
      // are issued before this group's MFMAs); steps past the slice add
      // zero products.
      Raw8<T> pa[kGramAhead], pb[kGramAhead];
#pragma unroll
      for (int u = 0; u < kGramAhead; ++u) {
        const int kk = 32 * (s_begin + u) + 8 * g;
        pa[u].load(xa, kk, dim);
        pb[u].load(xb, kk, dim);
      }
      f64x4 acc = {0.0, 0.0, 0.0, 0.0};
      for (int s0 = s_begin; s0 < s_end; s0 += kGramAhead) {
        Raw8<T> qa[kGramAhead], qb[kGramAhead];
#pragma unroll
        for (int u = 0; u < kGramAhead; ++u) {
          const int kk = 32 * (s0 + kGramAhead + u) + 8 * g;
          qa[u].load(xa, kk, dim);
          qb[u].load(xb, kk, dim);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < kGramAhead; ++u) {
          const bool valid = 32 * (s0 + u) + 8 * g < lim;
          double a[8], b[8];
          pa[u].get(a, valid);
          pb[u].get(b, valid);
#pragma unroll
          for (int e = 0; e < 8; ++e) acc = __builtin_amdgcn_mfma_f64_16x16x4f64(a[e], b[e], acc, 0, 0, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < kGramAhead; ++u) {
          pa[u] = qa[u];
          pb[u] = qb[u];
        }
      }
      // Partial tiles added in wave order.
      if (wave > 0) {
#pragma unroll
        for (int e = 0; e < 4; ++e) red[wave - 1][e * 64 + lane] = acc[e];
      }
      __syncthreads();
      if (wave == 0) {
#pragma unroll
        for (int q = 0; q < kGramSplit - 1; ++q)
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[e] += red[q][e * 64 + lane];
        // Raw dot products: k_dafps forms the cosines from them and the
        // diagonal, which went through the same MFMA sequence.
        double* G = gram + cc.gram_off + (int64_t)f * P * P;
        const int col = tj * kGramTile + r16;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int row = ti * kGramTile + 4 * e + g;
          if (row >= P || col >= P) continue;
          G[(int64_t)row * P + col] = acc[e];
          G[(int64_t)col * P + row] = acc[e];
        }
      }
      __syncthreads();
    }
  }
}

// ---------------------------------------------------------------------------
// Spatial CKA at w = 1 (alternative alignment scorer): for frame f, the rows
// R = [A~; V~] stack the audio tokens of its adaptive-pool bin and its P
// visual tokens, each centred in fp64 by its own mean (a_f and v_f of
// k_pool).  One wave per 16 x 16 tile of the upper triangle of R R^T (fp64
// MFMA, operand layout as in k_gram) adds the squared entries of its tile
// to the audio-audio, audio-visual and visual-visual sums; off-diagonal
// tiles of the symmetric blocks count twice, and the cross block counts
// once, in its audio-row orientation.  The per-tile sums go to
// part[frame][tile][3] and k_spatial_reduce adds them in tile order.
// ---------------------------------------------------------------------------
template <class T>
__device__ __forceinline__ void load8_centred(const T* x, const double* mu, double (&o)[8]) {
  load8(x, o);
#pragma unroll
  for (int e = 0; e < 8; ++e) o[e] -= mu[e];
}

template <class T>
__global__ __launch_bounds__(kGramWaves * 64) void k_spatial_gram(const ClipDev* __restrict__ clips,
                                                                  const FrameDev* __restrict__ frames, int dim,
                                                                  const T* __restrict__ xv, const T* __restrict__ xa,
                                                                  const double* __restrict__ vmean,
                                                                  const double* __restrict__ amean, int tiles,
                                                                  double* __restrict__ part) {
  const FrameDev fr = frames[blockIdx.x];
  const ClipDev c = clips[fr.clip];
  const int64_t frame = c.frame_off + fr.f;
  const int P = c.per_frame;
  const int64_t lo = ((int64_t)fr.f * c.n_audio) / c.n_frames;
  const int64_t hi = (((int64_t)fr.f + 1) * c.n_audio + c.n_frames - 1) / c.n_frames;
  const int na = (int)(hi - lo), m = na + P;
  const int nt = (m + kGramTile - 1) / kGramTile;
  const int t0 = blockIdx.y * kGramWaves + (threadIdx.x >> 6);
  if (t0 >= tiles) return;
  const int lane = threadIdx.x & 63, g = lane >> 4, r16 = lane & 15;
  double* out = part + (frame * tiles + t0) * 3;
  if (t0 >= nt * (nt + 1) / 2) {  // past this frame's triangle: contributes nothing
    if (lane < 3) out[lane] = 0.0;
    return;
  }
  int t = t0, ti = 0;
  while (t >= nt - ti) {
    t -= nt - ti;
    ++ti;
  }
  const int tj = ti + t;
  // Row r of R: audio row lo + r (centred by a_f) or visual token r - na (by v_f).
  auto row_ptr = [&](int r, const T*& x, const double*& mu) {
    r = min(r, m - 1);
    if (r < na) {
      x = xa + (c.aud_off + lo + r) * dim;
      mu = amean + frame * dim;
    } else {
      x = xv + (c.vis_off + (int64_t)fr.f * P + (r - na)) * dim;
      mu = vmean + frame * dim;
    }
  };
  const T *pa, *pb;
  const double *ma, *mb;
  row_ptr(ti * kGramTile + r16, pa, ma);
  row_ptr(tj * kGramTile + r16, pb, mb);
  f64x4 acc = {0.0, 0.0, 0.0, 0.0};
  for (int k0 = 0; k0 < dim; k0 += 32) {
    const int kk = k0 + 8 * g;
    double a[8], b[8];
    if (kk < dim) {
      load8_centred(pa + kk, ma + kk, a);
      load8_centred(pb + kk, mb + kk, b);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) a[e] = b[e] = 0.0;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) acc = __builtin_amdgcn_mfma_f64_16x16x4f64(a[e], b[e], acc, 0, 0, 0);
  }
  double s_aa = 0.0, s_av = 0.0, s_vv = 0.0;
  const int col = tj * kGramTile + r16;
  const double twice = ti == tj ? 1.0 : 2.0;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int row = ti * kGramTile + 4 * e + g;
    if (row >= m || col >= m) continue;
    const double x2 = acc[e] * acc[e];
    if (row < na && col < na)
      s_aa += twice * x2;
    else if (row >= na && col >= na)
      s_vv += twice * x2;
    else if (row < na)  // audio row, visual column; its transpose is not counted
      s_av += x2;
  }
  s_aa = wave_sum(s_aa);
  s_av = wave_sum(s_av);
  s_vv = wave_sum(s_vv);
  if (lane == 0) {
    out[0] = s_aa;
    out[1] = s_av;
    out[2] = s_vv;
  }
}

// c_f = S_av / (sqrt(S_aa) sqrt(S_vv)) from the tile sums, in tile order;
// 0 when a side is degenerate: its centred Gram norm sqrt(S) at most
// kCkaDegenerate of its raw trace (the sum of its tokens' squared norms).
__global__ __launch_bounds__(kBlk) void k_spatial_reduce(const ClipDev* __restrict__ clips,
                                                         const FrameDev* __restrict__ frames, int64_t n_frames,
                                                         int tiles, const double* __restrict__ part,
                                                         const double* __restrict__ nv, const double* __restrict__ na,
                                                         double* __restrict__ cka) {
  const int64_t f = (int64_t)blockIdx.x * kBlk + threadIdx.x;
  if (f >= n_frames) return;
  double s_aa = 0.0, s_av = 0.0, s_vv = 0.0;
  for (int t = 0; t < tiles; ++t) {
    const double* q = part + (f * tiles + t) * 3;
    s_aa += q[0];
    s_av += q[1];
    s_vv += q[2];
  }
  const FrameDev fr = frames[f];
  const ClipDev c = clips[fr.clip];
  const int64_t lo = ((int64_t)fr.f * c.n_audio) / c.n_frames;
  const int64_t hi = (((int64_t)fr.f + 1) * c.n_audio + c.n_frames - 1) / c.n_frames;
  double tr_a = 0.0, tr_v = 0.0;
  for (int64_t r = lo; r < hi; ++r) tr_a += na[c.aud_off + r];
  const int64_t row0 = c.vis_off + (int64_t)fr.f * c.per_frame;
  for (int p = 0; p < c.per_frame; ++p) tr_v += nv[row0 + p];
  const double sa = sqrt(s_aa), sv = sqrt(s_vv);
  cka[f] = (sa <= kCkaDegenerate * tr_a || sv <= kCkaDegenerate * tr_v) ? 0.0 : s_av / (sa * sv);
}

// v_max_f64 / v_min_f64 as single instructions.  In IEEE mode the
// compiler quiets possible signalling NaNs before fmax / fmin with an extra
// max of each operand with itself; no value here is a signalling NaN
// (every one comes from arithmetic or from the Gram), and a quiet NaN
// operand gives the other one, as fmax / fmin do.
__device__ __forceinline__ double max_f64(double a, double b) {
  double r;
  asm("v_max_f64 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
__device__ __forceinline__ double min_f64(double a, double b) {
  double r;
  asm("v_min_f64 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}

// Unsigned key with the numeric order of doubles: positive values (sign bit
// clear) get the sign bit set, negative ones are negated as 64-bit integers,
// so the larger magnitude gives the smaller key and -0 gets the key of +0.
// Equal values have equal keys; every key is above 0 except those of
// negative NaNs.
__device__ __forceinline__ uint64_t order_key(double v) {
  const uint64_t b = (uint64_t)__double_as_longlong(v);
  return (b >> 63) ? (uint64_t)0 - b : (b | 0x8000000000000000ull);
}

// Maximum of a 32-bit value over the 64 lanes, in every lane: DPP within
// 16-lane rows, then the row-pair and half swaps.  All lanes active.
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, true));   // quad_perm [1,0,3,2]
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, true));   // quad_perm [2,3,0,1]
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, true));  // row_half_mirror
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xF, 0xF, true));  // row_mirror
  const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  v = max((uint32_t)r[0], (uint32_t)r[1]);
  const auto h = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return max((uint32_t)h[0], (uint32_t)h[1]);
}

// Cosine of tokens i and j of an anchor frame from their Gram entry g, the
// Gram's diagonal entries d (squared norms, summed like every entry) and
// r = 1 / sqrt(d): exactly 1 when g equals both diagonal entries and is not
// 0, which is also exactly what g / sqrt(d_i d_j) gives there (a token and a
// bitwise copy of it); otherwise g (r_i r_j), within a few ulps of that
// quotient and symmetric in i and j; 0 for a zero-norm token (r = 0).  The
// three tests are combined without branches.
__device__ __forceinline__ double cos_gram(double g, double di, double ri, double dj, double rj) {
  const double c = g * (ri * rj);
  const bool one = (g == di) & (g == dj) & (g != 0.0);
  return one ? 1.0 : c;
}

// Running list of the KM largest values, sorted descending: a new value is
// carried down past the larger entries (static indices, all in registers).
template <int KM>
__device__ __forceinline__ void top_insert(double (&top)[KM], double v) {
#pragma unroll
  for (int q = 0; q < KM; ++q) {
    const double hi = max_f64(top[q], v);
    v = min_f64(top[q], v);
    top[q] = hi;
  }
}

// LDS of k_dafps, in doubles (160 KiB).
constexpr int kDafpsLds = 20480;

struct DafpsLds {
  double* rows;    // rows [0, R) of the frame's cosine matrix, P apart
  double* corner;  // entries (j, t), j and t in [R, P): (P - R)^2 of them
  double2* nrm;    // (d, r) per token
  double* rho;     // densities
  int R;
  bool has_corner;
};

// Density of token i: the mean of its dafps_k largest cosines to the other
// tokens of the frame, times one plus the number of those cosines at or
// above the coverage threshold.  Two lanes of a wave (2i and 2i + 1) share
// token i, each walking its own rows [lo, hi) of column i of the Gram (S is
// exactly symmetric: entries (i, j) and (j, i) are the same products summed
// in the same order); each entry becomes a cosine, written back over the
// Gram entry in LDS (rows below R) or into the corner block (rows and token
// at or past R), so that the pick loop reads cosines.  Rows at or past R
// come from the Gram in global memory, the first eight of a lane's share
// prefetched into `pre` before the rows were staged.  Reads are issued
// eight rows at a time; ns and ng bound, for every lane of the wave, the
// staged and global row counts.  The two halves' lists and counts are then
// merged across the lane pair.  KM >= min(dafps_k, P - 1): only the first
// min(dafps_k, P - 1) entries of the merged list enter the mean.  Every
// lane of the wave must take part (lanes of tokens past P with empty
// ranges).
template <int KM>
__device__ __forceinline__ double dafps_density(const DafpsLds& L, const double* __restrict__ S, int P, int i,
                                                int lo, int hi, int ns, int ng, const double (&pre)[8], double di,
                                                double ri, int k, double cover) {
  double top[KM];
#pragma unroll
  for (int q = 0; q < KM; ++q) top[q] = -INFINITY;
  int cov = 0;
  const int R = L.R, ic = min(i, P - 1);
  const int s_end = min(hi, R), g_lo = max(lo, R);
  auto take = [&](bool valid, int j, double c) {
    const bool use = valid & (j != i);
    cov += (int)(use & (c >= cover));
    top_insert(top, use ? c : -INFINITY);
  };
  for (int jj = 0; jj < ns; jj += 8) {
    double g[8];
    double2 nj[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int j = min(lo + jj + u, R - 1);
      g[u] = L.rows[j * P + ic];
      nj[u] = L.nrm[j];
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int j = lo + jj + u;
      const bool valid = j < s_end;
      const double c = cos_gram(g[u], di, ri, nj[u].x, nj[u].y);
      if (valid) L.rows[j * P + i] = c;
      take(valid, j, c);
    }
  }
  auto tail = [&](int j0, const double (&g)[8]) {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int j = j0 + u;
      const bool valid = j < hi;
      const double2 nj = L.nrm[min(j, P - 1)];
      const double c = cos_gram(g[u], di, ri, nj.x, nj.y);
      if (valid && L.has_corner && i >= R) L.corner[(j - R) * (P - R) + (i - R)] = c;
      take(valid, j, c);
    }
  };
  if (ng > 0) tail(g_lo, pre);
  for (int jj = 8; jj < ng; jj += 8) {
    double g[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) g[u] = S[(int64_t)min(g_lo + jj + u, P - 1) * P + ic];
    tail(g_lo + jj, g);
  }
  // Merge with the partner lane's list and count.
  double o[KM];
#pragma unroll
  for (int q = 0; q < KM; ++q) o[q] = dpp_f64<0xB1>(top[q]);
#pragma unroll
  for (int q = 0; q < KM; ++q) top_insert(top, o[q]);
  cov += __builtin_amdgcn_update_dpp(cov, cov, 0xB1, 0xF, 0xF, false);
  const int nt = min(k, P - 1);
  double knn = 0.0;
#pragma unroll
  for (int q = 0; q < KM; ++q)
    if (q < nt) knn += top[q];
  knn = nt > 0 ? knn / nt : 0.0;
  return fmax(knn, 0.0) * (1.0 + cov);
}

// DA-FPS picks in one wave: token t = lane + 64 u, u < KU; tc is t clamped
// into the frame (addresses of lanes past the end stay in bounds; those
// tokens count as taken).  The first pick is the densest token, each later
// one the token farthest from the picked set, weighted by density:
// argmax of (1 - max cosine to the picked set) rho^power.  The argmax is
// lexicographic (value desc, token asc): the wave's largest order key, then
// the lowest token holding it -- tokens 64u + lane ascend with u and then
// with the lane, so the first non-empty ballot in u order names it.  Taken
// tokens have key 0, below every value's key except a negative NaN's; should
// no untaken token reach the maximum key (negative NaNs only), the lowest
// untaken token is taken, so a pick is always valid.  The picked positions
// go to kept[out...] in ascending order, as rows base + t.
template <int KU>
__device__ __forceinline__ void dafps_pick(const DafpsLds& L, const double* __restrict__ S, int P, int k,
                                           double power, int lane, int32_t* __restrict__ kept, int64_t out,
                                           int64_t base) {
  const int R = L.R;
  double wgt[KU], smax[KU], dt[KU], rt[KU];
  uint64_t key[KU];
  // Taken tokens as wave-wide lane masks (the same in every lane), one per
  // u; tokens past P count as taken.
  uint64_t tk[KU], pad[KU];
  int tc[KU];
#pragma unroll
  for (int u = 0; u < KU; ++u) {
    const int t = lane + 64 * u;
    pad[u] = tk[u] = __ballot(t >= P);
    const bool tkn = t >= P;
    tc[u] = min(t, P - 1);
    const double rho = L.rho[tc[u]];
    wgt[u] = tkn ? 0.0 : pow(rho, power);
    key[u] = tkn ? 0 : order_key(rho);
    smax[u] = -INFINITY;
    const double2 n = L.nrm[tc[u]];
    dt[u] = n.x;
    rt[u] = n.y;
  }
  auto pick_of = [&]() {
    uint64_t kb = key[0];
#pragma unroll
    for (int u = 1; u < KU; ++u) kb = key[u] > kb ? key[u] : kb;
    const uint32_t mh = wave_max_u32((uint32_t)(kb >> 32));
    // Untaken tokens whose key has the maximal high word: when there is
    // one (the usual case) it is the pick, and the low words need no
    // reduction.
    uint64_t hb[KU];
    int cnt = 0;
#pragma unroll
    for (int u = 0; u < KU; ++u) {
      hb[u] = __ballot((uint32_t)(key[u] >> 32) == mh) & ~tk[u];
      cnt += __popcll(hb[u]);
    }
    int best = 0x7FFFFFFF;
    if (cnt == 1) {
#pragma unroll
      for (int u = 0; u < KU; ++u)
        if (hb[u]) best = 64 * u + (int)__builtin_ctzll(hb[u]);
      return best;
    }
    if (cnt > 1) {
      const uint32_t ml = wave_max_u32((uint32_t)(kb >> 32) == mh ? (uint32_t)kb : 0u);
      const uint64_t mk = ((uint64_t)mh << 32) | ml;
#pragma unroll
      for (int u = 0; u < KU; ++u) {
        const uint64_t b = __ballot(key[u] == mk) & ~tk[u];
        if (b && best == 0x7FFFFFFF) best = 64 * u + (int)__builtin_ctzll(b);
      }
    }
    if (best == 0x7FFFFFFF) {
#pragma unroll
      for (int u = 0; u < KU; ++u) {
        const uint64_t b = ~tk[u];
        if (b && best == 0x7FFFFFFF) best = 64 * u + (int)__builtin_ctzll(b);
      }
    }
    return best;
  };
  int pick = pick_of();
  for (int n = 0;; ++n) {
    double sv[KU];
    if (pick < R) {  // the same branch for the whole wave
#pragma unroll
      for (int u = 0; u < KU; ++u) sv[u] = L.rows[pick * P + tc[u]];
    } else {
      const double2 np = L.nrm[pick];
#pragma unroll
      for (int u = 0; u < KU; ++u) {
        if (tc[u] < R)
          sv[u] = L.rows[tc[u] * P + pick];
        else if (L.has_corner)
          sv[u] = L.corner[(pick - R) * (P - R) + (tc[u] - R)];
        else
          sv[u] = cos_gram(S[(int64_t)pick * P + tc[u]], np.x, np.y, dt[u], rt[u]);
      }
    }
#pragma unroll
    for (int u = 0; u < KU; ++u) {
      if ((pick >> 6) == u) tk[u] |= 1ull << (pick & 63);
      smax[u] = max_f64(smax[u], sv[u]);
    }
    if (n + 1 >= k) break;
#pragma unroll
    for (int u = 0; u < KU; ++u)
      key[u] = order_key((1.0 - smax[u]) * wgt[u]) & (__builtin_amdgcn_inverse_ballot_w64(tk[u]) ? 0ull : ~0ull);
    pick = pick_of();
  }
  // Ascending output of the picked positions.
#pragma unroll
  for (int u = 0; u < KU; ++u) {
    const uint64_t bal = tk[u] & ~pad[u];
    if ((bal >> lane) & 1ull) kept[out + __popcll(bal & ((1ull << lane) - 1ull))] = (int32_t)(base + lane + 64 * u);
    out += __popcll(bal);
  }
}

// ---------------------------------------------------------------------------
// DA-FPS on an anchor frame: one workgroup, two threads per token.
// ---------------------------------------------------------------------------
// The frame's raw Gram rows [0, R) go to LDS by direct loads; R is the
// largest row count for which those rows, the (P - R) x (P - R) corner block
// and the per-token arrays fit in 160 KiB (R = P up to P = 141, 139 rows of
// 144), else as many rows as fit without the corner.  The density pass
// (threads 2i and 2i + 1 on token i, rows split at (P + 1) / 2) turns every
// entry into a cosine (cos_gram).  The pick loop then runs in one wave,
// which holds up to four tokens per lane and finds each pick from order
// keys reduced by DPP (dafps_pick); a pick reads one cosine row from LDS:
// row `pick` itself when pick < R, else column `pick` of the staged rows
// (the same values, by symmetry) and the corner block -- or, when the
// corner did not fit, the Gram row in global memory, turned into cosines as
// it is read.
constexpr int kDafpsThreads = 2 * kMaxPerFrame;

__global__ __launch_bounds__(kDafpsThreads) void k_dafps(const ClipDev* __restrict__ clips,
                                                         const FrameDev* __restrict__ frames,
                                                         const FramePlanDev* __restrict__ plan, DynParamsDev prm,
                                                         const double* __restrict__ gram, int32_t* __restrict__ kept) {
  __shared__ __attribute__((aligned(16))) double lds[kDafpsLds];
  const FrameDev fr = frames[blockIdx.x];
  const ClipDev c = clips[fr.clip];
  const int64_t frame = c.frame_off + fr.f;
  const FramePlanDev fp = plan[frame];
  if (!fp.is_anchor || fp.budget == 0) return;
  const int P = c.per_frame, tid = threadIdx.x, i = tid >> 1, h = tid & 1;
  const int k = min(fp.budget, P);
  const double* S = gram + c.gram_off + (int64_t)fr.f * P * P;

  // LDS layout: the per-token arrays take 3 P doubles plus one of padding
  // (the (d, r) pairs are 16-byte aligned).
  const int fixed = 3 * P + 2;
  int R = P;
  while (R > P / 2 && R * P + (P - R) * (P - R) + fixed > kDafpsLds) --R;
  const bool has_corner = R * P + (P - R) * (P - R) + fixed <= kDafpsLds;
  if (!has_corner) R = min(P, (kDafpsLds - fixed) / P);
  DafpsLds L;
  L.R = R;
  L.rows = lds;
  L.has_corner = has_corner;
  L.corner = lds + R * P;
  const int nrm_off = (R * P + (has_corner ? (P - R) * (P - R) : 0) + 1) & ~1;
  L.nrm = reinterpret_cast<double2*>(lds + nrm_off);
  L.rho = lds + nrm_off + 2 * P;

  // Each thread's rows of column i: [0, Hs) or [Hs, P); ns and ng bound the
  // staged and global counts of either half (the same for every wave).
  const int Hs = (P + 1) / 2;
  const int lo = i < P ? (h ? Hs : 0) : 0, hi = i < P ? (h ? P : Hs) : 0;
  const int ns = max(min(Hs, R), max(min(P, R) - Hs, 0));
  const int ng = max(Hs - min(Hs, R), P - max(Hs, R));

  // Global reads first (diagonal entry, the first eight global rows of the
  // thread's share of column i), then the staged rows; all in flight
  // together.
  double di = 0.0, pre[8];
#pragma unroll
  for (int u = 0; u < 8; ++u) pre[u] = 0.0;
  if (i < P) {
    di = S[(int64_t)i * P + i];
    const int g_lo = max(lo, R);
    if (g_lo < hi) {
#pragma unroll
      for (int u = 0; u < 8; ++u) pre[u] = S[(int64_t)min(g_lo + u, P - 1) * P + i];
    }
  }
  if (((uintptr_t)S & 15) == 0 && (R * P) % 2 == 0) {
    // 16-byte direct-to-LDS loads: wave load j fills bytes [1024 j, 1024 j +
    // 1024), lane l the 16 bytes at 1024 j + 16 l (lanes past the end stay
    // idle; the byte count is a multiple of 16).
    typedef __attribute__((address_space(3))) void* lds_ptr_t;
    typedef __attribute__((address_space(1))) void* glb_ptr_t;
    const int bytes = R * P * 8;
    const int lane = tid & 63, wave = tid >> 6;
    for (int j = wave; j * 1024 < bytes; j += kDafpsThreads / 64) {
      const int off = j * 1024 + lane * 16;
      if (off < bytes)
        __builtin_amdgcn_global_load_lds((glb_ptr_t)(reinterpret_cast<const char*>(S) + off),
                                         (lds_ptr_t)(reinterpret_cast<char*>(lds) + j * 1024), 16, 0, 0);
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  } else {
    // S only 8-byte aligned (odd P * P before it) or an odd element count:
    // eight loads in flight per thread.
    for (int e0 = tid; e0 < R * P; e0 += 8 * kDafpsThreads) {
      double v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int e = e0 + u * kDafpsThreads;
        v[u] = e < R * P ? S[e] : 0.0;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int e = e0 + u * kDafpsThreads;
        if (e < R * P) lds[e] = v[u];
      }
    }
  }
  const double ri = di > 0.0 ? 1.0 / sqrt(di) : 0.0;
  if (i < P && h == 0) L.nrm[i] = make_double2(di, ri);
  __syncthreads();

  // Density of every token; the list length is the exact dafps_k up to 8.
  // Waves whose tokens all lie past P skip it (the test is the same for the
  // whole wave, so every lane of a working wave takes part).
  if (32 * (tid >> 6) < P) {
    const int dk = prm.dafps_k;
    const double cv = prm.cover;
    double rho;
    switch (dk) {
      case 1: rho = dafps_density<1>(L, S, P, i, lo, hi, ns, ng, pre, di, ri, dk, cv); break;
      case 2: rho = dafps_density<2>(L, S, P, i, lo, hi, ns, ng, pre, di, ri, dk, cv); break;
      case 3: rho = dafps_density<3>(L, S, P, i, lo, hi, ns, ng, pre, di, ri, dk, cv); break;
      case 4: rho = dafps_density<4>(L, S, P, i, lo, hi, ns, ng, pre, di, ri, dk, cv); break;
      case 5: rho = dafps_density<5>(L, S, P, i, lo, hi, ns, ng, pre, di, ri, dk, cv); break;
      case 6: rho = dafps_density<6>(L, S, P, i, lo, hi, ns, ng, pre, di, ri, dk, cv); break;
      case 7: rho = dafps_density<7>(L, S, P, i, lo, hi, ns, ng, pre, di, ri, dk, cv); break;
      case 8: rho = dafps_density<8>(L, S, P, i, lo, hi, ns, ng, pre, di, ri, dk, cv); break;
      default:
        rho = dk <= 16 ? dafps_density<16>(L, S, P, i, lo, hi, ns, ng, pre, di, ri, dk, cv)
                       : dafps_density<32>(L, S, P, i, lo, hi, ns, ng, pre, di, ri, dk, cv);
    }
    if (i < P && h == 0) L.rho[i] = rho;
  }
  __syncthreads();
  if (tid >= 64) return;

  // Wave 0 picks; lanes hold ceil(P / 64) tokens each.
  const int nu = (P + 63) / 64;
  int64_t out = fp.out_off;
  const int64_t base = c.vis_off + (int64_t)fr.f * P;
  if (nu == 1) dafps_pick<1>(L, S, P, k, prm.power, tid, kept, out, base);
  else if (nu == 2) dafps_pick<2>(L, S, P, k, prm.power, tid, kept, out, base);
  else if (nu == 3) dafps_pick<3>(L, S, P, k, prm.power, tid, kept, out, base);
  else dafps_pick<4>(L, S, P, k, prm.power, tid, kept, out, base);
}

// ---------------------------------------------------------------------------
// Non-anchor frames: keep the k_f positions least similar to the anchor
// token at the same position (lower position first on ties).
// ---------------------------------------------------------------------------
template <class T>
__global__ __launch_bounds__(kBlk) void k_dedup_sim(const ClipDev* __restrict__ clips,
                                                    const FrameDev* __restrict__ frames,
                                                    const FramePlanDev* __restrict__ plan, int dim,
                                                    const T* __restrict__ xv, double* __restrict__ sim) {
  // One wave per position: cosine of token p of frame f with token p of its
  // anchor, written to sim at the token's row.  The dot product and both
  // squared norms are summed the same way, so a position that repeats the
  // anchor's token has cosine exactly 1.
  const FrameDev fr = frames[blockIdx.x];
  const ClipDev c = clips[fr.clip];
  const FramePlanDev fp = plan[c.frame_off + fr.f];
  if (fp.is_anchor || fp.budget == 0) return;
  const int P = c.per_frame;
  const int lane = threadIdx.x & 63;
  const int p = blockIdx.y * (kBlk / 64) + (threadIdx.x >> 6);
  if (p >= P) return;
  const int64_t rowf = c.vis_off + (int64_t)fr.f * P + p, rowa = c.vis_off + (int64_t)fp.anchor * P + p;
  const T* x = xv + rowf * dim;
  const T* y = xv + rowa * dim;
  double xy = 0.0, xx = 0.0, yy = 0.0, o[8], q[8];
#pragma unroll 4
  for (int d = lane * 8; d < dim; d += 64 * 8) {
    load8(x + d, o);
    load8(y + d, q);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      xy = fma(o[e], q[e], xy);
      xx = fma(o[e], o[e], xx);
      yy = fma(q[e], q[e], yy);
    }
  }
  xy = wave_sum(xy);
  xx = wave_sum(xx);
  yy = wave_sum(yy);
  if (lane == 0) sim[rowf - c.vis_off + c.token_off] = cos_from(xy, xx, yy);
}

__global__ __launch_bounds__(kBlk) void k_dedup_pick(const ClipDev* __restrict__ clips,
                                                     const FrameDev* __restrict__ frames,
                                                     const FramePlanDev* __restrict__ plan,
                                                     const double* __restrict__ simg, int32_t* __restrict__ kept) {
  // The k_f positions least similar to the anchor, lower position first on
  // ties, written in ascending order.
  __shared__ double sim[kMaxPerFrame];
  __shared__ int wcount[kBlk / 64];
  const FrameDev fr = frames[blockIdx.x];
  const ClipDev c = clips[fr.clip];
  const FramePlanDev fp = plan[c.frame_off + fr.f];
  if (fp.is_anchor || fp.budget == 0) return;
  const int P = c.per_frame;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t rowf = c.vis_off + (int64_t)fr.f * P;
  const double* sg = simg + c.token_off + (int64_t)fr.f * P;
  for (int q = threadIdx.x; q < P; q += kBlk) sim[q] = sg[q];
  __syncthreads();
  const int p = threadIdx.x;
  bool kp = false;
  if (p < P) {
    int rank = 0;
    for (int q = 0; q < P; ++q)
      if (sim[q] < sim[p] || (sim[q] == sim[p] && q < p)) ++rank;
    kp = rank < fp.budget;
  }
  const uint64_t bal = __ballot(kp);
  if (lane == 0) wcount[wave] = __popcll(bal);
  __syncthreads();
  int64_t pos = fp.out_off;
  for (int w = 0; w < wave; ++w) pos += wcount[w];
  if (kp) kept[pos + __popcll(bal & ((1ull << lane) - 1ull))] = (int32_t)(rowf + p);
}

template <class T>
apack_status launch_t(const DynPlan& pl, const DynPtrs& dp, const DynParamsDev& prm, int dim, const T* xv,
                      const T* xa, const T* xq, float* frame_cka, float* frame_score, int32_t* frame_budget,
                      int32_t* segment_id, uint8_t* gate_fired, int32_t* kept, int64_t visual_rows,
                      int64_t audio_rows, hipStream_t s) {
  apack_status st;
  const int nf = (int)pl.frames.size(), nc = (int)pl.clips.size();
  const unsigned dchunks = (unsigned)((dim + kPoolSlice - 1) / kPoolSlice);
  const int64_t n_vis = pl.total_tokens, n_aud = pl.total_audio;
  hipLaunchKernelGGL(k_pool<T>, dim3((unsigned)((nf + nc) * dchunks)), dim3(kBlk), 0, s, dp.clips, dp.frames,
                     (int64_t)nf, dim, (int)dchunks, xv, xa, xq, dp.v, dp.a, dp.q, n_vis, n_vis + n_aud, dp.sqp);
  if ((st = launch_status("k_pool")) != APACK_OK) return st;
  if (nf > 0) {
    // Partners per frame: max(w, 2) <= kMaxWindow (checked on the host).
    const int wb = std::max(prm.window, 2);
    // (Windows past 8 keep 256 threads: 1024 would leave too few registers for their sums.)
    const bool wide = nf < kBandWideFrames && wb <= 8;
    auto band = wide ? (wb <= 2 ? k_band<2, 1024> : wb <= 4 ? k_band<4, 1024> : k_band<8, 1024>)
                     : (wb <= 2 ? k_band<2, kBlk> : wb <= 4 ? k_band<4, kBlk> : wb <= 8 ? k_band<8, kBlk>
                                                                                      : k_band<kMaxWindow, kBlk>);
    hipLaunchKernelGGL(band, dim3(nf), dim3(wide ? 1024 : kBlk), 0, s, dp.clips, dp.frames, dim, prm.window, dp.v,
                       dp.a, dp.q, dp.band_v, dp.band_a, dp.vq, dp.qq);
    if ((st = launch_status("k_band")) != APACK_OK) return st;
  }
  if (n_vis + n_aud > 0) {
    hipLaunchKernelGGL(k_norms, dim3((unsigned)((n_vis + n_aud + kBlk - 1) / kBlk)), dim3(kBlk), 0, s, n_vis, n_aud,
                       (int)dchunks, dp.sqp, dp.nv, dp.rv, dp.na, dp.maxkey);
    if ((st = launch_status("k_norms")) != APACK_OK) return st;
  }
  if (prm.alignment == APACK_ALIGN_SPATIAL_CKA && nf > 0) {
    const unsigned gy = (unsigned)((pl.spatial_tiles + kGramWaves - 1) / kGramWaves);
    hipLaunchKernelGGL(k_spatial_gram<T>, dim3(nf, gy), dim3(kGramWaves * 64), 0, s, dp.clips, dp.frames, dim, xv,
                       xa, dp.v, dp.a, pl.spatial_tiles, dp.spatial);
    if ((st = launch_status("k_spatial_gram")) != APACK_OK) return st;
    hipLaunchKernelGGL(k_spatial_reduce, dim3((unsigned)((nf + kBlk - 1) / kBlk)), dim3(kBlk), 0, s, dp.clips,
                       dp.frames, (int64_t)nf, pl.spatial_tiles, dp.spatial, dp.nv, dp.na, dp.cka);
    if ((st = launch_status("k_spatial_reduce")) != APACK_OK) return st;
  }
  auto cka = prm.window <= 2 ? k_cka<2> : prm.window <= 4 ? k_cka<4> : prm.window <= 8 ? k_cka<8> : k_cka<kMaxWindow>;
  hipLaunchKernelGGL(cka, dim3(nc), dim3(kBlk), 0, s, dp.clips, prm.window, prm.tau_gate, prm.alignment, dp.band_v,
                     dp.band_a, dp.cka, frame_cka, gate_fired);
  if ((st = launch_status("k_cka")) != APACK_OK) return st;
  if (pl.gemm_tiles > 0) {
    if constexpr (std::is_same<T, bf16_t>::value) {
      if (pl.use256) {
        if ((st = launch_gate_gemm256(dp.clips, dp.gemm, pl.gemm_tiles, dim, xv, xa, dp.na, dp.maxkey, s)) !=
            APACK_OK)
          return st;
      }
    }
    if (!pl.use256) {
      hipLaunchKernelGGL(k_gate_gemm<T>, dim3((unsigned)pl.gemm_tiles), dim3(kBlk), 0, s, dp.clips, dp.gemm, dim,
                         xv, xa, dp.na, dp.maxkey);
      if ((st = launch_status("k_gate_gemm")) != APACK_OK) return st;
    }
  }
  hipLaunchKernelGGL(k_plan, dim3(nc), dim3(kPlanBlk), 0, s, dp.clips, prm, dp.cka, dp.band_v, dp.vq, dp.qq, dp.rv,
                     dp.maxkey, dp.plan, dp.anchors, dp.scratch, (int64_t)(pl.total_frames + nc), frame_score,
                     frame_budget,
                     segment_id);
  if ((st = launch_status("k_plan")) != APACK_OK) return st;
  if (nf > 0) {
    if (pl.gram_items > 0) {
      const unsigned gb = (unsigned)std::min<int64_t>((pl.gram_items + 7) / 8 * 8, kGramBlocks);
      hipLaunchKernelGGL(k_gram<T>, dim3(gb), dim3(kGramSplit * 64), 0, s, dp.clips, nc, dp.anchors, dp.plan, dim,
                         xv, dp.gram);
    }
    if ((st = launch_status("k_gram")) != APACK_OK) return st;
    hipLaunchKernelGGL(k_dafps, dim3(nf), dim3(kDafpsThreads), 0, s, dp.clips, dp.frames, dp.plan, prm, dp.gram, kept);
    if ((st = launch_status("k_dafps")) != APACK_OK) return st;
    hipLaunchKernelGGL(k_dedup_sim<T>, dim3(nf, (pl.max_per_frame + kBlk / 64 - 1) / (kBlk / 64)), dim3(kBlk), 0, s,
                       dp.clips, dp.frames, dp.plan, dim, xv, dp.sim);
    if ((st = launch_status("k_dedup_sim")) != APACK_OK) return st;
    hipLaunchKernelGGL(k_dedup_pick, dim3(nf), dim3(kBlk), 0, s, dp.clips, dp.frames, dp.plan, dp.sim, kept);
    if ((st = launch_status("k_dedup_pick")) != APACK_OK) return st;
  }
  return APACK_OK;
}

}  // namespace

apack_status launch_dynamics(const DynPlan& pl, const DynPtrs& dp, const DynParamsDev& prm, apack_dtype dt, int dim,
                             const void* visual, const void* audio, const void* query, int64_t visual_rows,
                             int64_t audio_rows, float* frame_cka, float* frame_score, int32_t* frame_budget,
                             int32_t* segment_id, uint8_t* gate_fired, int32_t* kept, hipStream_t stream) {
  if (dt == APACK_BF16)
    return launch_t<bf16_t>(pl, dp, prm, dim, (const bf16_t*)visual, (const bf16_t*)audio, (const bf16_t*)query,
                            frame_cka, frame_score, frame_budget, segment_id, gate_fired, kept, visual_rows,
                            audio_rows, stream);
  return launch_t<float>(pl, dp, prm, dim, (const float*)visual, (const float*)audio, (const float*)query, frame_cka,
                         frame_score, frame_budget, segment_id, gate_fired, kept, visual_rows, audio_rows, stream);
}

}  // namespace apack
