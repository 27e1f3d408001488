// Per-modality top-k (Eq. 6 within each modality) and the ordered list of
// kept rows, spread over the whole GPU.
//
// Scores are non-negative fp32, so their bit patterns order like the
// values.  The k-th largest bit pattern T of each (sequence, modality) is
// found digit by digit: bits 30..20, then 19..9, then 8..0.  Each pass is one
// launch over row tiles of 1024 rows; a tile counts its rows' digits in LDS
// (rows whose higher digits match the prefix chosen so far) and adds the
// non-zero bins to a global histogram.  The last tile of a sequence to finish
// (a fenced atomic counter) picks the bin holding the k-th value, records it,
// clears the histogram and resets the counter for the next pass.
//
// Kept rows: every non-candidate row, every row above T, and the first
// (k - count_above) rows equal to T in row order (the lower row wins ties).
// A count kernel records each tile's (sure keeps, ties per modality); a
// write kernel adds up the tiles before it and places its rows with block
// scans.  No kernel waits on another workgroup.
#include <cfloat>

#include "common.hpp"
#include "prune_plan.hpp"

namespace apack {
namespace {

constexpr int kT = 256;              // threads per row tile
constexpr int kPer = kRowTile / kT;  // rows per thread (contiguous)
constexpr int kBins1 = 2048;

__device__ __forceinline__ uint32_t clamp_bits(float s) {
  return min(__float_as_uint(s), 0x7F800000u);
}

__device__ __forceinline__ uint32_t ld_agent(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Inclusive scan over the block (kT threads).
__device__ __forceinline__ uint32_t block_scan(uint32_t v, uint32_t* sh, uint32_t& total) {
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
  for (int w = 0; w < kT / 64; ++w) {
    const uint32_t x = sh[w];
    if (w < wave) base += x;
    total += x;
  }
  __syncthreads();
  return v + base;
}

// Digit of pass p and whether the row takes part (its higher digits match).
__device__ __forceinline__ bool digit_of(uint32_t bits, int pass, uint32_t prefix, uint32_t& d) {
  if (pass == 0) {
    d = bits >> 20;
    return true;
  }
  if (pass == 1) {
    d = (bits >> 9) & 0x7FFu;
    return (bits >> 20) == prefix;
  }
  d = bits & 0x1FFu;
  return (bits >> 9) == prefix;
}

// The last tile of a sequence picks the bin that holds the kk-th largest
// value, for each modality still selecting.
__device__ void pick_bins(SeqDev* sq, uint32_t* hist, int pass) {
  __shared__ uint32_t sh[kT / 64];
  const int tid = threadIdx.x;
  const int nb = pass == 2 ? 512 : kBins1;
  for (int m = 0; m < 2; ++m) {
    if (!sq->select[m]) continue;
    uint32_t* h = hist + m * kBins1;
    // Thread t holds 8 consecutive bins from the top: 2047-8t ... 2040-8t.
    uint32_t c[8], sum = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int b = nb - 1 - (tid * 8 + j);
      c[j] = b >= 0 ? ld_agent(h + b) : 0u;
      sum += c[j];
    }
    uint32_t total;
    const uint32_t incl = block_scan(sum, sh, total);
    uint32_t before = incl - sum;
    const uint32_t kk = sq->kk[m];
    if (before < kk && incl >= kk) {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        if (before < kk && before + c[j] >= kk) {
          const uint32_t b = (uint32_t)(nb - 1 - (tid * 8 + j));
          const uint32_t prefix = pass == 0 ? b : (sq->prefix[m] << (pass == 1 ? 11 : 9)) | b;
          sq->prefix[m] = prefix;
          sq->kk[m] = kk - before;
          if (pass == 2) {
            sq->thr[m] = prefix;
            sq->need[m] = (int32_t)(kk - before);
            sq->all_eq[m] = (kk - before == c[j]) ? 1 : 0;
          }
        }
        before += c[j];
      }
    }
    __syncthreads();
    for (int b = tid; b < kBins1; b += kT) h[b] = 0;
  }
}

// Counts the tile's participating digits and merges them into the global
// histogram; the last tile of the sequence picks the bins.
__device__ void hist_pass(SeqDev* sq, uint32_t* hist, const uint8_t* tg, const uint32_t (&bits)[kPer],
                          const uint8_t (&mt)[kPer], int pass, uint32_t* lh) {
  const int tid = threadIdx.x;
  const uint32_t pre[2] = {sq->prefix[0], sq->prefix[1]};
  const bool act[2] = {sq->select[0] != 0, sq->select[1] != 0};
  for (int b = tid; b < 2 * kBins1; b += kT) lh[b] = 0;
  __syncthreads();
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int m = mt[u] - 1;
    if (m < 0 || m > 1 || !act[m]) continue;
    uint32_t d;
    if (digit_of(bits[u], pass, pre[m], d)) atomicAdd(&lh[m * kBins1 + d], 1u);
  }
  __syncthreads();
  for (int b = tid; b < 2 * kBins1; b += kT) {
    const uint32_t v = lh[b];
    if (v) atomicAdd(&hist[b], v);
  }
  __threadfence();
  __syncthreads();
  __shared__ bool last;
  if (tid == 0) {
    const uint32_t prev = atomicAdd(&sq->done_cnt, 1u);
    last = prev == (uint32_t)sq->n_ftiles - 1;
  }
  __syncthreads();
  if (!last) return;
  __threadfence();
  pick_bins(sq, hist, pass);
  if (tid == 0) sq->done_cnt = 0;
}

__device__ __forceinline__ void tile_rows(const FTileDev& ft, const SeqDev& sq, int64_t& r0, int& n) {
  r0 = (int64_t)ft.idx * kRowTile;
  const int64_t left = sq.n_tokens - r0;
  n = left < kRowTile ? (int)left : kRowTile;
}

// ---------------------------------------------------------------------------
// I_j = (sum over groups, fixed order) / (Hq * T), 0 for non-candidates,
// followed by the first histogram pass.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kT) void k_finalize_hist(SeqDev* __restrict__ seqs, const FTileDev* __restrict__ ftiles,
                                                      const uint8_t* __restrict__ tags,
                                                      const float* __restrict__ colpart, int hq, int hkv,
                                                      float* __restrict__ scores, uint32_t* __restrict__ hist) {
  __shared__ uint32_t lh[2 * kBins1];
  const FTileDev ft = ftiles[blockIdx.x];
  SeqDev* sq = &seqs[ft.seq];
  int64_t r0;
  int n;
  tile_rows(ft, *sq, r0, n);
  const uint8_t* tg = tags + sq->tag_off;
  const int planes = hkv * sq->n_rg;
  const float denom = (float)(hq * sq->q_len);
  uint32_t bits[kPer];
  uint8_t mt[kPer];
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int i = threadIdx.x * kPer + u;
    const int64_t j = r0 + i;
    float v = 0.f;
    uint8_t m = 0xFF;
    if (i < n) {
      m = tg[j];
      if (m != 0 && sq->n_cand > 0) {
        const float* p = colpart + sq->colpart_off + j;
        float acc = 0.f;
        for (int pl = 0; pl < planes; ++pl) acc += p[(int64_t)pl * sq->n_tokens];
        v = acc / denom;
      }
      scores[sq->tok_off + j] = v;
    }
    bits[u] = clamp_bits(v);
    mt[u] = m;
  }
  if (sq->select[0] || sq->select[1]) hist_pass(sq, hist + (int64_t)ft.seq * 2 * kBins1, tg, bits, mt, 0, lh);
}

__global__ __launch_bounds__(kT) void k_select_pass(SeqDev* __restrict__ seqs, const FTileDev* __restrict__ ftiles,
                                                    const uint8_t* __restrict__ tags,
                                                    const float* __restrict__ scores, uint32_t* __restrict__ hist,
                                                    int pass) {
  __shared__ uint32_t lh[2 * kBins1];
  const FTileDev ft = ftiles[blockIdx.x];
  SeqDev* sq = &seqs[ft.seq];
  if (!(sq->select[0] || sq->select[1])) return;
  int64_t r0;
  int n;
  tile_rows(ft, *sq, r0, n);
  const uint8_t* tg = tags + sq->tag_off;
  uint32_t bits[kPer];
  uint8_t mt[kPer];
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int i = threadIdx.x * kPer + u;
    bits[u] = 0;
    mt[u] = 0xFF;
    if (i < n) {
      mt[u] = tg[r0 + i];
      bits[u] = clamp_bits(scores[sq->tok_off + r0 + i]);
    }
  }
  hist_pass(sq, hist + (int64_t)ft.seq * 2 * kBins1, tg, bits, mt, pass, lh);
}

// Per tile: (rows kept for sure, rows equal to T_audio, rows equal to T_visual).
__global__ __launch_bounds__(kT) void k_keep_count(const SeqDev* __restrict__ seqs,
                                                   const FTileDev* __restrict__ ftiles,
                                                   const uint8_t* __restrict__ tags,
                                                   const float* __restrict__ scores, uint32_t* __restrict__ cnt) {
  __shared__ uint32_t sh[kT / 64];
  const FTileDev ft = ftiles[blockIdx.x];
  const SeqDev& sq = seqs[ft.seq];
  int64_t r0;
  int n;
  tile_rows(ft, sq, r0, n);
  const uint8_t* tg = tags + sq.tag_off;
  uint32_t sure = 0, ea = 0, ev = 0;
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int i = threadIdx.x * kPer + u;
    if (i >= n) continue;
    const uint8_t m = tg[r0 + i];
    if (m == 0) {
      ++sure;
      continue;
    }
    const uint32_t b = clamp_bits(scores[sq.tok_off + r0 + i]);
    const uint32_t t = sq.thr[m - 1];
    if (b > t) ++sure;
    else if (b == t) (m == 1 ? ea : ev) += 1;
  }
  uint32_t tot;
  block_scan(sure, sh, tot);
  const uint32_t s_tot = tot;
  block_scan(ea | (ev << 16), sh, tot);
  if (threadIdx.x == 0) {
    cnt[3 * (int64_t)blockIdx.x + 0] = s_tot;
    cnt[3 * (int64_t)blockIdx.x + 1] = tot & 0xFFFFu;
    cnt[3 * (int64_t)blockIdx.x + 2] = tot >> 16;
  }
}

__global__ __launch_bounds__(kT) void k_keep_write(const SeqDev* __restrict__ seqs,
                                                   const FTileDev* __restrict__ ftiles,
                                                   const uint8_t* __restrict__ tags,
                                                   const float* __restrict__ scores,
                                                   const uint32_t* __restrict__ cnt, int32_t* __restrict__ kept) {
  __shared__ uint32_t sh[kT / 64];
  __shared__ uint64_t base_sh[3];
  const FTileDev ft = ftiles[blockIdx.x];
  const SeqDev& sq = seqs[ft.seq];
  int64_t r0;
  int n;
  tile_rows(ft, sq, r0, n);
  const uint8_t* tg = tags + sq.tag_off;
  const uint32_t need[2] = {(uint32_t)sq.need[0], (uint32_t)sq.need[1]};
  // Rows kept and ties seen by the tiles before this one.  The ties kept
  // before a tile add up to min(need, ties before it), so plain sums do.
  {
    uint32_t s = 0, a = 0, v = 0;
    const int64_t first = (int64_t)blockIdx.x - ft.idx;
    for (int64_t w = first + threadIdx.x; w < (int64_t)blockIdx.x; w += kT) {
      s += cnt[3 * w];
      a += cnt[3 * w + 1];
      v += cnt[3 * w + 2];
    }
    uint32_t ts, ta, tv;
    block_scan(s, sh, ts);
    block_scan(a, sh, ta);
    block_scan(v, sh, tv);
    if (threadIdx.x == 0) {
      base_sh[0] = (uint64_t)ts + min(ta, need[0]) + min(tv, need[1]);
      base_sh[1] = ta;
      base_sh[2] = tv;
    }
  }
  __syncthreads();
  uint32_t bits[kPer];
  uint8_t mt[kPer];
  uint32_t ea = 0, ev = 0;
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int i = threadIdx.x * kPer + u;
    mt[u] = 0xFF;
    bits[u] = 0;
    if (i < n) {
      mt[u] = tg[r0 + i];
      if (mt[u] != 0) bits[u] = clamp_bits(scores[sq.tok_off + r0 + i]);
    }
    if (mt[u] == 1 && bits[u] == sq.thr[0]) ++ea;
    if (mt[u] == 2 && bits[u] == sq.thr[1]) ++ev;
  }
  uint32_t tot;
  const uint32_t packed = ea | (ev << 16);
  const uint32_t ex = block_scan(packed, sh, tot) - packed;
  uint64_t rank_a = base_sh[1] + (ex & 0xFFFFu), rank_v = base_sh[2] + (ex >> 16);
  bool keep[kPer];
  uint32_t nk = 0;
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const uint8_t m = mt[u];
    bool kp = false;
    if (m == 0) kp = true;
    else if (m == 1 || m == 2) {
      const uint32_t t = sq.thr[m - 1];
      if (bits[u] > t) kp = true;
      else if (bits[u] == t) kp = (m == 1 ? rank_a++ : rank_v++) < need[m - 1];
    }
    keep[u] = kp;
    nk += kp;
  }
  const uint64_t pos0 = base_sh[0] + (block_scan(nk, sh, tot) - nk);
  int32_t* out = kept + sq.out_off;
  uint64_t pos = pos0;
#pragma unroll
  for (int u = 0; u < kPer; ++u)
    if (keep[u]) {
      if (pos < (uint64_t)sq.n_kept) out[pos] = (int32_t)(sq.tok_off + r0 + threadIdx.x * kPer + u);
      ++pos;
    }
}

__global__ __launch_bounds__(256) void k_zero(uint32_t* __restrict__ p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0;
}

}  // namespace

apack_status launch_select(const PrunePlan& pl, const DevPtrs& dp, int hq, int hkv, float* scores, int32_t* kept,
                           hipStream_t stream) {
  const int nf = (int)pl.ftiles.size();
  if (nf == 0) return APACK_OK;
  apack_status st;
  if (pl.any_select) {
    const int64_t words = (int64_t)pl.seqs.size() * 2 * kBins1;
    hipLaunchKernelGGL(k_zero, dim3((unsigned)std::min<int64_t>((words + 255) / 256, 1024)), dim3(256), 0, stream,
                       dp.hist, words);
    if ((st = launch_status("k_zero")) != APACK_OK) return st;
  }
  hipLaunchKernelGGL(k_finalize_hist, dim3(nf), dim3(kT), 0, stream, dp.seqs, dp.ftiles, dp.tags, dp.colpart, hq,
                     hkv, scores, dp.hist);
  if ((st = launch_status("k_finalize_hist")) != APACK_OK) return st;
  if (pl.any_select) {
    for (int pass = 1; pass <= 2; ++pass) {
      hipLaunchKernelGGL(k_select_pass, dim3(nf), dim3(kT), 0, stream, dp.seqs, dp.ftiles, dp.tags, scores,
                         dp.hist, pass);
      if ((st = launch_status("k_select_pass")) != APACK_OK) return st;
    }
  }
  hipLaunchKernelGGL(k_keep_count, dim3(nf), dim3(kT), 0, stream, dp.seqs, dp.ftiles, dp.tags, scores, dp.cnt);
  if ((st = launch_status("k_keep_count")) != APACK_OK) return st;
  hipLaunchKernelGGL(k_keep_write, dim3(nf), dim3(kT), 0, stream, dp.seqs, dp.ftiles, dp.tags, scores, dp.cnt,
                     kept);
  return launch_status("k_keep_write");
}

}  // namespace apack
