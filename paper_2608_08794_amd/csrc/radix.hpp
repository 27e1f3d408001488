// Device helpers of the per-modality radix select (Eq. 6 within each
// modality), shared by the score kernels (first digit) and the select
// kernels (later digits, threshold and kept list).
//
// Scores are non-negative fp32, so their bit patterns order like the
// values.  The k-th largest bit pattern of each (sequence, modality) is found
// digit by digit: bits 30..20, then 19..9, then 8..0.  A workgroup counts its
// rows' digits in LDS (rows whose higher digits match the prefix chosen so
// far), adds the non-zero bins to the sequence's global histogram, and the
// last workgroup of the sequence to finish (a fenced atomic counter) picks
// the bin holding the k-th value, records it in the sequence descriptor and
// clears the histogram for the next digit.
#pragma once

#include <cstdint>

#include "prune_plan.hpp"
#include "sync.hpp"

namespace apack {

constexpr int kRadixBins = 2048;

__device__ __forceinline__ uint32_t clamp_bits(float s) { return min(__float_as_uint(s), 0x7F800000u); }

// Inclusive scan over a block of NT threads; sh holds NT/64 words.
template <int NT>
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
  for (int w = 0; w < NT / 64; ++w) {
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

// Run by the last workgroup of a sequence: for each modality still
// selecting, the bin that holds the kk-th largest value; records the prefix,
// the rank left inside the bin and, after the last digit, the threshold.
// Clears the histogram.  Thread t covers bins nb-1-B*t ... nb-B*(t+1).
template <int NT>
__device__ void pick_bins(SeqDev* sq, uint32_t* hist, int pass) {
  constexpr int B = (kRadixBins + NT - 1) / NT;
  __shared__ uint32_t sh[NT / 64];
  const int tid = threadIdx.x;
  const int nb = pass == 2 ? 512 : kRadixBins;
  const bool act[2] = {sq->select[0] != 0, sq->select[1] != 0};
  // Both modalities' bins, ranks and prefixes are read first (one round
  // trip for the bins); the scans' barriers keep every read ahead of the
  // one thread that overwrites a rank or prefix below.
  uint32_t c[2][B];
#pragma unroll
  for (int m = 0; m < 2; ++m)
#pragma unroll
    for (int j = 0; j < B; ++j) {
      const int b = nb - 1 - (tid * B + j);
      c[m][j] = act[m] && b >= 0 ? ld_agent(hist + m * kRadixBins + b) : 0u;
    }
  const uint32_t kk2[2] = {sq->kk[0], sq->kk[1]}, prefix2[2] = {sq->prefix[0], sq->prefix[1]};
  for (int m = 0; m < 2; ++m) {
    if (!act[m]) continue;
    uint32_t* h = hist + m * kRadixBins;
    const uint32_t kk = kk2[m], prefix0 = prefix2[m];
    uint32_t sum = 0;
#pragma unroll
    for (int j = 0; j < B; ++j) sum += c[m][j];
    uint32_t total;
    const uint32_t incl = block_scan<NT>(sum, sh, total);
    uint32_t before = incl - sum;
    if (before < kk && incl >= kk) {
#pragma unroll
      for (int j = 0; j < B; ++j) {
        if (before < kk && before + c[m][j] >= kk) {
          const uint32_t b = (uint32_t)(nb - 1 - (tid * B + j));
          const uint32_t prefix = pass == 0 ? b : (prefix0 << (pass == 1 ? 11 : 9)) | b;
          sq->prefix[m] = prefix;
          sq->kk[m] = kk - before;
          if (pass == 2) {
            sq->thr[m] = prefix;
            sq->need[m] = (int32_t)(kk - before);
            sq->all_eq[m] = (kk - before == c[m][j]) ? 1 : 0;
          }
        }
        before += c[m][j];
      }
    }
    __syncthreads();
    for (int b = tid; b < kRadixBins; b += NT) h[b] = 0;
  }
}

// Adds a workgroup's LDS histogram (2 modalities x 2048 bins) to the
// sequence's global histogram, non-zero bins only.
template <int NT>
__device__ __forceinline__ void merge_hist(const uint32_t* lh, uint32_t* hist) {
  for (int b = threadIdx.x; b < 2 * kRadixBins; b += NT) {
    const uint32_t v = lh[b];
    if (v) atomicAdd(&hist[b], v);
  }
}

}  // namespace apack
