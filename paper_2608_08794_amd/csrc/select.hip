// Later digits of the per-modality top-k (Eq. 6 within each modality) and
// the ordered list of kept rows, spread over the whole GPU in row tiles of
// 1024 rows.  The scores and the first digit's bin come from the score
// kernels (the radix scheme is described with its helpers).
//
// Kept rows: every non-candidate row, every row above the threshold T, and
// the first (k - count above) rows equal to T in row order (the lower row
// wins ties).  A count kernel records each tile's (sure keeps, ties per
// modality); a write kernel adds up the tiles before it and places its rows
// with block scans.  No kernel waits on another workgroup.
#include <cfloat>

#include "common.hpp"
#include "prune_plan.hpp"
#include "radix.hpp"

namespace apack {
namespace {

constexpr int kT = 256;              // threads per row tile
constexpr int kPer = kRowTile / kT;  // rows per thread (contiguous)
constexpr int kBins1 = kRadixBins;

// Counts the tile's participating digits and merges them into the global
// histogram; the last tile of the sequence picks the bins.
__device__ void hist_pass(SeqDev* sq, uint32_t* hist, const uint32_t (&bits)[kPer], const uint8_t (&mt)[kPer],
                          int pass, uint32_t* lh) {
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
  merge_hist<kT>(lh, hist);
  if (!arrive_last<kT>(&sq->done_cnt, (uint32_t)sq->n_ftiles)) return;
  pick_bins<kT>(sq, hist, pass);
  if (tid == 0) sq->done_cnt = 0;
}

__device__ __forceinline__ void tile_rows(const FTileDev& ft, const SeqDev& sq, int64_t& r0, int& n) {
  r0 = (int64_t)ft.idx * kRowTile;
  const int64_t left = sq.n_tokens - r0;
  n = left < kRowTile ? (int)left : kRowTile;
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
    const int i = min((int)threadIdx.x * kPer + u, n - 1);
    mt[u] = tg[r0 + i];
    bits[u] = clamp_bits(scores[sq->tok_off + r0 + i]);
  }
#pragma unroll
  for (int u = 0; u < kPer; ++u)
    if ((int)threadIdx.x * kPer + u >= n) mt[u] = 0xFF;
  hist_pass(sq, hist + (int64_t)ft.seq * 2 * kBins1, bits, mt, pass, lh);
}

// Per tile: (rows kept for sure, rows equal to T_audio, rows equal to T_visual).
__global__ __launch_bounds__(kT) void k_keep_count(const SeqDev* __restrict__ seqs,
                                                   const FTileDev* __restrict__ ftiles,
                                                   const uint8_t* __restrict__ tags,
                                                   float* __restrict__ scores, uint32_t* __restrict__ cnt) {
  __shared__ uint32_t sh[kT / 64];
  const FTileDev ft = ftiles[blockIdx.x];
  const SeqDev sq = seqs[ft.seq];
  int64_t r0;
  int n;
  tile_rows(ft, sq, r0, n);
  const uint8_t* tg = tags + sq.tag_off;
  const uint32_t thr[2] = {sq.thr[0], sq.thr[1]};
  const bool no_cand = sq.n_cand == 0;
  uint32_t sure = 0, ea = 0, ev = 0;
  // Tags and scores are loaded together (rows past the tile re-read its last
  // row and are then skipped), so no score load waits for its tag.
  uint8_t mt[kPer];
  float sc[kPer];
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int i = min((int)threadIdx.x * kPer + u, n - 1);
    mt[u] = tg[r0 + i];
    sc[u] = scores[sq.tok_off + r0 + i];
  }
  // Counted without branches, so that the loads above are not moved into
  // per-row branches (and waited for one row at a time).
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int i = threadIdx.x * kPer + u;
    const uint8_t m = i < n ? mt[u] : 0xFF;
    const uint32_t b = clamp_bits(sc[u]);
    const uint32_t t = m == 2 ? thr[1] : thr[0];
    const bool cand = m == 1 || m == 2;
    sure += (m == 0 || (cand && b > t)) ? 1u : 0u;
    ea += (m == 1 && b == t) ? 1u : 0u;
    ev += (m == 2 && b == t) ? 1u : 0u;
  }
  // Scores of sequences with candidates are written by the score kernels; a
  // sequence without any has no score workgroups.
  if (no_cand) {
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int i = threadIdx.x * kPer + u;
      if (i < n && mt[u] == 0) scores[sq.tok_off + r0 + i] = 0.f;
    }
  }
  uint32_t tot;
  block_scan<kT>(sure, sh, tot);
  const uint32_t s_tot = tot;
  block_scan<kT>(ea | (ev << 16), sh, tot);
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
  const SeqDev sq = seqs[ft.seq];
  int64_t r0;
  int n;
  tile_rows(ft, sq, r0, n);
  const uint8_t* tg = tags + sq.tag_off;
  const uint32_t need0 = (uint32_t)sq.need[0], need1 = (uint32_t)sq.need[1];
  const uint32_t thr0 = sq.thr[0], thr1 = sq.thr[1];
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
    block_scan<kT>(s, sh, ts);
    block_scan<kT>(a, sh, ta);
    block_scan<kT>(v, sh, tv);
    if (threadIdx.x == 0) {
      base_sh[0] = (uint64_t)ts + min(ta, need0) + min(tv, need1);
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
    const int i = min((int)threadIdx.x * kPer + u, n - 1);
    mt[u] = tg[r0 + i];
    bits[u] = __float_as_uint(scores[sq.tok_off + r0 + i]);
  }
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    if ((int)threadIdx.x * kPer + u >= n) mt[u] = 0xFF;
    bits[u] = mt[u] != 0 ? clamp_bits(__uint_as_float(bits[u])) : 0u;
    if (mt[u] == 1 && bits[u] == thr0) ++ea;
    if (mt[u] == 2 && bits[u] == thr1) ++ev;
  }
  uint32_t tot;
  const uint32_t packed = ea | (ev << 16);
  const uint32_t ex = block_scan<kT>(packed, sh, tot) - packed;
  uint64_t rank_a = base_sh[1] + (ex & 0xFFFFu), rank_v = base_sh[2] + (ex >> 16);
  bool keep[kPer];
  uint32_t nk = 0;
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const uint8_t m = mt[u];
    bool kp = false;
    if (m == 0) kp = true;
    else if (m == 1 || m == 2) {
      const uint32_t t = m == 1 ? thr0 : thr1;
      if (bits[u] > t) kp = true;
      else if (bits[u] == t) kp = (m == 1 ? rank_a++ : rank_v++) < (m == 1 ? need0 : need1);
    }
    keep[u] = kp;
    nk += kp;
  }
  const uint64_t pos0 = base_sh[0] + (block_scan<kT>(nk, sh, tot) - nk);
  int32_t* out = kept + sq.out_off;
  uint64_t pos = pos0;
#pragma unroll
  for (int u = 0; u < kPer; ++u)
    if (keep[u]) {
      if (pos < (uint64_t)sq.n_kept) out[pos] = (int32_t)(sq.tok_off + r0 + threadIdx.x * kPer + u);
      ++pos;
    }
}

// ---------------------------------------------------------------------------
// Short sequences (up to kSmallRows rows): one workgroup per sequence holds
// every row's tag and score in registers and runs the last two digits with
// LDS histograms, the threshold, and the ordered kept list, in one launch
// instead of four.  Same rules as above: rows above the threshold, then the
// first `need` rows equal to it in row order.
// Wave w holds rows [1024 w, 1024 (w + 1)), lane l of it rows 1024 w + 64 u + l
// (u < 16), so every load is coalesced; ranks among ties and output slots
// come from ballots inside a wave and a scan over the 16 wave totals.
// ---------------------------------------------------------------------------
constexpr int kST = 1024;                 // threads
constexpr int kSPer = 16;                 // rows per thread
constexpr int kSWaves = kST / 64;
constexpr int kSmallRows = kST * kSPer;

// Lanes below this one with their bit set in a wave-wide mask.
__device__ __forceinline__ uint32_t below(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Exclusive prefix of the per-wave values in s[0 .. kSWaves) for wave w;
// every thread calls it (it holds a barrier before the reads).
__device__ __forceinline__ uint32_t wave_base(const uint32_t* s, int w) {
  __syncthreads();
  uint32_t b = 0;
#pragma unroll
  for (int i = 0; i < kSWaves; ++i)
    if (i < w) b += s[i];
  return b;
}

__global__ __launch_bounds__(kST) void k_select_small(const SeqDev* __restrict__ seqs,
                                                      const uint8_t* __restrict__ tags,
                                                      float* __restrict__ scores, int32_t* __restrict__ kept) {
  __shared__ uint32_t lh[2 * kBins1];
  __shared__ uint32_t sh[kST / 64];
  __shared__ uint32_t s_prefix[2], s_kk[2], s_thr[2], s_need[2], s_part[2];
  __shared__ uint32_t s_wave[2][kSWaves];
  const SeqDev sq = seqs[blockIdx.x];
  const int n = (int)sq.n_tokens;
  if (n == 0) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int row0 = wave * (64 * kSPer) + lane;   // row of u = 0; row(u) = row0 + 64 u
  const uint8_t* tg = tags + sq.tag_off;
  uint32_t bits[kSPer];
  uint8_t mt[kSPer];
  // Every tag and score load is issued before the first is used: a row
  // past the sequence re-reads its last row, and a score is kept only for a
  // candidate row, so no load waits behind another (a score load behind a
  // test of its tag had waited for the tag first, one row at a time).
#pragma unroll
  for (int u = 0; u < kSPer; ++u) {
    const int i = min(row0 + 64 * u, n - 1);
    mt[u] = tg[i];
    bits[u] = __float_as_uint(scores[sq.tok_off + i]);
  }
#pragma unroll
  for (int u = 0; u < kSPer; ++u) {
    const int i = row0 + 64 * u;
    if (i >= n) mt[u] = 0xFF;
    bits[u] = (mt[u] == 1 || mt[u] == 2) ? clamp_bits(__uint_as_float(bits[u])) : 0u;
  }
  // Scores of sequences with candidates are written by the score kernels; a
  // sequence without any has no score workgroups.
  if (sq.n_cand == 0) {
#pragma unroll
    for (int u = 0; u < kSPer; ++u)
      if (mt[u] == 0) scores[sq.tok_off + row0 + 64 * u] = 0.f;
  }
  if (tid < 2) {
    s_prefix[tid] = tid ? sq.prefix[1] : sq.prefix[0];
    s_kk[tid] = tid ? sq.kk[1] : sq.kk[0];
    s_thr[tid] = tid ? sq.thr[1] : sq.thr[0];
    s_need[tid] = (uint32_t)(tid ? sq.need[1] : sq.need[0]);
    s_part[tid] = 0;   // a modality that does not select keeps all or none of its rows
  }
  __syncthreads();
  const bool act0 = sq.select[0] != 0, act1 = sq.select[1] != 0;
  for (int pass = 1; pass <= 2 && (act0 || act1); ++pass) {
    for (int b = tid; b < 2 * kBins1; b += kST) lh[b] = 0;
    __syncthreads();
    const uint32_t pre0 = s_prefix[0], pre1 = s_prefix[1];
#pragma unroll
    for (int u = 0; u < kSPer; ++u) {
      const bool a = mt[u] == 1 && act0, v = mt[u] == 2 && act1;
      if (!a && !v) continue;
      uint32_t d;
      if (digit_of(bits[u], pass, a ? pre0 : pre1, d)) atomicAdd(&lh[(a ? 0 : kBins1) + d], 1u);
    }
    __syncthreads();
    // Bin holding the kk-th largest value of each modality: thread t covers
    // bins nb-1-2t and nb-2-2t (descending); one block scan serves both
    // modalities, their counts (at most kSmallRows) packed in 16-bit halves.
    const int nb = pass == 2 ? 512 : kRadixBins;
    uint32_t c[2][2], sum = 0;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int b = nb - 1 - (tid * 2 + j);
      c[0][j] = b >= 0 ? lh[b] : 0u;
      c[1][j] = b >= 0 ? lh[kBins1 + b] : 0u;
      sum += c[0][j] | (c[1][j] << 16);
    }
    // Ranks and prefixes are read before the scan, whose barriers keep every
    // read ahead of the writes below.
    const uint32_t kk[2] = {s_kk[0], s_kk[1]}, pf[2] = {s_prefix[0], s_prefix[1]};
    uint32_t total;
    const uint32_t incl = block_scan<kST>(sum, sh, total);
    for (int m = 0; m < 2; ++m) {
      if (!(m == 0 ? act0 : act1)) continue;
      const uint32_t in_m = (incl >> (16 * m)) & 0xFFFFu, s_m = c[m][0] + c[m][1];
      uint32_t before = in_m - s_m;
      if (before < kk[m] && in_m >= kk[m]) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          if (before < kk[m] && before + c[m][j] >= kk[m]) {
            const uint32_t b = (uint32_t)(nb - 1 - (tid * 2 + j));
            const uint32_t prefix = (pf[m] << (pass == 1 ? 11 : 9)) | b;
            s_prefix[m] = prefix;
            s_kk[m] = kk[m] - before;
            if (pass == 2) {
              s_thr[m] = prefix;
              s_need[m] = kk[m] - before;
              s_part[m] = kk[m] - before != c[m][j] ? 1u : 0u;
            }
          }
          before += c[m][j];
        }
      }
    }
    __syncthreads();
  }
  // Kept: every non-candidate row, every candidate above its modality's
  // threshold and the first `need` rows equal to it in row order.  When
  // every row equal to the threshold is kept (the usual case), no rank is
  // formed.  The tests are bitwise (no short-circuit), so they compile to
  // straight-line compares rather than nested branches.
  const uint32_t thr0 = s_thr[0], thr1 = s_thr[1], need0 = s_need[0], need1 = s_need[1];
  uint32_t keepbits = 0, nk = 0;
  if (!(s_part[0] | s_part[1])) {
#pragma unroll
    for (int u = 0; u < kSPer; ++u) {
      const bool kp = (mt[u] == 0) | ((mt[u] == 1) & (bits[u] >= thr0)) | ((mt[u] == 2) & (bits[u] >= thr1));
      keepbits |= (uint32_t)kp << u;
      nk += __popcll(__ballot(kp));
    }
  } else {
    // Ranks of the rows equal to each threshold: wave totals, then within
    // the wave by u and by lane.
    uint32_t ta = 0, tv = 0;
#pragma unroll
    for (int u = 0; u < kSPer; ++u) {
      ta += __popcll(__ballot((mt[u] == 1) & (bits[u] == thr0)));
      tv += __popcll(__ballot((mt[u] == 2) & (bits[u] == thr1)));
    }
    if (lane == 0) {
      s_wave[0][wave] = ta;
      s_wave[1][wave] = tv;
    }
    uint32_t ra = wave_base(s_wave[0], wave), rv = wave_base(s_wave[1], wave);
#pragma unroll
    for (int u = 0; u < kSPer; ++u) {
      const bool ea = (mt[u] == 1) & (bits[u] == thr0), ev = (mt[u] == 2) & (bits[u] == thr1);
      const uint64_t ma = __ballot(ea), mv = __ballot(ev);
      const int kp = (int)(mt[u] == 0) | ((int)(mt[u] == 1) & (int)(bits[u] > thr0)) |
                     ((int)(mt[u] == 2) & (int)(bits[u] > thr1)) | ((int)ea & (int)(ra + below(ma) < need0)) |
                     ((int)ev & (int)(rv + below(mv) < need1));
      ra += __popcll(ma);
      rv += __popcll(mv);
      keepbits |= (uint32_t)kp << u;
      nk += __popcll(__ballot(kp));
    }
    __syncthreads();   // every wave has read s_wave
  }
  if (lane == 0) s_wave[0][wave] = nk;
  uint32_t pos = wave_base(s_wave[0], wave);
  int32_t* out = kept + sq.out_off;
#pragma unroll
  for (int u = 0; u < kSPer; ++u) {
    const bool kp = (keepbits >> u) & 1u;
    const uint64_t mk = __ballot(kp);
    const uint32_t at = pos + below(mk);
    if (kp && at < (uint32_t)sq.n_kept) out[at] = (int32_t)(sq.tok_off + row0 + 64 * u);
    pos += __popcll(mk);
  }
}

}  // namespace

int64_t select_hist_words(int64_t n_seq) { return n_seq * 2 * kRadixBins; }

apack_status launch_select(const PrunePlan& pl, const DevPtrs& dp, float* scores, int32_t* kept,
                           hipStream_t stream) {
  const int nf = (int)pl.ftiles.size();
  if (nf == 0) return APACK_OK;
  apack_status st;
  // The scores and the first digit come from k_colsum, earlier on this stream.
  if (pl.max_tokens <= kSmallRows) {
    hipLaunchKernelGGL(k_select_small, dim3((unsigned)pl.seqs.size()), dim3(kST), 0, stream, dp.seqs, dp.tags,
                       scores, kept);
    return launch_status("k_select_small");
  }
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
