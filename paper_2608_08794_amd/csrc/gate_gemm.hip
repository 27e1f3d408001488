// Gate GEMM of the direct audio-visual distance (Section 3.1, "Gated fine
// pass"; the fine-pass term of Eq. 2): for every visual token i of a clip
// whose gate fired, max_j x_A[j] . x_V[i] / |x_A[j]|, from C = X_A X_V^T on
// bf16 MFMA with fp32 accumulation.  This is the kernel for bf16 inputs
// whose dim is a multiple of 64; k_gate_gemm in dynamics.hip covers the rest.
//
// Each workgroup owns a 256 x 256 tile (audio rows x visual columns); its
// eight waves (two per SIMD, so one wave's loads, waits and LDS reads hide
// under the other's MFMAs) own 128 x 64 blocks as 4 x 2 blocks of
// v_mfma_f32_32x32x16_bf16, so a wave reads 6 fragments from LDS per 8
// MFMAs.  K streams through two 64-element LDS stages (2 x 64 KiB), filled
// by 16-byte direct-to-LDS loads while the other stage is consumed; the
// 128-byte rows are stored with their 16-byte chunks XOR-swizzled by the
// row index, so the fragment reads of consecutive rows hit distinct banks
// without padding.  Every output element sees the same sequence of MFMAs
// (K in order, 16 at a time) as in k_gate_gemm, so the results are the same
// bits.  The epilogue scales by the inverse audio norms and folds the
// column maxima into order-preserving keys with atomicMax.
//
// Workgroups are dealt to the eight XCDs round-robin by index, so the host
// lists the tiles so that each XCD gets whole column blocks of one band of
// at most eight row tiles, and the workgroups resident on one XCD share
// both operands in that XCD's L2: a band's audio rows and a few column
// blocks of visual rows.
#include <algorithm>
#include <cmath>

#include "common.hpp"
#include "dynamics_plan.hpp"

namespace apack {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void* lds_ptr_t;
typedef __attribute__((address_space(1))) void* glb_ptr_t;

constexpr int kTile = 256;                     // rows and columns per workgroup
constexpr int kK = kGemm256K;                  // K elements per LDS stage
constexpr int kStages = 2;                     // stages in flight (loads kStages-1 ahead)
constexpr int kRowB = kK * 2;                  // bytes of one row per stage
constexpr int kChunks = kRowB / 16;            // 16-byte chunks per row
constexpr int kOpB = kTile * kRowB;            // one operand's stage
constexpr int kStageB = 2 * kOpB;
constexpr int kWaves = 8;
constexpr int kWN = 4;                         // waves along the visual columns
constexpr int kBI = kTile / (kWaves / kWN) / 32; // 32-row blocks per wave
constexpr int kBJ = kTile / kWN / 32;            // 32-column blocks per wave
constexpr int kLoadsPerWave = kOpB / 1024 / kWaves;  // 1 KiB loads per wave per operand
static_assert(kBI * kBJ == 8 && kBI + kBJ == 6, "the K-slice schedule interleaves 6 fragment reads with 8 MFMAs");
constexpr int kXcds = 8;

// Chunk c of row r sits at chunk c ^ swz(r).  A 16-byte LDS read is served
// sixteen lanes at a time across 64 four-byte banks (256 bytes); the
// sixteen consecutive rows those lanes read must then fill the 256 bytes
// once.  Rows share a 256-byte window kRowsPer256 at a time, so the XOR key
// is the row's index among the rows that fall on the same banks.
constexpr int kRowsPer256 = 256 / kRowB;
__device__ __forceinline__ int swz(int r) { return (r / kRowsPer256) & (kChunks - 1); }

// One operand's stage: rows r0 .. r0+255 (clamped to the last valid row),
// elements [k0, k0 + kK).  Load j fills LDS bytes [1024 j, 1024 j + 1024);
// lane l's 16 bytes land at row r = (1024 j + 16 l) / kRowB, chunk c, and
// come from global chunk c ^ swz(r).  off[i] is lane l's byte offset of load
// i from the stage's first byte (row r0, element k0), the same for every
// stage, so a stage only moves the scalar base.
__device__ __forceinline__ void operand_offsets(int64_t r0, int64_t n_rows, int dim, int wave, int lane,
                                                uint32_t (&off)[kLoadsPerWave]) {
#pragma unroll
  for (int i = 0; i < kLoadsPerWave; ++i) {
    const int j = wave * kLoadsPerWave + i;
    const int byte = j * 1024 + lane * 16;
    const int r = byte / kRowB;
    const int c = ((byte % kRowB) >> 4) ^ swz(r);
    const int64_t left = n_rows - 1 - r0;
    const int rr = left < r ? (int)left : r;
    off[i] = (uint32_t)rr * (uint32_t)dim * 2u + (uint32_t)c * 16u;
  }
}

__device__ __forceinline__ void issue_operand(char* lds, const char* base, const uint32_t (&off)[kLoadsPerWave],
                                              int wave) {
#pragma unroll
  for (int i = 0; i < kLoadsPerWave; ++i) {
    const int j = wave * kLoadsPerWave + i;
    __builtin_amdgcn_global_load_lds((glb_ptr_t)(base + off[i]), (lds_ptr_t)(lds + j * 1024), 16, 0, 0);
  }
}

// MFMA operand of rows row .. row+31 (row a multiple of 32 plus lane % 32)
// and K elements [16 ks, 16 ks + 16): lane l holds 8 elements at
// 16 ks + 8 (l / 32).
__device__ __forceinline__ bf16x8 lds_frag(const char* lds, int row, int ks, int lane) {
  const int c = (ks * 2 + (lane >> 5)) ^ swz(row);
  return *reinterpret_cast<const bf16x8*>(lds + row * kRowB + c * 16);
}

__global__ __launch_bounds__(kWaves * 64) __attribute__((amdgpu_waves_per_eu(2, 2))) void k_gate_gemm256(
    const ClipDev* __restrict__ clips, const GemmTileDev* __restrict__ tiles, int dim, const uint16_t* __restrict__ xv,
    const uint16_t* __restrict__ xa, const double* __restrict__ na, uint32_t* __restrict__ maxkey) {
  __shared__ __attribute__((aligned(16))) char lds[kStages * kStageB];
  const GemmTileDev tl = tiles[blockIdx.x];
  if (tl.clip < 0) return;  // padding of an XCD's share
  const ClipDev c = clips[tl.clip];
  if (!c.gate) return;
  const int64_t n_a = c.n_audio, n_v = (int64_t)c.n_frames * c.per_frame;
  const uint16_t* A = xa + c.aud_off * dim;
  const uint16_t* B = xv + c.vis_off * dim;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / kWN, wn = wave % kWN;

  f32x16 acc[kBI][kBJ];
#pragma unroll
  for (int i = 0; i < kBI; ++i)
#pragma unroll
    for (int j = 0; j < kBJ; ++j) acc[i][j] = f32x16{};

  const int n_k = dim / kK;
  uint32_t off_a[kLoadsPerWave], off_b[kLoadsPerWave];
  operand_offsets(tl.m0, n_a, dim, wave, lane, off_a);
  operand_offsets(tl.n0, n_v, dim, wave, lane, off_b);
  const char* base_a = reinterpret_cast<const char*>(A + tl.m0 * dim);
  const char* base_b = reinterpret_cast<const char*>(B + tl.n0 * dim);
  auto issue = [&](int k_stage) {
    char* st = lds + (k_stage % kStages) * kStageB;
    issue_operand(st, base_a + (size_t)k_stage * kK * 2, off_a, wave);
    issue_operand(st + kOpB, base_b + (size_t)k_stage * kK * 2, off_b, wave);
  };
  // Loads run kStages - 1 stages ahead of the MFMAs.
  for (int p = 0; p < kStages - 1 && p < n_k; ++p) issue(p);
  for (int it = 0; it < n_k; ++it) {
    const int buf = it % kStages;
    // Stage it has landed: each wave waits until at most the loads of the
    // later stages it issued are outstanding, then the barrier makes every
    // wave's share visible and guarantees the stage about to be refilled
    // (read at it - 1) is no longer read.
    const int ahead = std::min(kStages - 2, n_k - 1 - it);   // stages issued after this one
    if (ahead >= 2)
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * 2 * kLoadsPerWave) : "memory");
    else if (ahead == 1)
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * kLoadsPerWave) : "memory");
    else
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    const char* la = lds + buf * kStageB;
    const char* lb = la + kOpB;
    // Fragments of K slice ks + 1 are read while slice ks's MFMAs run.
    bf16x8 fa[2][kBI], fb[2][kBJ];
    auto read = [&](int ks, int h) {
#pragma unroll
      for (int i = 0; i < kBI; ++i) fa[h][i] = lds_frag(la, wm * kBI * 32 + i * 32 + (lane & 31), ks, lane);
#pragma unroll
      for (int j = 0; j < kBJ; ++j) fb[h][j] = lds_frag(lb, wn * kBJ * 32 + j * 32 + (lane & 31), ks, lane);
    };
    // The first slice's reads go out before the next stage's loads are
    // issued, so their latency runs under the load issue rather than ahead
    // of the first MFMA.
    read(0, 0);
    __builtin_amdgcn_sched_barrier(0);
    if (it + kStages - 1 < n_k) issue(it + kStages - 1);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int ks = 0; ks < kK / 16; ++ks) {
      const int h = ks & 1;
      // Slices run at raised wave priority, so a wave in its MFMAs issues
      // ahead of the other wave on the SIMD while that one waits at the
      // stage barrier or issues loads.
      __builtin_amdgcn_s_setprio(1);
      if (ks + 1 < kK / 16) read(ks + 1, h ^ 1);
#pragma unroll
      for (int i = 0; i < kBI; ++i)
#pragma unroll
        for (int j = 0; j < kBJ; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[h][i], fb[h][j], acc[i][j], 0, 0, 0);
      // Slice ks + 1's six fragment reads go one after each of slice ks's
      // first six MFMAs (the scheduler would otherwise sink each read to its
      // first use); nothing crosses into the next slice.
#pragma unroll
      for (int g = 0; g < 6; ++g) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // one LDS read
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_setprio(0);
    }
  }

  // Epilogue.  Inverse audio norms of the tile's rows in LDS (-inf past the
  // clip's audio, so those rows never win); acc[i][j][e] of lane l is audio
  // row 32 (kBI wm + i) + 8(e/4) + 4(l/32) + e%4, visual column
  // 32 (kBJ wn + j) + l%32.
  __syncthreads();
  float* inv = reinterpret_cast<float*>(lds);
  for (int r = tid; r < kTile; r += kWaves * 64) {
    const int64_t row = tl.m0 + r;
    float s = -INFINITY;
    if (row < n_a) {
      const double nn = na[c.aud_off + row];
      s = nn > 0.0 ? (float)(1.0 / sqrt(nn)) : 0.0f;
    }
    inv[r] = s;
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < kBJ; ++j) {
    float m = -INFINITY;
#pragma unroll
    for (int i = 0; i < kBI; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float s = inv[wm * kBI * 32 + i * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3)];
        m = fmaxf(m, s == -INFINITY ? -INFINITY : acc[i][j][e] * s);
      }
    m = fmaxf(m, __shfl_xor(m, 32));
    const int64_t col = tl.n0 + wn * kBJ * 32 + j * 32 + (lane & 31);
    if (lane < 32 && col < n_v && m > -INFINITY) atomicMax(&maxkey[c.vis_off + col], order_key(m));
  }
}

}  // namespace

std::vector<GemmTileDev> gate_gemm256_tiles(const std::vector<ClipDev>& clips) {
  // A clip's row tiles are cut into bands of at most kBandRows (as even as
  // possible); per band, column blocks (clip, n0) are dealt to the XCDs in
  // turn, and an XCD's share lists the band's row tiles of its blocks, block
  // after block.  A tall clip's audio then passes through each XCD's L2 once
  // per band and column block rather than once per column block.
  constexpr int kBandRows = 8;
  std::vector<std::vector<GemmTileDev>> share(kXcds);
  int next = 0;
  for (size_t s = 0; s < clips.size(); ++s) {
    const ClipDev& c = clips[s];
    const int64_t nv = (int64_t)c.n_frames * c.per_frame;
    if (nv == 0 || c.n_audio == 0) continue;
    const int mb = (int)((c.n_audio + kTile - 1) / kTile), nb = (int)((nv + kTile - 1) / kTile);
    const int n_band = (mb + kBandRows - 1) / kBandRows;
    for (int b = 0; b < n_band; ++b) {
      const int m0 = b * mb / n_band, m1 = (b + 1) * mb / n_band;
      for (int n = 0; n < nb; ++n, next = (next + 1) % kXcds)
        for (int m = m0; m < m1; ++m) share[next].push_back({(int32_t)s, m * kTile, n * kTile, 0});
    }
  }
  size_t rounds = 0;
  for (auto& q : share) rounds = std::max(rounds, q.size());
  std::vector<GemmTileDev> out;
  out.reserve(rounds * kXcds);
  for (size_t r = 0; r < rounds; ++r)
    for (int x = 0; x < kXcds; ++x) out.push_back(r < share[x].size() ? share[x][r] : GemmTileDev{-1, 0, 0, 0});
  // Trailing padding only costs empty workgroups; drop it.
  while (!out.empty() && out.back().clip < 0) out.pop_back();
  return out;
}

apack_status launch_gate_gemm256(const ClipDev* clips, const GemmTileDev* tiles, int64_t n_tiles, int dim,
                                 const uint16_t* xv, const uint16_t* xa, const double* na, uint32_t* maxkey,
                                 hipStream_t stream) {
  if (n_tiles == 0) return APACK_OK;
  hipLaunchKernelGGL(k_gate_gemm256, dim3((unsigned)n_tiles), dim3(kWaves * 64), 0, stream, clips, tiles, dim, xv, xa,
                     na, maxkey);
  return launch_status("k_gate_gemm256");
}

}  // namespace apack
