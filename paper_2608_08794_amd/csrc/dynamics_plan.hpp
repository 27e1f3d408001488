// Host plan and device descriptors of one apack_score_dynamics call.
#pragma once

#include <cstdint>
#include <vector>

#include "common.hpp"

namespace apack {

constexpr int kMaxWindow = 16;   // largest CKA window
constexpr int kMaxPerFrame = 256;
// A CKA input whose centred Gram has a Frobenius norm of at most this
// fraction of its raw Gram's trace has no variation that fp64 resolves
// through the Gram (repeated or zero frames): its c_f is 0.
constexpr double kCkaDegenerate = 1e-8;

// Cosine from a dot product and the two squared norms, each summed the same
// way: dot / sqrt(nx ny), so a vector and a bitwise copy of it give exactly
// 1 (the square root of a correctly rounded square is exact); 0 when a
// norm is 0.
__device__ __forceinline__ double cos_from(double dot, double nx, double ny) {
  return (nx == 0.0 || ny == 0.0) ? 0.0 : dot / sqrt(nx * ny);
}

// Per-clip descriptor on the device.
struct ClipDev {
  int64_t vis_off, aud_off, qry_off;  // first rows in the packed inputs
  int64_t n_audio, n_query;
  int64_t frame_off;                  // first frame in the [sum F] arrays
  int64_t token_off;                  // first visual token of the clip in [sum F*P] arrays
  int64_t kept_off;                   // first slot of the clip in kept_visual
  int64_t gram_off;                   // first anchor-Gram slot: frame f uses [gram_off + f*P*P ...)
  int64_t budget;                     // B_v
  int32_t n_frames, per_frame;
  int32_t gate;                       // written on the device
  int32_t n_seg;                      // written on the device
};

struct DynParamsDev {
  double tau_gate, beta, gamma, tau_sim, sigma, lambda_seg, cover, power;
  int32_t window, dafps_k, alignment;
};

// Per-frame work item: clip and frame index within it.
struct FrameDev {
  int32_t clip, f;
};

struct GemmTileDev {
  int32_t clip, m0, n0, pad;  // audio row block, visual column block
};

struct DynPlan {
  std::vector<ClipDev> clips;
  std::vector<FrameDev> frames;      // one entry per frame of every clip
  std::vector<int64_t> budgets;
  int64_t total_frames = 0, total_tokens = 0, total_audio = 0, total_kept = 0, total_gram = 0;
  int max_per_frame = 1;
  int64_t gemm_tiles = 0;            // gate GEMM workgroups over all clips
  int32_t spatial_tiles = 0;         // spatial CKA Gram tiles per frame (0 unless selected)
  std::vector<GemmTileDev> gemm;
  std::vector<GemmTileDev> gemm256;  // 256 x 256 tiles (dim a multiple of 64), XCD-ordered
  bool use256 = false;               // set per call: bf16 inputs and gemm256 planned
  // Workspace layout (byte offsets).
  size_t off_clips = 0, off_frames = 0, off_gemm = 0, blob_bytes = 0;
  size_t off_v = 0, off_a = 0, off_q = 0, off_band_v = 0, off_band_a = 0, off_vq = 0, off_qq = 0;
  size_t off_cka = 0, off_nv = 0, off_rv = 0, off_na = 0, off_maxkey = 0, off_plan = 0, off_gram = 0, off_scratch = 0;
  size_t off_spatial = 0, off_sim = 0, off_anchors = 0, off_sqp = 0;
  int64_t gram_items = 0;            // (frame, Gram tile) pairs over all clips: the anchor Gram's items at most
  size_t ws_bytes = 0;
};

// Order-preserving 32-bit keys of fp32 values, so an integer atomicMax
// finds the largest cosine whatever its sign (the visual max-cosine slots
// start at key 0, below every real value).
__device__ __forceinline__ uint32_t order_key(float x) {
  const uint32_t u = __float_as_uint(x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key_value(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

// Per-frame plan written by k_plan and read by the token-selection kernels.
struct FramePlanDev {
  double score;        // s_f
  double dist;         // d_f (0 when the gate did not fire)
  int32_t seg;         // segment id within the clip
  int32_t anchor;      // first frame of the segment (clip-local)
  int32_t budget;      // k_f
  int32_t is_anchor;
  int64_t out_off;     // first kept_visual slot of the frame
};


apack_status build_dyn_plan(int32_t n_seq, const apack_av_seq* seqs, int32_t dim, const apack_dyn_params* p,
                            DynPlan& plan);

struct DynPtrs {
  ClipDev* clips;
  FrameDev* frames;
  GemmTileDev* gemm;
  double *v, *a, *q, *band_v, *band_a, *vq, *qq, *cka, *nv, *rv, *na, *gram, *scratch, *spatial, *sim;
  double* sqp;       // per-slice row sums of squares [slice][visual rows, then audio rows]
  uint32_t* maxkey;
  FramePlanDev* plan;
  int32_t* anchors;  // first frame of each segment, clip c's at frame_off + m
};

// The gate GEMM on 256 x 256 tiles for bf16 inputs whose dim is a multiple
// of 64 (gate_gemm.hip); `tiles` holds one tile per workgroup, already in
// the order the launch expects.
apack_status launch_gate_gemm256(const ClipDev* clips, const GemmTileDev* tiles, int64_t n_tiles, int dim,
                                 const uint16_t* xv, const uint16_t* xa, const double* na, uint32_t* maxkey,
                                 hipStream_t stream);
std::vector<GemmTileDev> gate_gemm256_tiles(const std::vector<ClipDev>& clips);
constexpr int kGemm256K = 64;   // dim must be a multiple of this for the 256-tile kernel
constexpr int kPoolSlice = 512;  // embedding elements per coarse-pass block (8 per lane)

apack_status launch_dynamics(const DynPlan& pl, const DynPtrs& dp, const DynParamsDev& prm, apack_dtype dt,
                             int dim, const void* visual, const void* audio, const void* query, int64_t visual_rows,
                             int64_t audio_rows, float* frame_cka,
                             float* frame_score, int32_t* frame_budget, int32_t* segment_id, uint8_t* gate_fired,
                             int32_t* kept, hipStream_t stream);

}  // namespace apack
