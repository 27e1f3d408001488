// Host side of apack_score_dynamics (pre-LLM scorer, Section 3.1):
// validation, planning, descriptor upload and the launch sequence.
#include <algorithm>
#include <cmath>
#include <cstring>

#include "common.hpp"
#include "dynamics_plan.hpp"

namespace apack {

static apack_status check_params(const apack_dyn_params* p) {
  APACK_CHECK(p, APACK_E_ARG, "params is NULL");
  APACK_CHECK(p->window >= 1 && p->window <= kMaxWindow, APACK_E_ARG, "window must lie in [1, %d]", kMaxWindow);
  APACK_CHECK(p->dafps_k >= 1 && p->dafps_k <= 32, APACK_E_ARG, "dafps_k must lie in [1, 32]");
  APACK_CHECK(p->sigma > 0.0 && p->sigma <= 15.0, APACK_E_ARG, "sigma must lie in (0, 15]");
  APACK_CHECK(std::isfinite(p->tau_gate) && std::isfinite(p->tau_sim), APACK_E_ARG, "thresholds must be finite");
  APACK_CHECK(p->beta >= 0.0 && p->beta <= 1.0 && p->gamma >= 0.0 && p->gamma <= 1.0 && p->lambda_seg >= 0.0 &&
                  p->lambda_seg <= 1.0,
              APACK_E_ARG, "beta, gamma and lambda_seg must lie in [0, 1]");
  APACK_CHECK(p->cover_thresh >= -1.0 && p->cover_thresh <= 1.0, APACK_E_ARG, "cover_thresh must lie in [-1, 1]");
  APACK_CHECK(p->dafps_power >= 0.0 && std::isfinite(p->dafps_power), APACK_E_ARG, "dafps_power must be >= 0");
  APACK_CHECK(p->r_pre >= 0.0 && p->r_pre <= 1.0, APACK_E_ARG, "r_pre must lie in [0, 1]");
  APACK_CHECK(p->alignment >= APACK_ALIGN_GATED_CKA && p->alignment <= APACK_ALIGN_SPATIAL_CKA, APACK_E_ARG,
              "alignment must be one of APACK_ALIGN_*");
  return APACK_OK;
}

apack_status build_dyn_plan(int32_t n_seq, const apack_av_seq* seqs, int32_t dim, const apack_dyn_params* p,
                            DynPlan& pl) {
  APACK_CHECK(n_seq >= 0, APACK_E_ARG, "n_seq must be >= 0");
  APACK_CHECK(n_seq == 0 || seqs, APACK_E_ARG, "seqs is NULL");
  APACK_CHECK(dim > 0 && dim % 8 == 0 && dim <= 16384, APACK_E_SHAPE, "dim must be a positive multiple of 8, <= 16384");
  apack_status st = check_params(p);
  if (st != APACK_OK) return st;
  pl = DynPlan();
  int64_t frames = 0, kept = 0, gram = 0, vis_end = 0, aud_end = 0, tokens = 0;
  for (int s = 0; s < n_seq; ++s) {
    const apack_av_seq& a = seqs[s];
    APACK_CHECK(a.n_frames >= 0 && a.tokens_per_frame >= 1 && a.tokens_per_frame <= kMaxPerFrame, APACK_E_SHAPE,
                "clip %d: n_frames >= 0 and tokens_per_frame in [1, %d] required", s, kMaxPerFrame);
    APACK_CHECK(a.n_audio >= 1 && a.n_query >= 1, APACK_E_SHAPE, "clip %d: n_audio and n_query must be >= 1", s);
    APACK_CHECK(a.vis_off >= 0 && a.aud_off >= 0 && a.qry_off >= 0, APACK_E_SHAPE, "clip %d: negative offset", s);
    ClipDev c;
    std::memset(&c, 0, sizeof c);
    c.vis_off = a.vis_off;
    c.aud_off = a.aud_off;
    c.qry_off = a.qry_off;
    c.n_audio = a.n_audio;
    c.n_query = a.n_query;
    c.n_frames = a.n_frames;
    c.per_frame = a.tokens_per_frame;
    c.frame_off = frames;
    c.token_off = tokens;
    c.kept_off = kept;
    c.gram_off = gram;
    const int64_t nv = (int64_t)a.n_frames * a.tokens_per_frame;
    c.budget = apack_visual_budget(p->r_pre, a.n_audio, nv);
    APACK_CHECK(c.budget >= 0, APACK_E_ARG, "clip %d: bad visual budget", s);
    pl.budgets.push_back(c.budget);
    for (int f = 0; f < a.n_frames; ++f) pl.frames.push_back({s, f});
    frames += a.n_frames;
    tokens += nv;
    kept += c.budget;
    gram += nv * a.tokens_per_frame;
    const int64_t nt = (a.tokens_per_frame + 15) / 16;
    pl.gram_items += (int64_t)a.n_frames * (nt * (nt + 1) / 2);
    vis_end = std::max(vis_end, a.vis_off + nv);
    aud_end = std::max(aud_end, a.aud_off + a.n_audio);
    pl.max_per_frame = std::max(pl.max_per_frame, a.tokens_per_frame);
    pl.clips.push_back(c);
  }
  // Spatial CKA: one 16 x 16 tile per upper-triangle block of the stacked
  // [co-timed audio; visual] rows of a frame, sized for the largest frame.
  if (p->alignment == APACK_ALIGN_SPATIAL_CKA) {
    int64_t m = 0;
    for (int s = 0; s < n_seq; ++s) {
      const apack_av_seq& a = seqs[s];
      if (a.n_frames == 0) continue;
      m = std::max<int64_t>(m, (a.n_audio + a.n_frames - 1) / a.n_frames + 1 + a.tokens_per_frame);
    }
    const int64_t nt = (m + 15) / 16;
    pl.spatial_tiles = (int32_t)(nt * (nt + 1) / 2);
  }
  pl.total_frames = frames;
  pl.total_tokens = vis_end;
  pl.total_audio = aud_end;
  pl.total_kept = kept;
  pl.total_gram = gram;
  // Gate GEMM tiles: columns (visual) in groups of eight share an XCD.
  std::vector<GemmTileDev> tiles;
  for (int s = 0; s < n_seq; ++s) {
    const ClipDev& c = pl.clips[s];
    const int64_t nv = (int64_t)c.n_frames * c.per_frame;
    if (nv == 0) continue;
    const int mb = (int)((c.n_audio + 127) / 128), nb = (int)((nv + 127) / 128);
    for (int g0 = 0; g0 < nb; g0 += 8)
      for (int m = 0; m < mb; ++m)
        for (int n = g0; n < std::min(g0 + 8, nb); ++n) tiles.push_back({s, m * 128, n * 128, 0});
  }
  pl.gemm_tiles = (int64_t)tiles.size();
  if (dim % kGemm256K == 0) pl.gemm256 = gate_gemm256_tiles(pl.clips);
  // The blob holds whichever list the call uses.
  const size_t n_tiles = std::max(tiles.size(), pl.gemm256.size());
  // Workspace layout.
  const int64_t nc = n_seq;
  Carver c(nullptr);
  c.take<ClipDev>(nc);
  pl.off_frames = c.used;
  c.take<FrameDev>(pl.frames.size());
  pl.off_gemm = c.used;
  c.take<GemmTileDev>(n_tiles);
  pl.blob_bytes = c.used;
  pl.off_v = c.used;
  c.take<double>(frames * dim);
  pl.off_a = c.used;
  c.take<double>(frames * dim);
  pl.off_q = c.used;
  c.take<double>(nc * dim);
  pl.off_band_v = c.used;
  c.take<double>(frames * kMaxWindow);
  pl.off_band_a = c.used;
  c.take<double>(frames * kMaxWindow);
  pl.off_vq = c.used;
  c.take<double>(frames);
  pl.off_qq = c.used;
  c.take<double>(nc);
  pl.off_cka = c.used;
  c.take<double>(frames);
  pl.off_nv = c.used;
  c.take<double>(vis_end);
  pl.off_rv = c.used;
  c.take<double>(vis_end);
  pl.off_na = c.used;
  c.take<double>(aud_end);
  pl.off_maxkey = c.used;
  c.take<uint32_t>(vis_end);
  pl.off_plan = c.used;
  c.take<FramePlanDev>(frames);
  pl.off_gram = c.used;
  c.take<double>(gram);
  pl.off_scratch = c.used;
  c.take<double>(16 * (frames + nc + 1));
  pl.off_sim = c.used;
  c.take<double>(tokens);
  pl.off_spatial = c.used;
  c.take<double>((size_t)frames * pl.spatial_tiles * 3);
  pl.off_anchors = c.used;
  c.take<int32_t>(frames);
  pl.off_sqp = c.used;
  c.take<double>((size_t)((dim + kPoolSlice - 1) / kPoolSlice) * (vis_end + aud_end));
  pl.ws_bytes = std::max<size_t>(c.used, kAlign);
  pl.gemm = std::move(tiles);
  return APACK_OK;
}

}  // namespace apack

using namespace apack;

extern "C" {

apack_status apack_score_dynamics_query(int32_t n_seq, const apack_av_seq* seqs, int32_t dim,
                                        const apack_dyn_params* p, int64_t* n_kept_visual,
                                        size_t* workspace_bytes) {
  clear_error();
  DynPlan pl;
  apack_status st = build_dyn_plan(n_seq, seqs, dim, p, pl);
  if (st != APACK_OK) return st;
  if (n_kept_visual)
    for (int s = 0; s < n_seq; ++s) n_kept_visual[s] = pl.budgets[s];
  if (workspace_bytes) *workspace_bytes = pl.ws_bytes;
  return APACK_OK;
}

apack_status apack_score_dynamics(int32_t n_seq, const apack_av_seq* seqs, apack_dtype dtype, int32_t dim,
                                  const void* visual, int64_t visual_rows, const void* audio,
                                  int64_t audio_rows, const void* query, int64_t query_rows,
                                  const apack_dyn_params* p, float* frame_cka, float* frame_score,
                                  int32_t* frame_budget, int32_t* segment_id, uint8_t* gate_fired,
                                  int32_t* kept_visual, int64_t kept_capacity, int64_t* n_kept_visual,
                                  void* workspace, size_t workspace_bytes, void* stream) {
  clear_error();
  APACK_CHECK(dtype_ok(dtype), APACK_E_DTYPE, "unknown dtype %d", (int)dtype);
  DynPlan pl;
  apack_status st = build_dyn_plan(n_seq, seqs, dim, p, pl);
  if (st != APACK_OK) return st;
  const size_t es = dtype_size(dtype);
  APACK_CHECK(visual_rows >= 0 && audio_rows >= 0 && query_rows >= 0, APACK_E_SHAPE, "negative row count");
  for (int s = 0; s < n_seq; ++s) {
    const apack_av_seq& a = seqs[s];
    APACK_CHECK(a.vis_off + (int64_t)a.n_frames * a.tokens_per_frame <= visual_rows, APACK_E_SHAPE,
                "clip %d: visual rows exceed visual_rows", s);
    APACK_CHECK(a.aud_off + a.n_audio <= audio_rows, APACK_E_SHAPE, "clip %d: audio rows exceed audio_rows", s);
    APACK_CHECK(a.qry_off + a.n_query <= query_rows, APACK_E_SHAPE, "clip %d: query rows exceed query_rows", s);
  }
  APACK_CHECK(kept_capacity >= pl.total_kept, APACK_E_SHAPE, "kept_capacity %lld < %lld kept visual rows",
              (long long)kept_capacity, (long long)pl.total_kept);
  if (n_kept_visual)
    for (int s = 0; s < n_seq; ++s) n_kept_visual[s] = pl.budgets[s];
  if (n_seq == 0) return APACK_OK;
  APACK_CHECK(visual && audio && query, APACK_E_ARG, "visual, audio and query must be non-NULL");
  APACK_CHECK(pl.total_kept == 0 || kept_visual, APACK_E_ARG, "kept_visual is NULL");
  auto al16 = [](const void* q) { return ((uintptr_t)q % 16) == 0; };
  APACK_CHECK(al16(visual) && al16(audio) && al16(query), APACK_E_ARG, "inputs must be 16-byte aligned");
  const size_t vb = (size_t)visual_rows * dim * es, ab = (size_t)audio_rows * dim * es,
               qb = (size_t)query_rows * dim * es;
  const int64_t nf = pl.total_frames;
  const std::pair<const void*, size_t> outs[] = {{frame_cka, (size_t)nf * 4},   {frame_score, (size_t)nf * 4},
                                                 {frame_budget, (size_t)nf * 4}, {segment_id, (size_t)nf * 4},
                                                 {gate_fired, (size_t)n_seq},    {kept_visual, (size_t)pl.total_kept * 4}};
  for (size_t i = 0; i < sizeof outs / sizeof outs[0]; ++i) {
    const auto& o = outs[i];
    if (!o.first) continue;
    APACK_CHECK(!overlaps(o.first, o.second, visual, vb) && !overlaps(o.first, o.second, audio, ab) &&
                    !overlaps(o.first, o.second, query, qb),
                APACK_E_ALIAS, "an output overlaps an input");
    for (size_t j = 0; j < i; ++j)
      APACK_CHECK(!outs[j].first || !overlaps(o.first, o.second, outs[j].first, outs[j].second), APACK_E_ALIAS,
                  "two outputs overlap");
  }
  APACK_CHECK(workspace && ((uintptr_t)workspace % kAlign) == 0, APACK_E_WORKSPACE,
              "workspace must be non-NULL and %zu-byte aligned", kAlign);
  APACK_CHECK(workspace_bytes >= pl.ws_bytes, APACK_E_WORKSPACE, "workspace of %zu bytes < %zu needed",
              workspace_bytes, pl.ws_bytes);

  // bf16 inputs with dim a multiple of 64 take the 256 x 256 gate GEMM.
  if (dtype == APACK_BF16 && !pl.gemm256.empty()) {
    pl.use256 = true;
    pl.gemm = pl.gemm256;
    pl.gemm_tiles = (int64_t)pl.gemm.size();
  }
  Staging* blk;
  void* host;
  if ((st = staging_acquire(pl.blob_bytes, &blk, &host)) != APACK_OK) return st;
  char* h = static_cast<char*>(host);
  std::memcpy(h, pl.clips.data(), pl.clips.size() * sizeof(ClipDev));
  if (!pl.frames.empty()) std::memcpy(h + pl.off_frames, pl.frames.data(), pl.frames.size() * sizeof(FrameDev));
  if (pl.gemm_tiles) std::memcpy(h + pl.off_gemm, pl.gemm.data(), pl.gemm.size() * sizeof(GemmTileDev));
  hipStream_t hs = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  if ((st = staging_upload(blk, ws, pl.blob_bytes, hs)) != APACK_OK) return st;
  DynPtrs dp;
  dp.clips = reinterpret_cast<ClipDev*>(ws);
  dp.frames = reinterpret_cast<FrameDev*>(ws + pl.off_frames);
  dp.gemm = reinterpret_cast<GemmTileDev*>(ws + pl.off_gemm);
  dp.v = reinterpret_cast<double*>(ws + pl.off_v);
  dp.a = reinterpret_cast<double*>(ws + pl.off_a);
  dp.q = reinterpret_cast<double*>(ws + pl.off_q);
  dp.band_v = reinterpret_cast<double*>(ws + pl.off_band_v);
  dp.band_a = reinterpret_cast<double*>(ws + pl.off_band_a);
  dp.vq = reinterpret_cast<double*>(ws + pl.off_vq);
  dp.qq = reinterpret_cast<double*>(ws + pl.off_qq);
  dp.cka = reinterpret_cast<double*>(ws + pl.off_cka);
  dp.nv = reinterpret_cast<double*>(ws + pl.off_nv);
  dp.rv = reinterpret_cast<double*>(ws + pl.off_rv);
  dp.na = reinterpret_cast<double*>(ws + pl.off_na);
  dp.maxkey = reinterpret_cast<uint32_t*>(ws + pl.off_maxkey);
  dp.plan = reinterpret_cast<FramePlanDev*>(ws + pl.off_plan);
  dp.gram = reinterpret_cast<double*>(ws + pl.off_gram);
  dp.scratch = reinterpret_cast<double*>(ws + pl.off_scratch);
  dp.spatial = reinterpret_cast<double*>(ws + pl.off_spatial);
  dp.sim = reinterpret_cast<double*>(ws + pl.off_sim);
  dp.anchors = reinterpret_cast<int32_t*>(ws + pl.off_anchors);
  dp.sqp = reinterpret_cast<double*>(ws + pl.off_sqp);
  DynParamsDev prm;
  prm.tau_gate = p->tau_gate;
  prm.beta = p->beta;
  prm.gamma = p->gamma;
  prm.tau_sim = p->tau_sim;
  prm.sigma = p->sigma;
  prm.lambda_seg = p->lambda_seg;
  prm.cover = p->cover_thresh;
  prm.power = p->dafps_power;
  prm.window = p->window;
  prm.dafps_k = p->dafps_k;
  prm.alignment = p->alignment;
  // AV cosine is the fine-pass term alone: the Eq. 2 blend with beta = 1.
  if (p->alignment == APACK_ALIGN_AV_COSINE) prm.beta = 1.0;
  const apack_status ls = launch_dynamics(pl, dp, prm, dtype, dim, visual, audio, query, pl.total_tokens,
                                          pl.total_audio, frame_cka, frame_score, frame_budget, segment_id, gate_fired,
                                          kept_visual, hs);
  const apack_status rs = staging_release(blk, hs);
  return ls != APACK_OK ? ls : rs;
}

}  // extern "C"
