// Host side of apack_prune_layer: validation, planning, descriptor upload and
// the launch sequence.  Everything here runs before the first enqueue, so a
// rejected call has no device-side effect.
#include <algorithm>
#include <cmath>
#include <cstring>

#include "common.hpp"
#include "prune_plan.hpp"

namespace apack {

apack_status build_prune_plan(int32_t n_seq, const apack_seq* seqs, int32_t hq, int32_t hkv, int32_t d,
                              PrunePlan& pl) {
  APACK_CHECK(n_seq >= 0, APACK_E_ARG, "n_seq must be >= 0 (got %d)", n_seq);
  APACK_CHECK(n_seq == 0 || seqs, APACK_E_ARG, "seqs is NULL");
  APACK_CHECK(hq > 0 && hkv > 0 && hq % hkv == 0, APACK_E_SHAPE,
              "hq (%d) must be a positive multiple of hkv (%d)", hq, hkv);
  APACK_CHECK(d == 64 || d == 128, APACK_E_UNSUPPORTED, "head dim %d not built (64 or 128)", d);
  const int n_rep = hq / hkv;
  pl = PrunePlan();
  pl.seqs.resize(n_seq);
  pl.n_kept.resize(n_seq);
  int64_t tag = 0, stats = 0, colpart = 0, kept = 0;
  int waves = 1;
  // Total work units so the chunk length can target a few workgroups per CU.
  int64_t weighted = 0;
  for (int s = 0; s < n_seq; ++s) {
    const apack_seq& a = seqs[s];
    APACK_CHECK(a.n_tokens >= 0 && a.tok_off >= 0, APACK_E_SHAPE, "seq %d: negative offset or length", s);
    APACK_CHECK(a.n_tokens < (int64_t(1) << 31), APACK_E_UNSUPPORTED, "seq %d: n_tokens >= 2^31", s);
    APACK_CHECK(a.q_len >= 1 && a.q_len <= 65536 && a.q_off >= 0, APACK_E_SHAPE,
                "seq %d: q_len must lie in [1, 65536] (got %lld)", s, (long long)a.q_len);
    APACK_CHECK(a.flags == 0 || a.flags == APACK_RANK_JOINT, APACK_E_ARG, "seq %d: unknown flags %d", s,
                (int)a.flags);
    const bool joint = a.flags == APACK_RANK_JOINT;
    APACK_CHECK(!joint || (a.keep[1] == 0.0 && a.keep_basis[1] == 0), APACK_E_ARG,
                "seq %d: joint ranking takes keep[0] and keep_basis[0]; keep[1] and keep_basis[1] must be 0", s);
    APACK_CHECK(a.n_spans >= 0 && (a.n_spans == 0 || a.spans), APACK_E_ARG, "seq %d: spans is NULL", s);
    int64_t cnt[2] = {0, 0};
    int64_t prev_end = 0;
    for (int i = 0; i < a.n_spans; ++i) {
      const apack_span& sp = a.spans[i];
      APACK_CHECK(sp.reserved == 0, APACK_E_ARG, "seq %d span %d: reserved field must be 0", s, i);
      APACK_CHECK(sp.modality >= APACK_OTHER && sp.modality <= APACK_VISUAL, APACK_E_ARG,
                  "seq %d span %d: bad modality %d", s, i, sp.modality);
      APACK_CHECK(sp.begin >= prev_end && sp.len >= 0 && sp.begin + sp.len <= a.n_tokens, APACK_E_SHAPE,
                  "seq %d span %d: spans must be ascending, disjoint and inside [0, %lld)", s, i,
                  (long long)a.n_tokens);
      prev_end = sp.begin + sp.len;
      if (sp.modality != APACK_OTHER) cnt[joint ? 0 : sp.modality - 1] += sp.len;
    }
    SeqDev& sd = pl.seqs[s];
    std::memset(&sd, 0, sizeof sd);
    sd.tok_off = a.tok_off;
    sd.n_tokens = a.n_tokens;
    sd.q_off = a.q_off;
    sd.q_len = (int32_t)a.q_len;
    int64_t k_m[2];
    for (int m = 0; m < 2; ++m) {
      APACK_CHECK(a.keep[m] >= 0.0 && a.keep[m] <= 1.0, APACK_E_ARG,
                  "seq %d: keep[%d] = %g outside [0, 1]", s, m, a.keep[m]);
      APACK_CHECK(a.keep_basis[m] >= 0, APACK_E_ARG, "seq %d: keep_basis[%d] < 0", s, m);
      const int64_t basis = a.keep_basis[m] ? a.keep_basis[m] : cnt[m];
      k_m[m] = apack_keep_count(a.keep[m], basis);
      APACK_CHECK(k_m[m] >= 0 && k_m[m] <= cnt[m], APACK_E_ARG,
                  "seq %d: keep count %lld for modality %d exceeds its %lld candidates", s,
                  (long long)k_m[m], m + 1, (long long)cnt[m]);
      sd.k_sel[m] = (int32_t)k_m[m];
      sd.n_mod[m] = (int32_t)cnt[m];
      sd.select[m] = (k_m[m] > 0 && k_m[m] < cnt[m]) ? 1 : 0;
      if (k_m[m] == 0) {
        sd.thr[m] = 0xFFFFFFFFu;
        sd.need[m] = 0;
      } else {
        sd.thr[m] = 0u;  // k == n: every row is above or equal to 0
        sd.need[m] = (int32_t)cnt[m];
      }
      sd.all_eq[m] = 1;
      sd.kk[m] = (uint32_t)k_m[m];
      pl.any_select |= sd.select[m] != 0;
    }
    sd.n_cand = (int32_t)(cnt[0] + cnt[1]);
    const int64_t n_other = a.n_tokens - cnt[0] - cnt[1];
    pl.n_kept[s] = n_other + k_m[0] + k_m[1];
    sd.out_off = kept;
    sd.n_kept = pl.n_kept[s];
    kept += pl.n_kept[s];
    sd.tag_off = tag;
    tag += a.n_tokens;
    sd.n_ftiles = (int32_t)((a.n_tokens + kRowTile - 1) / kRowTile);
    for (int f = 0; f < sd.n_ftiles; ++f) pl.ftiles.push_back({s, f});
    pl.max_tokens = std::max<int64_t>(pl.max_tokens, a.n_tokens);
    // Query-row groups: at most kMaxWaves * kRowsPerWave rows each.
    const int64_t rows_g = (int64_t)n_rep * a.q_len;
    const int64_t cap = (int64_t)kMaxWaves * kRowsPerWave;
    sd.n_rg = (int32_t)((rows_g + cap - 1) / cap);
    const int64_t per = (rows_g + sd.n_rg - 1) / sd.n_rg;
    sd.rows_per_rg = (int32_t)((per + kRowsPerWave - 1) / kRowsPerWave * kRowsPerWave);
    sd.rows_pad = sd.n_rg * sd.rows_per_rg;
    waves = std::max<int>(waves, sd.rows_per_rg / kRowsPerWave);
    if (sd.n_cand > 0) weighted += a.n_tokens * (int64_t)hkv * sd.n_rg;
  }
  // Sequences may not overlap in K (their scores would collide).
  {
    std::vector<std::pair<int64_t, int64_t>> r;
    for (int s = 0; s < n_seq; ++s)
      if (seqs[s].n_tokens) r.emplace_back(seqs[s].tok_off, seqs[s].tok_off + seqs[s].n_tokens);
    std::sort(r.begin(), r.end());
    for (size_t i = 1; i < r.size(); ++i)
      APACK_CHECK(r[i].first >= r[i - 1].second, APACK_E_SHAPE, "sequences overlap in k");
  }
  // Keys per workgroup: about one score workgroup per CU over the whole
  // call (one 7- or 8-wave workgroup fills a CU), so the chip runs a single
  // round and each workgroup loads its query fragments once.
  const int64_t target = APACK_TILE_TARGET;
  for (int s = 0; s < n_seq; ++s) {
    SeqDev& sd = pl.seqs[s];
    if (sd.n_cand == 0) continue;
    int64_t ch = (weighted + target - 1) / target;
    ch = (ch + kKeyTile - 1) / kKeyTile * kKeyTile;
    ch = std::max<int64_t>(kKeyTile, std::min<int64_t>(ch, kMaxChunk));
    sd.chunk = (int32_t)ch;
    sd.n_chunks = (int32_t)((sd.n_tokens + ch - 1) / ch);
    sd.stats_off = stats;
    stats += (int64_t)hkv * sd.rows_pad * sd.n_chunks;
    sd.colpart_off = colpart;
    colpart += (int64_t)hkv * sd.n_rg * sd.n_tokens;
    sd.ctr_off = (int32_t)pl.total_ctr;
    pl.total_ctr += sd.n_chunks + 1;
    // Tiles: chunks of one (g, rg) eight apart so that both query-row
    // groups of a key chunk land on the same XCD's L2.
    for (int g = 0; g < hkv; ++g)
      for (int c0 = 0; c0 < sd.n_chunks; c0 += 8)
        for (int rg = 0; rg < sd.n_rg; ++rg)
          for (int c = c0; c < std::min(c0 + 8, sd.n_chunks); ++c) pl.tiles.push_back({s, g, rg, c});
  }
  pl.waves = waves <= 1 ? 1 : waves <= 2 ? 2 : waves <= 4 ? 4 : waves == 7 ? 7 : 8;
  pl.total_tok = tag;
  pl.total_stats = stats;
  pl.total_colpart = colpart;
  pl.total_kept = kept;
  // Workspace layout.
  Carver c(nullptr);
  c.take<SeqDev>(pl.seqs.size());
  pl.off_tiles = c.used;
  c.take<TileDev>(pl.tiles.size());
  pl.off_ftiles = c.used;
  c.take<FTileDev>(pl.ftiles.size());
  pl.off_tags = c.used;
  c.take<uint8_t>(pl.total_tok);
  pl.off_ctr = c.used;
  c.take<uint32_t>(pl.total_ctr);
  pl.blob_bytes = c.used;
  pl.off_stats = c.used;
  c.take<float2>(pl.total_stats);
  pl.off_colpart = c.used;
  c.take<float>(pl.total_colpart);
  pl.off_hist = c.used;
  c.take<uint32_t>(pl.any_select ? select_hist_words((int64_t)pl.seqs.size()) : 0);
  pl.off_cnt = c.used;
  c.take<uint32_t>(3 * pl.ftiles.size());
  pl.ws_bytes = std::max<size_t>(c.used, kAlign);
  return APACK_OK;
}

}  // namespace apack

using namespace apack;

extern "C" {

apack_status apack_prune_layer_query(int32_t n_seq, const apack_seq* seqs, int32_t hq, int32_t hkv,
                                     int32_t d, int64_t* n_kept, size_t* workspace_bytes) {
  clear_error();
  PrunePlan pl;
  apack_status st = build_prune_plan(n_seq, seqs, hq, hkv, d, pl);
  if (st != APACK_OK) return st;
  if (n_kept)
    for (int s = 0; s < n_seq; ++s) n_kept[s] = pl.n_kept[s];
  if (workspace_bytes) *workspace_bytes = pl.ws_bytes;
  return APACK_OK;
}

apack_status apack_prune_layer(int32_t n_seq, const apack_seq* seqs, apack_dtype dtype, int32_t hq,
                               int32_t hkv, int32_t d, const void* q, int64_t q_head_stride, int64_t q_rows,
                               const void* k, int64_t k_head_stride, int64_t k_rows, float* scores,
                               int32_t* kept_rows, int64_t kept_capacity, int64_t* n_kept, void* workspace,
                               size_t workspace_bytes, void* stream) {
  clear_error();
  APACK_CHECK(dtype_ok(dtype), APACK_E_DTYPE, "unknown dtype %d", (int)dtype);
  PrunePlan pl;
  apack_status st = build_prune_plan(n_seq, seqs, hq, hkv, d, pl);
  if (st != APACK_OK) return st;
  const size_t es = dtype_size(dtype);
  APACK_CHECK(q_rows >= 0 && k_rows >= 0, APACK_E_SHAPE, "negative row count");
  APACK_CHECK(q_head_stride >= q_rows * d && k_head_stride >= k_rows * d, APACK_E_SHAPE,
              "head strides must be >= rows * d");
  for (int s = 0; s < n_seq; ++s) {
    APACK_CHECK(seqs[s].q_off + seqs[s].q_len <= q_rows, APACK_E_SHAPE, "seq %d: query rows exceed q_rows", s);
    APACK_CHECK(seqs[s].tok_off + seqs[s].n_tokens <= k_rows, APACK_E_SHAPE, "seq %d: rows exceed k_rows", s);
  }
  APACK_CHECK(kept_capacity >= pl.total_kept, APACK_E_SHAPE, "kept_capacity %lld < %lld kept rows",
              (long long)kept_capacity, (long long)pl.total_kept);
  if (pl.total_tok > 0) {
    APACK_CHECK(q && k && scores && kept_rows, APACK_E_ARG, "q, k, scores and kept_rows must be non-NULL");
    APACK_CHECK(((uintptr_t)q % 16) == 0 && ((uintptr_t)k % 16) == 0 && (q_head_stride * es) % 16 == 0 &&
                    (k_head_stride * es) % 16 == 0,
                APACK_E_ARG, "q, k and their head strides must be 16-byte aligned");
    APACK_CHECK(((uintptr_t)scores % 4) == 0 && ((uintptr_t)kept_rows % 4) == 0, APACK_E_ARG,
                "scores and kept_rows must be 4-byte aligned");
    const size_t kbytes = (size_t)((hkv - 1) * k_head_stride + k_rows * d) * es;
    const size_t qbytes = (size_t)((hq - 1) * q_head_stride + q_rows * d) * es;
    APACK_CHECK(!overlaps(scores, k_rows * 4, k, kbytes) && !overlaps(scores, k_rows * 4, q, qbytes) &&
                    !overlaps(kept_rows, pl.total_kept * 4, k, kbytes) &&
                    !overlaps(kept_rows, pl.total_kept * 4, scores, k_rows * 4),
                APACK_E_ALIAS, "outputs overlap inputs");
  }
  APACK_CHECK(workspace && ((uintptr_t)workspace % kAlign) == 0, APACK_E_WORKSPACE,
              "workspace must be non-NULL and %zu-byte aligned", kAlign);
  APACK_CHECK(workspace_bytes >= pl.ws_bytes, APACK_E_WORKSPACE, "workspace of %zu bytes < %zu needed",
              workspace_bytes, pl.ws_bytes);
  if (n_kept)
    for (int s = 0; s < n_seq; ++s) n_kept[s] = pl.n_kept[s];
  if (pl.total_tok == 0) return APACK_OK;

  // Host blob: sequence descriptors, tiles and per-row modality tags.
  Staging* blk;
  void* host;
  if ((st = staging_acquire(pl.blob_bytes, &blk, &host)) != APACK_OK) return st;
  char* h = static_cast<char*>(host);
  std::memcpy(h, pl.seqs.data(), pl.seqs.size() * sizeof(SeqDev));
  if (!pl.tiles.empty()) std::memcpy(h + pl.off_tiles, pl.tiles.data(), pl.tiles.size() * sizeof(TileDev));
  if (!pl.ftiles.empty())
    std::memcpy(h + pl.off_ftiles, pl.ftiles.data(), pl.ftiles.size() * sizeof(FTileDev));
  uint8_t* tags = reinterpret_cast<uint8_t*>(h + pl.off_tags);
  std::memset(tags, 0, pl.total_tok);
  // Tag = selection slot + 1: the modality, or slot 1 for every candidate of
  // a jointly ranked sequence.
  for (int s = 0; s < n_seq; ++s)
    for (int i = 0; i < seqs[s].n_spans; ++i) {
      const apack_span& sp = seqs[s].spans[i];
      if (sp.modality != APACK_OTHER)
        std::memset(tags + pl.seqs[s].tag_off + sp.begin, seqs[s].flags == APACK_RANK_JOINT ? 1 : sp.modality,
                    (size_t)sp.len);
    }
  std::memset(h + pl.off_ctr, 0, pl.total_ctr * sizeof(uint32_t));
  hipStream_t hs = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  if ((st = staging_upload(blk, ws, pl.blob_bytes, hs)) != APACK_OK) return st;
  DevPtrs dp;
  dp.seqs = reinterpret_cast<SeqDev*>(ws);
  dp.tiles = reinterpret_cast<TileDev*>(ws + pl.off_tiles);
  dp.ftiles = reinterpret_cast<FTileDev*>(ws + pl.off_ftiles);
  dp.hist = reinterpret_cast<uint32_t*>(ws + pl.off_hist);
  dp.cnt = reinterpret_cast<uint32_t*>(ws + pl.off_cnt);
  dp.ctr = reinterpret_cast<uint32_t*>(ws + pl.off_ctr);
  dp.tags = reinterpret_cast<uint8_t*>(ws + pl.off_tags);
  dp.stats = reinterpret_cast<float2*>(ws + pl.off_stats);
  dp.colpart = reinterpret_cast<float*>(ws + pl.off_colpart);
  const apack_status ls = launch_prune(pl, dp, dtype, d, hq, hkv, q, q_head_stride, k, k_head_stride, scores,
                                       kept_rows, hs);
  const apack_status rs = staging_release(blk, hs);
  return ls != APACK_OK ? ls : rs;
}

}  // extern "C"
