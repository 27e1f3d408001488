// Host plan and device descriptors of one apack_prune_layer call.
#pragma once

#include <cstdint>
#include <vector>

#include "common.hpp"

namespace apack {

#ifndef APACK_KEY_TILE
#define APACK_KEY_TILE 128
#endif
#ifndef APACK_ROW_BLOCKS
#define APACK_ROW_BLOCKS 2
#endif
#ifndef APACK_TILE_TARGET
#define APACK_TILE_TARGET 256
#endif
constexpr int kKeyTile = APACK_KEY_TILE;       // keys per LDS stage of the score kernels
constexpr int kRB = APACK_ROW_BLOCKS;          // 32-row query blocks held by one wave
constexpr int kRowsPerWave = 32 * kRB;
constexpr int kMaxWaves = 8;                   // waves per score workgroup
#ifndef APACK_MAX_CHUNK
#define APACK_MAX_CHUNK 4096
#endif
constexpr int kMaxChunk = APACK_MAX_CHUNK;    // keys per score workgroup, at most
constexpr int kRowTile = 1024;   // rows per workgroup of the select and compaction kernels

// Per-sequence descriptor on the device (uploaded once per call).  The
// select kernel fills thr / need / all_eq for modalities it ranks.
struct SeqDev {
  int64_t tok_off;      // first packed row of the sequence in K / scores
  int64_t n_tokens;
  int64_t q_off;        // first packed query row
  int64_t out_off;      // first slot in kept_rows
  int64_t n_kept;       // kept rows of the sequence (bound on the scan's writes)
  int64_t tag_off;      // first byte of the sequence in the tag array
  int64_t stats_off;    // first (max, sum) partial: [g][chunk][rows_pad]
  int64_t colpart_off;  // first per-group column partial: [g*n_rg + rg][n_tokens]
  int32_t q_len;
  int32_t n_rg;         // query-row groups per KV head
  int32_t rows_per_rg;  // rows per group (multiple of 64)
  int32_t rows_pad;     // n_rg * rows_per_rg
  int32_t chunk;        // keys per score workgroup (multiple of kKeyTile)
  int32_t n_chunks;
  int32_t n_cand;
  int32_t k_sel[2];     // keep count per modality (audio, visual)
  int32_t n_mod[2];     // candidate count per modality
  int32_t select[2];    // 1 when a radix select is needed (0 < k < n)
  uint32_t thr[2];      // threshold bits: rows above are kept
  int32_t need[2];      // rows equal to thr kept, lowest rows first
  int32_t all_eq[2];    // every row equal to thr is kept
  uint32_t prefix[2];   // radix digits chosen so far
  uint32_t kk[2];       // rank of the k-th value inside the chosen bucket
  uint32_t done_cnt;    // row tiles finished in the current select pass
  int32_t n_ftiles;     // row tiles of the sequence
  int32_t ctr_off;      // arrival counters: [n_chunks key chunks][1 sequence]
};

struct FTileDev {
  int32_t seq, idx;     // sequence and row tile within it (rows idx*kRowTile ...)
};

struct TileDev {
  int32_t seq, g, rg, chunk;
};

struct PrunePlan {
  std::vector<SeqDev> seqs;
  std::vector<TileDev> tiles;
  std::vector<FTileDev> ftiles;
  std::vector<int64_t> n_kept;
  int64_t total_tok = 0;    // sum of n_tokens (tag bytes)
  int64_t max_tokens = 0;   // longest sequence
  int64_t total_stats = 0;  // (max, sum) partials
  int64_t total_colpart = 0;
  int64_t total_kept = 0;
  int64_t total_ctr = 0;    // arrival counters (zeroed by the upload)
  int waves = 1;
  bool any_select = false;
  // Workspace layout (byte offsets).
  size_t off_seqs = 0, off_tiles = 0, off_ftiles = 0, off_tags = 0, off_ctr = 0, blob_bytes = 0;
  size_t off_stats = 0, off_colpart = 0, off_hist = 0, off_cnt = 0, ws_bytes = 0;
};

struct DevPtrs {
  SeqDev* seqs;
  TileDev* tiles;
  uint8_t* tags;
  FTileDev* ftiles;
  float2* stats;
  float* colpart;
  uint32_t* hist;       // [n_seq][2][2048] radix histograms
  uint32_t* cnt;        // [n_ftiles][3] per-tile keep counts
  uint32_t* ctr;        // arrival counters of the score kernels
};

apack_status build_prune_plan(int32_t n_seq, const apack_seq* seqs, int32_t hq, int32_t hkv, int32_t d,
                              PrunePlan& plan);

int64_t select_hist_words(int64_t n_seq);   // radix histogram words of n_seq sequences

apack_status launch_select(const PrunePlan& pl, const DevPtrs& dp, float* scores, int32_t* kept,
                           hipStream_t stream);

apack_status launch_prune(const PrunePlan& pl, const DevPtrs& dp, apack_dtype dt, int d, int hq, int hkv,
                          const void* q, int64_t q_hs, const void* k, int64_t k_hs, float* scores,
                          int32_t* kept, hipStream_t stream);

}  // namespace apack
