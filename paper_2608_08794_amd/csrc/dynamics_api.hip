// Host side of apack_score_dynamics (pre-LLM scorer, Section 3.1).
#include "common.hpp"

using namespace apack;

extern "C" {

apack_status apack_score_dynamics_query(int32_t n_seq, const apack_av_seq* seqs, int32_t dim,
                                        const apack_dyn_params* p, int64_t* n_kept_visual,
                                        size_t* workspace_bytes) {
  clear_error();
  (void)n_seq; (void)seqs; (void)dim; (void)p; (void)n_kept_visual; (void)workspace_bytes;
  return fail(APACK_E_UNSUPPORTED, "apack_score_dynamics is not built yet");
}

apack_status apack_score_dynamics(int32_t n_seq, const apack_av_seq* seqs, apack_dtype dtype, int32_t dim,
                                  const void* visual, int64_t visual_rows, const void* audio,
                                  int64_t audio_rows, const void* query, int64_t query_rows,
                                  const apack_dyn_params* p, float* frame_cka, float* frame_score,
                                  int32_t* frame_budget, int32_t* segment_id, uint8_t* gate_fired,
                                  int32_t* kept_visual, int64_t kept_capacity, int64_t* n_kept_visual,
                                  void* workspace, size_t workspace_bytes, void* stream) {
  clear_error();
  return fail(APACK_E_UNSUPPORTED, "apack_score_dynamics is not built yet");
}

}  // extern "C"
