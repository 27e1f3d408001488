// Analytic prefill-FLOPs accounting (Appendix G): the compute a token-length
// schedule implies, so a caller can state what a run of the prune path saves.
// Host-only arithmetic; nothing here touches the device.
#include <cmath>

#include "common.hpp"

using namespace apack;

extern "C" {

double apack_layer_flops(int64_t n, int64_t d_model, int64_t d_ffn) {
  if (n < 0 || d_model < 0 || d_ffn < 0) return -1.0;
  const double nn = (double)n, d = (double)d_model, m = (double)d_ffn;
  // Q, K, V and O projections; quadratic attention; feed-forward block.
  return 4.0 * nn * d * d + 2.0 * nn * nn * d + 2.0 * nn * d * m;
}

apack_status apack_prefill_flops(int32_t n_layers, const int64_t* lengths, int64_t n0, int64_t d_model,
                                 int64_t d_ffn, double* f_pre, double* ratio) {
  clear_error();
  APACK_CHECK(n_layers > 0 && lengths, APACK_E_ARG, "need at least one layer length");
  APACK_CHECK(n0 > 0 && d_model > 0 && d_ffn > 0, APACK_E_ARG, "n0, d_model and d_ffn must be positive");
  double sum = 0.0;
  for (int32_t i = 0; i < n_layers; ++i) {
    APACK_CHECK(lengths[i] >= 0, APACK_E_ARG, "layer %d: negative length", i);
    sum += apack_layer_flops(lengths[i], d_model, d_ffn);
  }
  if (f_pre) *f_pre = sum;
  if (ratio) *ratio = sum / ((double)n_layers * apack_layer_flops(n0, d_model, d_ffn));
  return APACK_OK;
}

apack_status apack_schedule_lengths(int32_t n_layers, int64_t n_start, int32_t n_prunes, const int32_t* prune_layers,
                                    const int64_t* n_after, int64_t* lengths) {
  clear_error();
  APACK_CHECK(n_layers > 0 && lengths, APACK_E_ARG, "need at least one layer");
  APACK_CHECK(n_start >= 0, APACK_E_ARG, "negative start length");
  APACK_CHECK(n_prunes >= 0 && (n_prunes == 0 || (prune_layers && n_after)), APACK_E_ARG,
              "prune_layers and n_after must be given for n_prunes > 0");
  for (int32_t j = 0; j < n_prunes; ++j) {
    APACK_CHECK(prune_layers[j] >= 0 && prune_layers[j] < n_layers, APACK_E_ARG,
                "prune %d: layer %d outside [0, %d)", j, prune_layers[j], n_layers);
    APACK_CHECK(j == 0 || prune_layers[j] > prune_layers[j - 1], APACK_E_ARG,
                "prune layers must be strictly increasing");
    APACK_CHECK(n_after[j] >= 0, APACK_E_ARG, "prune %d: negative length", j);
  }
  int64_t n = n_start;
  int32_t j = 0;
  for (int32_t i = 0; i < n_layers; ++i) {
    lengths[i] = n;
    // A prune scores with layer i's attention and shortens what enters i + 1.
    if (j < n_prunes && prune_layers[j] == i) n = n_after[j++];
  }
  return APACK_OK;
}

}  // extern "C"
