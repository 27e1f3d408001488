/*
 * apack.h -- C ABI of the A-PACK hot path on MI355X (gfx950).
 *
 * Two halves of the method of "Deferred Audio Pruning with Local Audio-Visual
 * Dynamics for Omni-LLMs":
 *
 *   apack_score_dynamics  pre-LLM local audio-visual dynamics scorer
 *                         (Section 3.1, Eq. 1-4; Algorithm 1, first loop)
 *   apack_prune_layer     in-LLM query-conditioned scoring and per-modality
 *                         top-k (Section 3.2, Eq. 5-6; Algorithm 1, inner loop)
 *   apack_compact_kv      gather of the kept rows of the K/V cache, hidden
 *                         states and position ids (Section 3.2, last
 *                         sentence; Algorithm 1, "slice their KV-cache entries")
 *   apack_compact_kv_inplace  the same slicing done in place, for callers
 *                         that cannot hold the cache twice
 *   apack_prefill_flops   analytic prefill FLOPs of a token-length schedule
 *                         (Appendix G)
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Tensor arguments are DEVICE pointers on the current HIP device.
 *   Descriptor arrays (apack_seq, apack_span, apack_av_seq, pointer tables)
 *   and the n_kept outputs are HOST pointers.
 * - `stream` is a hipStream_t handle (NULL = the null stream).  Every kernel
 *   and copy is enqueued on it; calls never synchronise the device.  Device
 *   outputs are valid once the stream has reached the point of the call;
 *   host outputs (n_kept, n_kept_visual) are valid when the call returns.
 * - The caller owns every buffer.  The library allocates no device memory:
 *   scratch space comes from the caller's `workspace` (size from the
 *   matching *_query call, 256-byte aligned).  The library keeps no pointer
 *   after a call returns.  Small host descriptors are copied to the device
 *   through library-owned pinned staging buffers.
 * - Errors: arguments are validated on the host before anything is enqueued.
 *   On error nothing is launched, outputs are untouched, the status is
 *   returned and apack_last_error() (thread-local) says why.  A failed HIP
 *   launch or copy returns APACK_E_HIP.
 * - Concurrent calls are safe when each uses its own workspace and outputs.
 * - bf16 tensors hold raw bfloat16 values (1 sign, 8 exponent, 7 mantissa
 *   bits); all inputs must be finite.
 */
#ifndef APACK_H
#define APACK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum apack_status {
  APACK_OK = 0,
  APACK_E_ARG = 1,        /* bad scalar argument or null pointer            */
  APACK_E_SHAPE = 2,      /* inconsistent sizes, spans or offsets           */
  APACK_E_DTYPE = 3,      /* unknown dtype or dtype/shape combination       */
  APACK_E_WORKSPACE = 4,  /* workspace missing, misaligned or too small     */
  APACK_E_ALIAS = 5,      /* an output overlaps an input                    */
  APACK_E_HIP = 6,        /* a HIP runtime call failed                      */
  APACK_E_UNSUPPORTED = 7 /* valid but outside what the library implements */
} apack_status;

/* The two bounding enumerators make every int32 value a valid apack_dtype,
 * so a wrong value passed by a caller is rejected (APACK_E_DTYPE) rather
 * than being undefined behaviour in the library. */
typedef enum apack_dtype {
  APACK_BF16 = 0,
  APACK_F32 = 1,
  APACK_DTYPE_MIN_ENUM_ = -0x7FFFFFFF - 1,
  APACK_DTYPE_MAX_ENUM_ = 0x7FFFFFFF
} apack_dtype;

typedef enum apack_modality {
  APACK_OTHER = 0,  /* text, system and any row not covered by a span */
  APACK_AUDIO = 1,
  APACK_VISUAL = 2
} apack_modality;

/* ------------------------------------------------------------------------ */
/* Helpers                                                                  */
/* ------------------------------------------------------------------------ */

const char* apack_version(void);
const char* apack_last_error(void);   /* message of this thread's last error */
const char* apack_status_string(apack_status s);

/* k = ceil(keep * n) for the decimal ratio `keep` means (Eq. 6's count
 * TopK_{ceil((1-P)|S|)}).  The product is formed in binary64 and a slack of
 * n * 2^-50 absorbs the binary representation error of a decimal ratio with
 * up to six fractional digits, so 0.55 * 100 gives 55 (a plain binary64
 * ceiling gives 56).  Exact for n < 2^29.  Returns -1 when keep is outside
 * [0, 1] or n < 0. */
int64_t apack_keep_count(double keep, int64_t n);

/* Pre-LLM visual budget (supplement, pre-LLM compression details): the joint
 * budget B = ceil(r_pre * (n_audio + n_visual)) keeps every audio token and
 * gives video the rest, B_v = clamp(B - n_audio, 0, n_visual).  Returns -1
 * on bad arguments. */
int64_t apack_visual_budget(double r_pre, int64_t n_audio, int64_t n_visual);

/* ------------------------------------------------------------------------ */
/* In-LLM query-conditioned prune (Section 3.2, Eq. 5 and Eq. 6)            */
/* ------------------------------------------------------------------------ */

/* A run of rows of one modality, relative to its sequence's first row. */
typedef struct apack_span {
  int64_t begin;
  int64_t len;
  int32_t modality;  /* APACK_AUDIO, APACK_VISUAL or APACK_OTHER */
  int32_t reserved;  /* must be 0 */
} apack_span;

/* apack_seq.flags: rank the audio and visual candidates together (Eq. 6 as
 * written) instead of per modality.  keep[0] / keep_basis[0] then apply to
 * the whole candidate set S, and keep[1] / keep_basis[1] must be 0. */
#define APACK_RANK_JOINT 1

/* One sequence of a (possibly ragged) packed batch at a prune layer. */
typedef struct apack_seq {
  int64_t tok_off;          /* first row of the sequence in the packed K     */
  int64_t n_tokens;         /* rows of the sequence (N)                      */
  const apack_span* spans;  /* HOST; ascending, disjoint, inside [0, N)      */
  int32_t n_spans;
  int32_t flags;            /* 0 (per-modality ranking) or APACK_RANK_JOINT  */
  int64_t q_off;            /* first query row of the sequence in packed Q   */
  int64_t q_len;            /* query rows (>= 1); 1 = the paper's last query */
  double keep[2];           /* keep ratio for [audio, visual], in [0, 1]     */
  int64_t keep_basis[2];    /* n in ceil(keep*n); 0 = current modality count */
} apack_seq;

/* Validates `seqs` for a prune step and reports the kept-row count of every
 * sequence (n_kept, HOST [n_seq], may be NULL) and the workspace size that
 * apack_prune_layer needs (workspace_bytes, may be NULL). */
apack_status apack_prune_layer_query(int32_t n_seq, const apack_seq* seqs,
                                     int32_t hq, int32_t hkv, int32_t d,
                                     int64_t* n_kept, size_t* workspace_bytes);

/* Scores the candidate rows S (audio and visual rows) of every sequence by
 * the attention mass of its query rows (Eq. 5), averaged over all hq heads
 * and q_len query rows, and selects per modality the ceil(keep*n) highest
 * (Eq. 6 applied within each modality), or the ceil(keep[0]*n) highest of S
 * with APACK_RANK_JOINT (Eq. 6 as written); ties go to the lower row.
 *
 *   q       [hq][q_rows][d] query projections of the query span (post-RoPE,
 *           as the decoder holds them); head h starts at q + h*q_head_stride
 *           elements, rows are contiguous d-element vectors.
 *   k       [hkv][k_rows][d] keys of the prune layer (post-RoPE); head g
 *           starts at k + g*k_head_stride elements.  Query head h reads key
 *           head h / (hq/hkv).  Logits are q.k / sqrt(d).
 *   scores  [k_rows] fp32 out: I_j for candidate rows of every sequence,
 *           0 for its other rows; rows outside every sequence are untouched.
 *   kept_rows  int32 out: for each sequence in order, the ascending packed
 *           rows (tok_off + local row) it keeps: every non-candidate row and
 *           the selected audio and visual rows.  kept_capacity >= sum n_kept.
 *   n_kept  HOST [n_seq] out (may be NULL).
 *
 * dtype: APACK_BF16 or APACK_F32 for both q and k; d must be 64 or 128.
 * Row counts: q_off+q_len <= q_rows, tok_off+n_tokens <= k_rows, head
 * strides >= rows*d; sequences may not overlap in k.
 */
apack_status apack_prune_layer(int32_t n_seq, const apack_seq* seqs, apack_dtype dtype,
                               int32_t hq, int32_t hkv, int32_t d,
                               const void* q, int64_t q_head_stride, int64_t q_rows,
                               const void* k, int64_t k_head_stride, int64_t k_rows,
                               float* scores, int32_t* kept_rows, int64_t kept_capacity,
                               int64_t* n_kept,
                               void* workspace, size_t workspace_bytes, void* stream);

/* Gathers rows: out[i] = in[src_rows[i]] for i < n_out, on raw bits, for
 *   - every K and V tensor of n_layers layers, each [hkv][rows][d] with head
 *     strides head_stride_in / head_stride_out (elements);
 *   - the hidden states [rows][hidden_dim] (hidden_in/hidden_out, nullable
 *     pair; hidden_dim 0 when absent);
 *   - the position ids [pos_rows][rows] int32 (nullable pair; row strides
 *     pos_stride_in / pos_stride_out elements; 3 rows for TMRoPE ids).
 * src_rows is a DEVICE int32 array of n_out indices into [0, n_in), usually
 * apack_prune_layer's kept_rows; an index outside [0, n_in) copies nothing
 * for that row.  k_in, v_in, k_out, v_out are HOST arrays of n_layers device
 * pointers (n_layers <= 64); v_in and v_out may both be NULL, and then only
 * the n_layers tensors of k_in move (any [hkv][rows][d] planes: a single
 * layer's K, or V tensors passed in the K slots).  Outputs may not overlap
 * inputs (APACK_E_ALIAS): compaction is out of place.
 */
apack_status apack_compact_kv(int64_t n_out, const int32_t* src_rows, int64_t n_in,
                              int32_t n_layers,
                              const void* const* k_in, const void* const* v_in,
                              void* const* k_out, void* const* v_out,
                              int32_t hkv, int32_t d, apack_dtype dtype,
                              int64_t head_stride_in, int64_t head_stride_out,
                              const void* hidden_in, void* hidden_out, int32_t hidden_dim,
                              const int32_t* pos_in, int32_t* pos_out, int32_t pos_rows,
                              int64_t pos_stride_in, int64_t pos_stride_out,
                              void* stream);

/* Workspace bytes apack_compact_kv_inplace needs for n_out kept rows
 * (0 for a negative n_out): 68 bytes per 128 kept rows and a few hundred more. */
size_t apack_compact_kv_inplace_workspace(int64_t n_out);

/* In-place form of apack_compact_kv (Section 3.2, last sentence; Algorithm 1,
 * "slice their KV-cache entries"): x[i] = x[src_rows[i]] for i < n_out in
 * every plane, on raw bits, without a second copy of the cache.
 *   - k[l] (and v[l]): [hkv][rows][d] tensors, head stride head_stride
 *     elements; k and v are HOST arrays of n_layers device pointers, v may
 *     be NULL (only the K planes move);
 *   - hidden: [rows][hidden_dim] (nullable; hidden_dim 0 when absent);
 *   - pos: [pos_rows][rows] int32 with row stride pos_stride (nullable;
 *     pos_rows <= 16).
 * src_rows is a DEVICE int32 array of n_out <= n_in indices that must be
 * strictly increasing and lie in [0, n_in), as apack_prune_layer's
 * kept_rows are; then rows [0, n_out) of every plane end up exactly as
 * apack_compact_kv would write them and rows [n_out, n_in) keep their old
 * contents.  For any other src_rows the call still ends and stays inside
 * the planes, but the contents of rows [0, n_out) are unspecified.
 * Planes may not overlap each other, src_rows or the workspace
 * (APACK_E_ALIAS).  The workspace (DEVICE, 256-byte aligned, size from
 * apack_compact_kv_inplace_workspace) holds per-call counters: calls that
 * share a workspace must not run concurrently.
 */
apack_status apack_compact_kv_inplace(int64_t n_out, const int32_t* src_rows, int64_t n_in,
                                      int32_t n_layers, void* const* k, void* const* v,
                                      int32_t hkv, int32_t d, apack_dtype dtype,
                                      int64_t head_stride,
                                      void* hidden, int32_t hidden_dim,
                                      int32_t* pos, int32_t pos_rows, int64_t pos_stride,
                                      void* workspace, size_t workspace_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * in-place compaction as apack_compact_kv_inplace, with the same arguments
 * and results, whose per-call counters live in a library-owned static device
 * array instead of a caller workspace.  The call allocates nothing, on the
 * device or the host.  Limit: n_out <= 2^20 kept rows (about 545 KiB of
 * scratch per GPU, held until the process ends); a larger n_out returns
 * APACK_E_UNSUPPORTED before anything is launched.  Every call on one GPU
 * shares that GPU's array, so calls on one GPU that overlap in time (on
 * different streams, or from different threads) race and must be ordered
 * by the caller.  The first call on a device looks up that device's copy of
 * the array; make it outside any graph capture.  A give-up of an ordering
 * wait (see apack_set_inplace_wait_limit) is not reported for this variant:
 * apack_compact_kv_inplace_status needs a caller workspace. */
apack_status apack_compact_kv_inplace_static(int64_t n_out, const int32_t* src_rows, int64_t n_in,
                                             int32_t n_layers, void* const* k, void* const* v,
                                             int32_t hkv, int32_t d, apack_dtype dtype,
                                             int64_t head_stride,
                                             void* hidden, int32_t hidden_dim,
                                             int32_t* pos, int32_t pos_rows, int64_t pos_stride,
                                             void* stream);

/* Reports whether the last apack_compact_kv_inplace call that moved rows
 * with this workspace gave up one of its waits.  The ordering waits are
 * bounded (see apack_set_inplace_wait_limit); a ticket whose wait gives up
 * stores nothing, so no row that another output row still has to read is
 * overwritten, but some of rows [0, n_out) keep their old contents and the
 * result is unusable.  Only a stalled GPU reaches the default limit.
 * Synchronises `stream`, then sets *gave_up (HOST) to 1 or 0. */
apack_status apack_compact_kv_inplace_status(const void* workspace, size_t workspace_bytes,
                                             int32_t* gave_up, void* stream);

/* Bound on one ordering wait of apack_compact_kv_inplace, in polls of a few
 * hundred nanoseconds each (default 2^22, a few seconds); returns the
 * previous bound.  Applies to calls made after it returns, process-wide.
 * A bound of 0 makes every wait that has earlier stripes to wait for give
 * up at once, so the give-up report can be exercised without a stall. */
uint32_t apack_set_inplace_wait_limit(uint32_t polls);

/* ------------------------------------------------------------------------ */
/* Prefill-FLOPs accounting (Appendix G)                                    */
/* ------------------------------------------------------------------------ */

/* Prefill cost of one decoder layer at sequence length n: 4 n d^2 for the
 * Q, K, V and O projections, 2 n^2 d for the attention and 2 n d m for the
 * feed-forward block, with d = d_model and m = d_ffn (Appendix G, per-layer
 * equation; Qwen2.5-Omni-7B: d 3584, m 18944, 28 layers; 3B: 2048, 11008,
 * 36).  Host only; -1 for a negative argument. */
double apack_layer_flops(int64_t n, int64_t d_model, int64_t d_ffn);

/* F_pre = sum over layers of apack_layer_flops(lengths[i]) and its ratio to
 * n_layers layers at the full length n0 (Appendix G, prefill and ratio
 * equations).  lengths is a HOST array of n_layers lengths entering each
 * layer; f_pre and ratio are HOST outputs (either may be NULL). */
apack_status apack_prefill_flops(int32_t n_layers, const int64_t* lengths, int64_t n0,
                                 int64_t d_model, int64_t d_ffn, double* f_pre, double* ratio);

/* The lengths entering each of n_layers layers (numbered from 0) when the
 * sequence starts at n_start and the prune at layer prune_layers[j] leaves
 * n_after[j] tokens: a prune scores with its layer's attention and takes
 * effect from the next layer (Algorithm 1, loop over layers from L_mid).
 * prune_layers (strictly increasing, in [0, n_layers)), n_after and lengths
 * are HOST arrays; n_after[j] is usually apack_prune_layer's n_kept. */
apack_status apack_schedule_lengths(int32_t n_layers, int64_t n_start, int32_t n_prunes,
                                    const int32_t* prune_layers, const int64_t* n_after,
                                    int64_t* lengths);

/* ------------------------------------------------------------------------ */
/* Pre-LLM local audio-visual dynamics scorer (Section 3.1)                 */
/* ------------------------------------------------------------------------ */

/* Hyper-parameters of the pre-LLM stage (Table S1). */
typedef struct apack_dyn_params {
  int32_t window;       /* w: frames per CKA window (3)                       */
  int32_t dafps_k;      /* neighbours in the DA-FPS density (5)               */
  double tau_gate;      /* CKA gate tau (0.78): fires when mean c_f < tau     */
  double beta;          /* fine-blend weight beta (0.90), Eq. 2               */
  double gamma;         /* visual-score weight gamma (0.9)                    */
  double tau_sim;       /* continuity threshold (0.97)                        */
  double sigma;         /* continuity smoothing width (1.0)                   */
  double lambda_seg;    /* peak/sustained balance lambda in Eq. 3 (0.5)       */
  double cover_thresh;  /* DA-FPS coverage cosine threshold (0.8)             */
  double dafps_power;   /* power on the DA-FPS density (0.5)                  */
  double r_pre;         /* pre-LLM joint retention R_pre (0.50)               */
  int32_t alignment;    /* frame alignment scorer, APACK_ALIGN_* (gated CKA)  */
} apack_dyn_params;

/* Frame alignment scorers (the supplement's comparison of alignment-scoring
 * rules and its window sweep); the rest of the scorer is unchanged.
 *   GATED_CKA    Eq. 1 over the window and the gate of Eq. 2 (the paper's).
 *   CKA          Eq. 1 alone: alpha_f = c_f for every clip, never gated.
 *   AV_COSINE    alpha_f = 1 - d_hat_f for every clip: each visual token's
 *                strongest cosine to any audio token of the clip, averaged
 *                over the frame and min-max normalised -- a token-wise match
 *                that ignores time (the "static" similarity).
 *   SPATIAL_CKA  the w = 1 variant: within frame f, linear CKA between the
 *                covariance of its visual tokens and that of the audio
 *                tokens of its adaptive-pool bin, each set centred by its
 *                own mean: c_f = ||A~ V~^T||^2 / (||A~ A~^T|| ||V~ V~^T||)
 *                (0 for a bin of one token); c_f then enters Eq. 2's gate.
 * frame_cka reports the c_f the mode uses (the window CKA for the first
 * three). */
#define APACK_ALIGN_GATED_CKA 0
#define APACK_ALIGN_CKA 1
#define APACK_ALIGN_AV_COSINE 2
#define APACK_ALIGN_SPATIAL_CKA 3

void apack_dyn_params_default(apack_dyn_params* p);

/* One clip of a packed batch. */
typedef struct apack_av_seq {
  int32_t n_frames;          /* F                                              */
  int32_t tokens_per_frame;  /* P (visual tokens of one frame, <= 256)         */
  int64_t n_audio;           /* N_A (>= 1)                                     */
  int64_t n_query;           /* query-span rows (>= 1)                         */
  int64_t vis_off;           /* first row of the clip in packed visual         */
  int64_t aud_off;           /* first row of the clip in packed audio          */
  int64_t qry_off;           /* first row of the clip in packed query          */
} apack_av_seq;

/* Validates and reports each clip's visual budget B_v (n_kept_visual, HOST
 * [n_seq], may be NULL) and the workspace size apack_score_dynamics needs. */
apack_status apack_score_dynamics_query(int32_t n_seq, const apack_av_seq* seqs, int32_t dim,
                                        const apack_dyn_params* p,
                                        int64_t* n_kept_visual, size_t* workspace_bytes);

/* Per clip: frame pooling and audio resampling (coarse pass), window CKA
 * c_f (Eq. 1), the gate and direct audio-visual distance (Eq. 2),
 * continuity segmentation, segment scores (Eq. 3), segment and frame
 * budgets (Eq. 4) and anchor DA-FPS / non-anchor dedup token selection.
 *
 *   visual [visual_rows][dim], audio [audio_rows][dim], query
 *   [query_rows][dim]: embeddings, row-major, dtype APACK_BF16 or APACK_F32.
 *   Frame arrays are [sum F], clip s starting at the sum of the previous
 *   clips' F: frame_cka c_f, frame_score s_f, frame_budget k_f and
 *   segment_id (0-based within the clip) -- each nullable.
 *   gate_fired [n_seq] (nullable).
 *   kept_visual int32 out: for each clip in order, the ascending packed
 *   visual rows (vis_off + f*P + p) it keeps; kept_capacity >= sum B_v.
 *   n_kept_visual HOST [n_seq] out (may be NULL).
 * dim must be a multiple of 8 and at most 16384.  Outputs may overlap neither
 * the inputs nor each other (APACK_E_ALIAS).
 */
apack_status apack_score_dynamics(int32_t n_seq, const apack_av_seq* seqs, apack_dtype dtype,
                                  int32_t dim,
                                  const void* visual, int64_t visual_rows,
                                  const void* audio, int64_t audio_rows,
                                  const void* query, int64_t query_rows,
                                  const apack_dyn_params* p,
                                  float* frame_cka, float* frame_score, int32_t* frame_budget,
                                  int32_t* segment_id, uint8_t* gate_fired,
                                  int32_t* kept_visual, int64_t kept_capacity,
                                  int64_t* n_kept_visual,
                                  void* workspace, size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* APACK_H */
