/*
 * libkvec — prefill-time KV-cache eviction with coverage (K-VEC) on MI355X.
 *
 * C ABI.  Plain pointers and sizes; device pointers are HIP device memory
 * (hipMalloc or a framework allocator), host pointers are ordinary memory.
 *
 * What the library computes (paper: "Coverage-Driven KV Cache Eviction for
 * Efficient and Improved Inference of LLM"):
 *
 *   kvec_score        the windowed eviction score P (Sec. 4.1, Eq. eviction),
 *                     the same score over the extended window O' (Sec. 4.1,
 *                     cross-head coverage) and the global importance I
 *                     (Sec. 4.2), for every KV head of one layer.
 *   kvec_select_cover the rest of Algorithm 1 on those scores: max-pooling,
 *                     head focus sigma, the delta lowest-sigma heads H_top
 *                     switched to the extended-window score, the preserve set
 *                     (top beta*B per head), the coverage bonus
 *                     P' = P + lambda * I * (1 - n_t/(l+1)), then the top-B
 *                     selection per head (Sec. 4.1) and the layer's entry in
 *                     the token-coverage bitmap that defines n_t (Sec. 4.2).
 *   kvec_compact      the cache store of the kept tokens (Sec. 4.1: the K/V of
 *                     the selected B tokens is stored for decoding).
 *   kvec_evict_layer  the three calls above for one layer.
 *   kvec_evict_model  the whole prefill eviction step for all layers.
 *   kvec_coverage     the coverage C = number of unique tokens kept across
 *                     heads and layers (Sec. 3.2).
 *   kvec_decode_attention
 *                     the consumer of the compacted cache: one decode token's
 *                     attention over the kept K/V (Sec. 4.1 keeps them for the
 *                     decoding phase).
 *   kvec_score_lse, kvec_evict_model_lse
 *                     the same scores and step when the caller already holds
 *                     the softmax normaliser of every window row: K-VEC runs
 *                     inside the prefill of each layer (Sec. 5.1), whose
 *                     attention computes that log-sum-exp for all query rows,
 *                     so the scores then need one pass over K instead of two.
 *
 * Conventions common to every call
 *   - Heads are KV heads.  Query head j belongs to KV head j / G with
 *     G = n_q_heads / n_kv_heads; A of a KV head is the mean of its G query
 *     heads' attention.  The observation window is the last O positions
 *     [T-O, T); it is always kept, and each head keeps B-O more tokens chosen
 *     from the candidates [0, T-O) ("Tc" below = T - O).
 *   - Element strides are in elements, not bytes; the head dimension d is
 *     contiguous.  Base pointers must be 16-byte aligned and every stride
 *     times the element size a multiple of 16 bytes (KVEC_ERR_INVALID).
 *   - Ownership: the caller owns every buffer.  The library never allocates
 *     device memory and keeps no state between calls; scratch memory is the
 *     caller's workspace `ws` of at least kvec_workspace_size() bytes.
 *   - All device work is enqueued on `stream` and is asynchronous; no call
 *     synchronises the host.  Calls on one workspace must be stream-ordered.
 *   - Errors: argument validation happens before any launch; on a validation
 *     error nothing is written.  A failed kernel launch returns
 *     KVEC_ERR_DEVICE (outputs are then undefined).
 *   - Ties: every ranking orders by (score descending, token index ascending);
 *     sigma ties order by lower head index.
 */
#ifndef KVEC_H
#define KVEC_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum kvec_status {
  KVEC_OK = 0,
  KVEC_ERR_INVALID = 1,      /* bad argument, shape, alignment or null pointer */
  KVEC_ERR_UNSUPPORTED = 2,  /* valid but not implemented (head count, head_dim, group size) */
  KVEC_ERR_WORKSPACE = 3,    /* workspace smaller than kvec_workspace_size() */
  KVEC_ERR_DEVICE = 4        /* a HIP launch or runtime call failed */
} kvec_status;

/* How H_top picks the heads that are rescored over O' (Sec. 4.1). */
typedef enum kvec_head_criterion {
  KVEC_HEADS_STD = 0,     /* the delta heads with the lowest std of pooled P (Sec. 4.1) */
  KVEC_HEADS_ENTROPY = 1  /* the delta heads with the highest entropy of pooled P taken as a
                             distribution over the candidates (the alternative criterion of
                             the head-selection ablation, Sec. 5.4) */
} kvec_head_criterion;

typedef enum kvec_dtype {
  KVEC_BF16 = 0,  /* Q, K, V and the compacted cache are bfloat16 */
  KVEC_F32 = 1    /* ... are IEEE float32 */
} kvec_dtype;

/* Shape and hyper-parameters of one eviction problem (Algorithm 1 inputs). */
typedef struct kvec_config {
  int32_t batch;          /* independent sequences, >= 1 */
  int32_t n_layers;       /* L, 1..255 (rows of the coverage bitmap; n_t is kept in 8 bits) */
  int32_t n_kv_heads;     /* H in {1, 2, 4, 8} */
  int32_t n_q_heads;      /* multiple of H; G = n_q_heads / H in 1..8 */
  int32_t head_dim;       /* d in {64, 128} */
  int32_t seq_len;        /* T, prefix length including the window, 1..262144 */
  int32_t window;         /* O, 1 <= O <= T */
  int32_t window_ext;     /* O' >= O (clamped to T); O' == O turns cross-head off */
  int32_t budget;         /* B per KV head including the window, B >= O */
  int32_t pool_kernel;    /* odd, 1..63: max-pool width along t (1 = none) */
  int32_t n_adjust_heads; /* delta, 0..H: heads switched to the O' score */
  float lambda;           /* >= 0: cross-layer bonus weight (0 = off) */
  float beta;             /* in [0, 1]: preserve K = min(floor(beta*B), B-O) per head */
  int32_t dtype;          /* kvec_dtype of Q, K, V and the compacted cache */
  int32_t head_criterion; /* kvec_head_criterion of H_top (KVEC_HEADS_STD is the paper's) */
} kvec_config;

/* Bytes of workspace the score/select/evict calls need for `cfg`.
 * Host-only; never touches the device. */
kvec_status kvec_workspace_size(const kvec_config* cfg, size_t* bytes);

/* Window scores of one layer (Sec. 4.1 Eq. eviction and its O' variant;
 * Sec. 4.2 global importance).
 *   q_win      device, [batch][n_q_heads][O'][d] rows at positions T-O'..T-1
 *              (post-RoPE), strides q_strides = {batch, head, row}.
 *   k          device, [batch][H][T][d], strides k_strides = {batch, head, t}.
 *   p_raw      device out, fp32 [batch][H][Tc]: P[h,t] = (1/O) sum over the
 *              last O window rows of A (causal softmax, scale 1/sqrt(d)).
 *   p_ext_raw  device out, fp32 [batch][H][Tc]: the same over all O' rows.
 *   imp        device out, fp32 [batch][Tc]: I[t] = (1/O) sum over the last
 *              O rows of the max over KV heads of A.
 * Scores are not pooled.  Tc = T - O must be >= 1. */
kvec_status kvec_score(const kvec_config* cfg,
                       const void* q_win, const int64_t q_strides[3],
                       const void* k, const int64_t k_strides[3],
                       float* p_raw, float* p_ext_raw, float* imp,
                       void* ws, size_t ws_bytes, hipStream_t stream);

/* Window scores of one layer, as kvec_score, from the caller's row
 * normalisers (the log-sum-exp the layer's prefill attention computed for
 * its query rows; Sec. 4.1 Eq. eviction divides by exactly this sum).
 *   lse          device, fp32 [batch][n_q_heads][O'] with strides
 *                lse_strides = {batch, head} in elements and rows contiguous;
 *                lse[b][j][r] = ln sum_{t <= T-O'+r} exp(q_{b,j,r} . k_{b,j/G,t}
 *                / sqrt(d)), natural log, over the same causal keys as the
 *                scores.  4-byte aligned (else KVEC_ERR_INVALID).
 *   other arguments, outputs and errors as kvec_score.  Only the accuracy of
 *   lse bounds the scores' accuracy: an error e in lse scales that row's
 *   probabilities by exp(-e). */
kvec_status kvec_score_lse(const kvec_config* cfg,
                           const void* q_win, const int64_t q_strides[3],
                           const float* lse, const int64_t lse_strides[2],
                           const void* k, const int64_t k_strides[3],
                           float* p_raw, float* p_ext_raw, float* imp,
                           void* ws, size_t ws_bytes, hipStream_t stream);

/* Selection of one layer from its scores (Algorithm 1, then top-B, Sec. 4.1-4.2).
 * H_top follows cfg->head_criterion; sigma and the entropy are float64 sums
 * over the pooled P of the candidates.
 *   layer       0-based index l; coverage uses n_t/(l+1).
 *   p_raw, p_ext_raw, imp  device fp32, as written by kvec_score.
 *   cover_bits  device uint64 [batch][n_layers][ceil(T/64)]: bit (l', t) set
 *               when layer l' kept token t in at least one head.  Rows
 *               l' < layer are read (n_t = number of those rows holding t);
 *               row `layer` is overwritten (cleared, then the kept tokens and
 *               the window set); rows > layer are not touched.  Layers are
 *               called in increasing order, so that rows 0..layer-1 hold this
 *               problem's earlier selections (layer 0 reads nothing).
 *   idx         device out, int32 [batch][H][B]: the B-O prefix picks in
 *               ascending order, then the window T-O..T-1.  If T <= B every
 *               token is kept: 0..T-1, remaining slots -1.
 *   htop_mask   device out, nullable, uint32 [batch]: bit h set when head h
 *               used the extended-window score (H_top). */
kvec_status kvec_select_cover(const kvec_config* cfg, int32_t layer,
                              const float* p_raw, const float* p_ext_raw, const float* imp,
                              uint64_t* cover_bits, int32_t* idx, uint32_t* htop_mask,
                              void* ws, size_t ws_bytes, hipStream_t stream);

/* Cache store (Sec. 4.1): k_out[b][h][i] = k[b][h][idx[b][h][i]] and the same
 * for v, byte-exact; rows with idx -1 are zero-filled.
 *   k, v         device, [batch][H][T][d] with strides {batch, head, t}.
 *   idx          device int32 [batch][H][B].
 *   k_out, v_out device out, contiguous [batch][H][B][d]. */
kvec_status kvec_compact(const kvec_config* cfg,
                         const void* k, const int64_t k_strides[3],
                         const void* v, const int64_t v_strides[3],
                         const int32_t* idx, void* k_out, void* v_out, hipStream_t stream);

/* One layer: kvec_score + kvec_select_cover + kvec_compact. */
kvec_status kvec_evict_layer(const kvec_config* cfg, int32_t layer,
                             const void* q_win, const int64_t q_strides[3],
                             const void* k, const int64_t k_strides[3],
                             const void* v, const int64_t v_strides[3],
                             uint64_t* cover_bits, int32_t* idx, void* k_out, void* v_out,
                             void* ws, size_t ws_bytes, hipStream_t stream);

/* The whole prefill eviction step: every layer, the selection in order 0..L-1.
 *   q_win, k, v  device, strides {layer, batch, head, row/t}.
 *   cover_bits   device uint64 [batch][L][ceil(T/64)]; every row is written.
 *   idx          device out int32 [L][batch][H][B].
 *   k_out, v_out device out, contiguous [L][batch][H][B][d].
 *   events       nullable; else kvec_profile_points(cfg) caller-created HIP
 *                events.  The step runs as a sequence of fused launches;
 *                events[i] is recorded on `stream` before launch i and the
 *                last event after the final launch (profiling only). */
kvec_status kvec_evict_model(const kvec_config* cfg,
                             const void* q_win, const int64_t q_strides[4],
                             const void* k, const int64_t k_strides[4],
                             const void* v, const int64_t v_strides[4],
                             uint64_t* cover_bits, int32_t* idx, void* k_out, void* v_out,
                             void* ws, size_t ws_bytes, hipStream_t stream,
                             hipEvent_t* events);

/* The whole step, as kvec_evict_model, also handing out every layer's window
 * scores as the pipeline computed them: P over the last O rows (Sec. 4.1,
 * Eq. eviction), P over the extended window O' of the H_top heads (Sec. 4.1)
 * and the global importance I (Sec. 4.2), all before pooling, and the H_top
 * set of each layer.
 *   p_raw_out   device out, fp32 [L][batch][H][T-O], contiguous.
 *   p_ext_out   device out, fp32 [L][batch][H][T-O], contiguous; only the rows
 *               of the heads in that layer's H_top are written (the pipeline
 *               scores the extended window for those heads only), the others
 *               are left as the caller set them.
 *   imp_out     device out, fp32 [L][batch][T-O], contiguous.
 *   htop_out    device out, uint32 [L][batch]: bit h set for h in H_top.
 * All four are required and 4-byte aligned (else KVEC_ERR_INVALID).  When
 * T <= B nothing is scored and they are left unchanged.  Other arguments,
 * outputs and errors as kvec_evict_model (no profiling events). */
kvec_status kvec_evict_model_scores(const kvec_config* cfg,
                                    const void* q_win, const int64_t q_strides[4],
                                    const void* k, const int64_t k_strides[4],
                                    const void* v, const int64_t v_strides[4],
                                    uint64_t* cover_bits, int32_t* idx, void* k_out, void* v_out,
                                    float* p_raw_out, float* p_ext_out, float* imp_out,
                                    uint32_t* htop_out, void* ws, size_t ws_bytes,
                                    hipStream_t stream);

/* Several independent whole steps in one call: the eviction of n_steps
 * prefills (Sec. 4.1-4.2 for each, exactly as kvec_evict_model computes it),
 * run as one layer pipeline over their n_steps x L layers in order, so the
 * closing launches of one step overlap the opening launches of the next
 * (n_steps x L + 11 fused launches instead of n_steps x (L + 11)).  For
 * throughput across back-to-back prefills; every step's outputs equal those
 * of a kvec_evict_model call on that step's inputs.
 *   n_steps      >= 1, n_steps x n_layers <= 2^20.
 *   q_win, k, v  device, as kvec_evict_model with one more leading stride:
 *                strides {step, layer, batch, head, row/t} in elements (a
 *                step stride of 0 evicts the same prefill n_steps times).
 *   cover_bits   device uint64 [n_steps][batch][L][ceil(T/64)].
 *   idx          device out int32 [n_steps][L][batch][H][B].
 *   k_out, v_out device out, contiguous [n_steps][L][batch][H][B][d].
 * Other arguments and errors as kvec_evict_model (no profiling events). */
kvec_status kvec_evict_model_steps(const kvec_config* cfg, int32_t n_steps,
                                   const void* q_win, const int64_t q_strides[5],
                                   const void* k, const int64_t k_strides[5],
                                   const void* v, const int64_t v_strides[5],
                                   uint64_t* cover_bits, int32_t* idx, void* k_out, void* v_out,
                                   void* ws, size_t ws_bytes, hipStream_t stream);

/* Several steps, as kvec_evict_model_steps, with every step's window-row
 * normalisers from the caller, as kvec_evict_model_lse (Sec. 5.1).
 *   lse          device, fp32 [n_steps][L][batch][n_q_heads][O'] with strides
 *                lse_strides = {step, layer, batch, head} in elements (any
 *                non-negative values, 0 included), rows contiguous.  Required
 *                even when T <= B (then unread).
 * Other arguments, outputs and errors as kvec_evict_model_steps. */
kvec_status kvec_evict_model_lse_steps(const kvec_config* cfg, int32_t n_steps,
                                       const void* q_win, const int64_t q_strides[5],
                                       const float* lse, const int64_t lse_strides[4],
                                       const void* k, const int64_t k_strides[5],
                                       const void* v, const int64_t v_strides[5],
                                       uint64_t* cover_bits, int32_t* idx, void* k_out,
                                       void* v_out, void* ws, size_t ws_bytes,
                                       hipStream_t stream);

/* Number of events kvec_evict_model records when given an event array
 * (n_layers + 12; 0 when T <= B), or -1 for an invalid configuration. */
int32_t kvec_profile_points(const kvec_config* cfg);

/* One layer, as kvec_evict_layer, with that layer's window-row normalisers
 * from the caller: the call a model makes inside the prefill of layer l, right
 * after its attention has produced them (Sec. 5.1).
 *   lse          device, fp32 [batch][n_q_heads][O'], strides {batch, head},
 *                rows contiguous (see kvec_score_lse).  Required even when
 *                T <= B (then unread). */
kvec_status kvec_evict_layer_lse(const kvec_config* cfg, int32_t layer,
                                 const void* q_win, const int64_t q_strides[3],
                                 const float* lse, const int64_t lse_strides[2],
                                 const void* k, const int64_t k_strides[3],
                                 const void* v, const int64_t v_strides[3],
                                 uint64_t* cover_bits, int32_t* idx, void* k_out, void* v_out,
                                 void* ws, size_t ws_bytes, hipStream_t stream);

/* The whole prefill eviction step, as kvec_evict_model, with the window rows'
 * normalisers from the caller (K-VEC applied inside each layer's prefill,
 * Sec. 5.1; see kvec_score_lse for their definition).
 *   lse          device, fp32 [L][batch][n_q_heads][O'] with strides
 *                lse_strides = {layer, batch, head} in elements, rows
 *                contiguous.  Required even when T <= B (then unread).
 *   events       nullable; else kvec_profile_points_lse(cfg) events.
 *   other arguments, outputs and errors as kvec_evict_model. */
kvec_status kvec_evict_model_lse(const kvec_config* cfg,
                                 const void* q_win, const int64_t q_strides[4],
                                 const float* lse, const int64_t lse_strides[3],
                                 const void* k, const int64_t k_strides[4],
                                 const void* v, const int64_t v_strides[4],
                                 uint64_t* cover_bits, int32_t* idx, void* k_out, void* v_out,
                                 void* ws, size_t ws_bytes, hipStream_t stream,
                                 hipEvent_t* events);

/* Number of events kvec_evict_model_lse records (n_layers + 8; 0 when
 * T <= B), or -1 for an invalid configuration. */
int32_t kvec_profile_points_lse(const kvec_config* cfg);

/* Coverage C (Sec. 3.2) per sequence over layers 0..upto_layer:
 * count_per_seq[b] = popcount of the OR of those layers' bitmaps.
 *   count_per_seq  device out, int64 [batch]. */
kvec_status kvec_coverage(const kvec_config* cfg, const uint64_t* cover_bits,
                          int32_t upto_layer, int64_t* count_per_seq, hipStream_t stream);

/* Workspace bytes of kvec_decode_attention for `cfg` and n_ctx cache rows
 * (host-only).  n_ctx in 1..2^20. */
kvec_status kvec_decode_workspace_size(const kvec_config* cfg, int32_t n_ctx, size_t* bytes);

/* Decode-step attention over the compacted cache (the kept K/V of Sec. 4.1
 * serve the decoding phase).  For every sequence b and query head j:
 *   out[b][j] = sum_i softmax_i(q_j . k_{h,i} / sqrt(d)) v_{h,i},  h = j / G,
 * over the cache rows i < n_ctx of KV head h, leaving out rows i < B whose
 * idx is negative (the padding kvec_compact writes when T <= B).
 *   q             device, cfg->dtype [batch][n_q_heads][d] (the new token's
 *                 post-RoPE queries), strides q_strides = {batch, head}.
 *   k_cache, v_cache  device, cfg->dtype [batch][H][n_ctx][d] with strides
 *                 cache_strides = {batch, head}, rows contiguous: the
 *                 compacted cache (rows 0..B-1 as kvec_compact writes them;
 *                 rows B.. may hold tokens appended after the prefill).
 *   n_ctx         rows per (sequence, head), 1..2^20 (>= B when idx is given).
 *   idx           nullable device int32 [batch][H][B] (kvec_compact's idx).
 *   out           device out, fp32 [batch][n_q_heads][d], contiguous; a
 *                 head with no unmasked row gets zeros.
 *   ws            device workspace of kvec_decode_workspace_size() bytes.
 * Errors as elsewhere (alignment 16 bytes for q and the caches, 4 for out). */
kvec_status kvec_decode_attention(const kvec_config* cfg,
                                  const void* q, const int64_t q_strides[2],
                                  const void* k_cache, const void* v_cache,
                                  const int64_t cache_strides[2], int32_t n_ctx,
                                  const int32_t* idx, float* out,
                                  void* ws, size_t ws_bytes, hipStream_t stream);

/* kvec_decode_attention for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same computation, with no workspace argument.  The
 * partial states live in a fixed device array of the library (4 MiB per
 * device, held until the process ends); the call allocates nothing.
 *   Arguments, outputs and errors as kvec_decode_attention, plus
 *   KVEC_ERR_WORKSPACE when the partial states would exceed 4 MiB, i.e. when
 *   kvec_decode_workspace_size(cfg, n_ctx) > 4 MiB (checked before any
 *   device call).  Every call on one device shares the array: calls that
 *   overlap on the same device (other streams, other host threads) race.
 *   The device is the current one; `stream` must belong to it. */
kvec_status kvec_decode_attention_noalloc(const kvec_config* cfg,
                                          const void* q, const int64_t q_strides[2],
                                          const void* k_cache, const void* v_cache,
                                          const int64_t cache_strides[2], int32_t n_ctx,
                                          const int32_t* idx, float* out, hipStream_t stream);

/* Static description of a status code. */
const char* kvec_status_string(kvec_status status);

#ifdef __cplusplus
}
#endif

#endif /* KVEC_H */
