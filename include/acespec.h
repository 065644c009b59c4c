/*
 * acespec.h -- C ABI of the MI355X (gfx950) tree-verification library.
 *
 * The library implements the cloud side of AceSpec's edge-cloud speculative decoding
 * (Section III-B, "Verify Loop"): one forward pass of a decoder-only target model over a
 * batch of drafted token trees, each node attending to its session's KV prefix and to its
 * own ancestors (Section III-C, tree attention mask), followed by the per-node reduction
 * of the target distribution to what the downlink carries (Algorithm 1, RECEIVE_WAIT
 * returns the rejection index and a sparse target distribution): the min(1, p/q)
 * acceptance test against the draft distribution, the residual max(0, p - q) resample,
 * a bonus sample, and a top-k sparse distribution; then the per-session path walk with
 * the sibling-hit rule of Algorithm 1 (the resampled token looked up among the drafted
 * alternatives).
 *
 * Conventions for every entry point:
 *  - All tensor pointers are DEVICE pointers, owned by the caller; the library never
 *    frees them.  Layouts are dense row-major with the shapes given in the comments.
 *  - Work is enqueued on `stream`; the call returns without synchronising and the
 *    outputs are valid once the stream has completed.
 *  - Argument and shape errors are reported synchronously, before anything is
 *    launched, by a negative return code; acespec_last_error() then holds a message.
 *  - Malformed per-session data found on the device sets status[b] for that session
 *    only; its other outputs are then unspecified but every access stays in bounds:
 *      ACESPEC_EBADTREE    a parent index that is not an earlier row, a token id outside
 *                          the vocabulary, a prefix length that does not fit the cache;
 *      ACESPEC_EBADDRAFT   a draft distribution the step reads holds a NaN, infinite or
 *                          negative entry (dense draft_q rows with children), or a scalar
 *                          q_hat outside [0, 1];
 *      ACESPEC_ENONFINITE  a target logit of the session is not finite: an activation
 *                          left the range of the 16-bit type it is handed on in (fp16
 *                          between the kernels of a bf16 model, max 65504), or the
 *                          weights, KV cache or hidden states hold NaN/inf.
 *    When several apply the first in this list that the step detects is reported
 *    (tree checks run before the forward pass; of the two data errors the
 *    non-finite logits win).
 *  - No C++ exception crosses this interface.
 *  - A context must not be used by two calls that overlap in time (its workspace is
 *    shared by all calls on it).
 */
#ifndef ACESPEC_H
#define ACESPEC_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  ACESPEC_OK = 0,
  ACESPEC_EINVAL = -1,        /* bad argument (null pointer, size out of range, ...)   */
  ACESPEC_EUNSUPPORTED = -2,  /* valid but not supported by these kernels            */
  ACESPEC_ENOMEM = -3,        /* workspace allocation failed in acespec_create        */
  ACESPEC_EHIP = -4,          /* a HIP runtime call failed                            */
  ACESPEC_EBADTREE = -5,      /* per-session status only: malformed tree or prefix    */
  ACESPEC_EBADDRAFT = -6,     /* per-session status only: NaN/inf/negative draft data  */
  ACESPEC_ENONFINITE = -7     /* per-session status only: non-finite target logits     */
} acespec_status;

typedef enum { ACESPEC_F32 = 0, ACESPEC_BF16 = 1 } acespec_dtype;

/* Decoder shape.  The paper names only the model families (Qwen, LLaMA; Section V-A);
 * the reading implemented is a Llama-style pre-norm decoder: RMSNorm with gains,
 * rotate-half RoPE (theta_i = rope_base^(-2i/head_dim)), grouped-query attention with
 * scale 1/sqrt(head_dim), SwiGLU MLP, no biases, untied LM head.
 * Supported: head_dim in {64, 128}; n_heads % n_kv_heads == 0;
 * d_model, n_heads*head_dim and d_ff multiples of 64; vocab a multiple of 4. */
typedef struct {
  int n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ff, vocab;
  float rope_base;   /* e.g. 10000 */
  float rms_eps;     /* e.g. 1e-5  */
  acespec_dtype dtype;  /* weights, activations between kernels and KV cache */
} acespec_model_desc;

/* Per-layer weights, all in the model dtype, row-major [out, in] (K contiguous). */
typedef struct {
  const void *attn_norm;   /* [d_model]                                              */
  const void *wqkv;        /* [(n_heads + 2 n_kv_heads) head_dim, d_model]: q, k, v rows */
  const void *wo;          /* [d_model, n_heads head_dim]                             */
  const void *mlp_norm;    /* [d_model]                                               */
  const void *w_gate_up;   /* [2 d_ff, d_model]: gate rows then up rows                */
  const void *w_down;      /* [d_model, d_ff]                                         */
} acespec_layer_weights;

/* Storage of the dense matrices of a bf16 model (wqkv, wo, w_gate_up, w_down, lm_head).
 * The embedding and the RMSNorm gains are always row-major in the model dtype. */
typedef enum {
  ACESPEC_LAYOUT_ROWS = 0,    /* bf16, row-major [out, in] as above                       */
  ACESPEC_LAYOUT_PACKED = 1   /* fp16 in the fragment order of acespec_pack_weight (same
                                 size); bf16 models only, vocab a multiple of 16           */
} acespec_layout;

typedef struct {
  const void *embed;                     /* [vocab, d_model]                           */
  const acespec_layer_weights *layers;   /* HOST array of n_layers entries              */
  const void *final_norm;                /* [d_model]                                  */
  const void *lm_head;                   /* [vocab, d_model]                           */
  acespec_layout layout;                 /* of the dense matrices; 0 = row-major        */
} acespec_weights;

/* KV cache, in the model dtype.  Keys: k [n_layers][B][n_kv_heads][capacity][head_dim],
 * stored after RoPE.  Values are head-dim-major: v [n_layers][B][n_kv_heads][head_dim]
 * [capacity] (slot s of a head is column s), so that the attention's contraction over
 * slots reads contiguous memory.  Slots [0, prefix_len[b]) hold session b's verified
 * context and are only read.  The verify call writes the tree's keys and values into
 * slots prefix_len[b] + r for tree rows r = 0..N (nothing is committed: calling again
 * with the same inputs gives the same result). */
typedef struct {
  void *k, *v;
  int capacity;                 /* slots per (layer, session, kv head); multiple of 64 */
  const int32_t *prefix_len;    /* [B] DEVICE; needs prefix_len[b] + N + 1 <= capacity */
} acespec_kv_cache;

/* Target sampling parameters (Section III-B: nucleus sampling on the target side). */
typedef struct {
  float temperature;   /* > 0: logits are divided by it                               */
  float top_p;         /* (0, 1]: smallest most-probable set reaching this mass        */
  int top_k;           /* 1..256 and <= vocab: size of the sparse downlink payload     */
} acespec_params;

/* Caller-allocated device outputs.  Row counts: B*(N+1) rows for verify_tree (row 0 of
 * each session is the root), R rows for verify_tail. */
typedef struct {
  uint8_t *accept;          /* [rows] 1 if the row's token is accepted by its parent's
                               distribution (root rows: 1)                             */
  int32_t *acc_prefix_len;  /* [rows] leading accepted nodes on the root-to-row path  */
  int32_t *resample_token;  /* [rows] residual inverse-CDF sample (root rows: -1)     */
  int32_t *bonus_token;     /* [rows] sample from the row's own target distribution   */
  int32_t *topk_ids;        /* [rows, top_k] most probable first                      */
  float   *topk_probs;      /* [rows, top_k] renormalised over the k ids (0 outside
                               the top-p nucleus)                                     */
  int32_t *path;            /* [B, N+1] kept drafted rows root-first, -1 padded       */
  int32_t *path_len;        /* [B] drafted tokens kept                                */
  int32_t *next_token;      /* [B] token emitted after the kept path                  */
  uint8_t *sibling_hit;     /* [B] 1 if the walk continued through a drafted sibling */
  int32_t *status;          /* [B] ACESPEC_OK, or EBADTREE / EBADDRAFT / ENONFINITE   */
  float   *logits_out;      /* optional [rows, vocab] fp32 logits; NULL = not kept    */
} acespec_outputs;

typedef struct acespec_ctx acespec_ctx;

/* Creates a context on the current HIP device and allocates its workspace for up to
 * max_batch sessions of up to max_nodes drafted nodes (max_nodes <= 64), i.e.
 * max_batch*(max_nodes+1) rows.  The same bound limits verify_tail's row count.
 * Returns ACESPEC_OK and *out, or an error (ENOMEM if the workspace does not fit). */
int acespec_create(const acespec_model_desc *desc, int max_batch, int max_nodes,
                   acespec_ctx **out);

/* Frees the workspace (synchronises the device first).  NULL is accepted. */
void acespec_destroy(acespec_ctx *ctx);

/* One verify step over B drafted trees of N drafted nodes each.
 *  tree_tokens [B, N+1] int32: row 0 is the root (the last committed token, not yet in
 *                the cache), rows 1..N the drafted tokens.
 *  parent_idx  [B, N+1] int32: parent_idx[b,0] = -1 and 0 <= parent_idx[b,r] < r.
 *                The lowest-index child of a row is its main-chain child.
 *  draft_q     [B, N+1, vocab] fp32: row r holds the draft distribution that proposed
 *                r's children; only rows with children are read.
 *  uniforms    [B, N+1, 3] fp32 in (0, 1): per row (accept, residual, bonus).
 * Writes every field of *outs (logits_out only if non-NULL). */
int acespec_verify_tree(acespec_ctx *ctx, const acespec_weights *weights,
                        const acespec_kv_cache *kv, const int32_t *tree_tokens,
                        const int32_t *parent_idx, const float *draft_q,
                        const float *uniforms, int B, int N, const acespec_params *params,
                        const acespec_outputs *outs, hipStream_t stream);

/* The same step for the paper's own uplink (Section III-B, Algorithm 1: the edge sends
 * the drafted tokens and a compressed draft distribution; the cloud does no resampling of
 * its own and returns the rejection index with a sparse target distribution):
 *  q_hat [B, N+1] fp32: q_hat[b, r] = the draft probability of row r's own token under
 *                its parent's draft distribution (row 0 unused) -- one float per node
 *                instead of a vocabulary-sized row.
 * Per row: accept (u[.., 0] * q_hat < p), acc_prefix_len, topk_ids / topk_probs as in
 * acespec_verify_tree; resample_token = bonus_token = -1 (no cloud-side sampling).
 * Per session: path / path_len along accepted main children (no sibling hits: they need
 * the resample token), next_token = -1, sibling_hit = 0.  The edge resamples from the
 * top-k payload of row path_len (acc. position) against its own draft distribution;
 * that is exact only where the payload covers the target's nucleus. */
int acespec_verify_tree_scalar_q(acespec_ctx *ctx, const acespec_weights *weights,
                                 const acespec_kv_cache *kv, const int32_t *tree_tokens,
                                 const int32_t *parent_idx, const float *q_hat,
                                 const float *uniforms, int B, int N,
                                 const acespec_params *params, const acespec_outputs *outs,
                                 hipStream_t stream);

/* LM head and verification only, over R given hidden states (the last stage of
 * verify_tree on its own).  Each row r is the parent of one drafted token
 * draft_tokens[r]; rows form chains of chain_len consecutive rows (R % chain_len == 0).
 *  lm_head [vocab, d_model] in the layout lm_head_layout (ACESPEC_LAYOUT_PACKED: as
 *          written by acespec_pack_weight, for bf16 models with vocab a multiple of 16;
 *          another value: ACESPEC_EINVAL, a packed head otherwise ACESPEC_EUNSUPPORTED),
 *  final_norm [d_model] or NULL (no normalisation),
 *  hidden [R, d_model] in the model dtype, draft_q [R, vocab], uniforms [R, 3].
 * Per row: accept, resample_token, bonus_token, topk_*, acc_prefix_len (leading accepts
 * within its chain, counting the row).  Per chain c: path_len[c] = leading accepts,
 * path[c, 0..chain_len) = kept row indices within the chain (-1 padded),
 * next_token[c] = resample at the first rejected row, or -1 when the whole chain is
 * accepted (the bonus then needs the row after the chain); sibling_hit[c] = 0;
 * status[c] = OK, EBADTREE (a draft token outside the vocabulary), or EBADDRAFT /
 * ENONFINITE for a row of the chain (without final_norm, hidden values beyond the fp16
 * range of a bf16 model overflow and give ENONFINITE).  path is [R/chain_len, chain_len]. */
int acespec_verify_tail(acespec_ctx *ctx, const void *lm_head, acespec_layout lm_head_layout,
                        const void *final_norm, const void *hidden, const int32_t *draft_tokens,
                        const float *draft_q, const float *uniforms, int R, int chain_len,
                        const acespec_params *params, const acespec_outputs *outs,
                        hipStream_t stream);

/* acespec_verify_tail without a context, for callers that cannot allocate device memory
 * at all (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same kernels and results as acespec_verify_tail, the intermediate data
 * in a fixed device array of the library (48 MiB per device, held from the first call on
 * that device until the process ends).  Nothing is allocated, by this call or at set-up.
 *  desc: the model (only dtype, d_model, vocab and rms_eps are read).
 *  outs->logits_out is REQUIRED: the fp32 logits [R, vocab] are written there.
 * R is limited by the array: R * (4 + 4 ceil(vocab / 128) + d_model * 2) bytes (d_model * 4
 * for an fp32 model with a final norm; no d_model term for an fp32 model without one) must
 * fit in 48 MiB, else ACESPEC_EINVAL before anything is launched (e.g. R <= 4096 at
 * d_model 4096, vocab 128256).  The LM head is never sliced along K here.
 * All calls on one device share the array: two calls that overlap in time on the same
 * device race (serialise them, e.g. on one stream).  Every byte a call reads from the
 * array it has written first, so no clearing is needed between calls. */
int acespec_verify_tail_noalloc(const acespec_model_desc *desc, const void *lm_head,
                                acespec_layout lm_head_layout, const void *final_norm,
                                const void *hidden,
                                const int32_t *draft_tokens, const float *draft_q,
                                const float *uniforms, int R, int chain_len,
                                const acespec_params *params, const acespec_outputs *outs,
                                hipStream_t stream);

/* Commits the accepted path of every session into its KV cache (Algorithm 1, the
 * cloud's COMPACT_KV after RECEIVE_WAIT: only the state of the kept prefix survives a
 * verify round).  Inputs are a verify_tree call's outputs over the same cache:
 *  path [B, N+1], path_len [B]: the kept drafted rows root-first (outs->path, path_len);
 *  status [B] or NULL: sessions whose status is not ACESPEC_OK are not committed.
 * For every layer and kv head, the keys and values of row 0 (the root) and of the kept
 * rows path[b, 0 .. path_len[b]) move from slots prefix_len[b] + row to the contiguous
 * slots prefix_len[b] + 0 .. prefix_len[b] + path_len[b] -- the slots a causal decode of
 * the accepted tokens fills, since a kept node at depth i sits at RoPE position
 * prefix_len[b] + i.  Slots below prefix_len[b] are not touched; the tree slots past the
 * new end keep stale entries.
 *  new_prefix_len [B] DEVICE output: prefix_len[b] + 1 + path_len[b], or -1 for a session
 *  that was not committed (bad status, prefix_len + N + 1 > capacity, path_len outside
 *  [0, N] or a kept row outside [1, N]); nothing of such a session is moved.  It must not
 *  overlap kv->prefix_len (every workgroup of a session reads prefix_len[b] while one of
 *  them writes new_prefix_len[b]): an overlapping pair returns ACESPEC_EINVAL before
 *  anything is launched.  Copy new_prefix_len into prefix_len after the call instead.
 * The next round's root is the verify step's next_token (not yet in the cache). */
int acespec_commit_kv(acespec_ctx *ctx, const acespec_kv_cache *kv, const int32_t *path,
                      const int32_t *path_len, const int32_t *status, int B, int N,
                      int32_t *new_prefix_len, hipStream_t stream);

/* Re-lays one row-major bf16 weight matrix [rows, cols] (rows % 16 == 0, cols % 32 == 0)
 * out into the packed layout (ACESPEC_LAYOUT_PACKED): for every 16-row block and 32-column
 * step, the 1 KB operand of one 16x16x32 matrix-core instruction, contiguous, its values
 * widened to fp16.  The packed matrix holds the operands the verify pass multiplies by
 * anyway (the row-major path widens each bf16 weight to fp16 the same way before its
 * products, so the two layouts differ at most in how a product's k-slices are summed in
 * fp32); packed, each wave of the GEMMs loads its weight operands straight into
 * registers, and only the activations pass through LDS.  Weights
 * beyond the fp16 range (|w| > 65504) become +-inf, as they do on the row-major path.
 * Not part of the verify step: a caller packs its weights once (e.g. at load time).
 *  src [rows, cols] bf16, dst rows*cols*2 bytes; both DEVICE, caller-owned, no overlap.
 * Enqueued on stream; ACESPEC_EINVAL for a NULL pointer or a shape outside the above. */
int acespec_pack_weight(const void *src, void *dst, int rows, int cols, hipStream_t stream);

/* Value-cache layout conversion, for callers that keep values slot-major like the keys
 * (v[planes][capacity][head_dim], slot s of a head is row s): the verify step reads the
 * head-dim-major layout of acespec_kv_cache (v[planes][head_dim][capacity]), in which the
 * attention's sum over slots (Section III-C) streams contiguous memory.  Not part of the
 * verify step: a caller converts a session's prefix once when it loads it, and converts
 * back when it needs slot-major values again.
 *  planes     = n_layers * B * n_kv_heads (the leading dimensions, same order in both),
 *  capacity   slots per plane, a positive multiple of 64 (as in acespec_kv_cache),
 *  head_dim   >= 1,  dtype: ACESPEC_BF16 or ACESPEC_F32 (element size 2 or 4 bytes),
 *  direction  ACESPEC_V_TO_HEAD_DIM_MAJOR (src slot-major) or ACESPEC_V_TO_SLOT_MAJOR
 *             (src head-dim-major, the inverse),
 *  src, dst   DEVICE, caller-owned, planes*capacity*head_dim elements each, no overlap.
 * Values are copied bit for bit.  Enqueued on stream; ACESPEC_EINVAL (nothing launched)
 * for a NULL pointer, overlap, an unknown dtype or direction, a size outside the above,
 * or more than 2^31 - 1 tiles of 32 x 32 (convert in parts). */
typedef enum { ACESPEC_V_TO_HEAD_DIM_MAJOR = 0, ACESPEC_V_TO_SLOT_MAJOR = 1 } acespec_v_direction;
int acespec_convert_v_cache(const void *src, void *dst, int planes, int capacity, int head_dim,
                            acespec_dtype dtype, acespec_v_direction direction,
                            hipStream_t stream);

/* Message for the last non-OK return on this thread ("" if none). */
const char *acespec_last_error(void);

/* Per-kernel timing with HIP events recorded on the launch stream around every
 * kernel.  enable != 0 turns it on for subsequent calls.  acespec_timing_read waits
 * for the recorded events, returns per-kernel-kind totals accumulated since the last
 * read (names[i], total_ms[i], launches[i] for i < returned count, at most max
 * entries) and clears them.  names point to static strings. */
int acespec_timing_enable(acespec_ctx *ctx, int enable);
int acespec_timing_read(acespec_ctx *ctx, const char **names, double *total_ms,
                        int *launches, int max);
/* Restricts the timing events to the kernels of one kind (a name acespec_timing_read
 * reports, e.g. "gemm_gate_up"); NULL restores every kind.  Each timed launch adds two
 * event records to the stream, so timing one kind keeps the cost to the measured step
 * small.  Unknown names return ACESPEC_EINVAL and leave the selection unchanged. */
int acespec_timing_only(acespec_ctx *ctx, const char *kind);

#ifdef __cplusplus
}
#endif
#endif /* ACESPEC_H */
