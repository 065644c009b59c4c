// Host side of the verify library: context and workspace, argument validation, the
// launch sequence of one verify step, per-kernel event timing and error reporting.
//
// One verify step (Section III-B: the cloud runs one forward pass over the received
// tokens, then checks them): tree prep -> embedding -> for each layer {RMSNorm, QKV
// GEMM, RoPE + tree K/V write, tree attention, O GEMM + residual, RMSNorm, gate/up GEMM
// + SwiGLU, down GEMM + residual} -> final RMSNorm -> LM head GEMM (fp32 logits) ->
// fused vocabulary verify -> path walk.  Everything is enqueued on the caller's stream
// without synchronisation and without allocation.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "common.h"

using namespace acespec;

namespace {

thread_local std::string g_err;

int fail(int code, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

enum Kind {
  K_TREE, K_EMBED, K_RMSNORM, K_GEMM_QKV, K_ROPE, K_ATTN, K_GEMM_O, K_GEMM_GATE_UP,
  K_GEMM_DOWN, K_GEMM_LM, K_VOCAB, K_WALK, K_COMMIT, K_COUNT
};
const char *kKindNames[K_COUNT] = {"tree_prep",    "embed",       "rmsnorm",
                                   "gemm_qkv",     "rope_table",  "tree_attention",
                                   "gemm_o",       "gemm_gate_up", "gemm_down",
                                   "gemm_lm_head", "vocab_verify", "path_walk",
                                   "commit_kv"};

size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }

constexpr int kCandCap = 4096;  // threshold-bin candidates kept per row (16 KB)

}  // namespace

struct acespec_ctx {
  acespec_model_desc d;
  int max_batch = 0, max_nodes = 0, max_rows = 0;
  size_t esz = 0;  // bytes per model-dtype element
  void *ws = nullptr;
  float *x = nullptr, *logits = nullptr, *part_o = nullptr, *part_ml = nullptr;
  void *a = nullptr, *attn = nullptr, *q = nullptr, *h = nullptr;  // activation type
  float *qkv = nullptr;                                              // fp32 projection
  long long part_cap = 0;
  float *gpart = nullptr;     // split-K partials of the GEMMs
  long long gpart_cap = 0;
  int cus = 256;
  double *inv_freq = nullptr;
  float2 *rot = nullptr;      // RoPE (cos, sin) per tree row and frequency, per step
  float *tile_max = nullptr;  // LM-head row maxima per column tile
  uint32_t *cand = nullptr;   // vocabulary kernel: threshold-bin candidates per row
  int32_t *rowflag = nullptr; // vocabulary kernel: per-row data-error code (0 = none)
  TreeMeta meta{};
  // timing
  bool timing = false;
  uint32_t timing_mask = ~0u;  // kinds timed while timing is on
  struct Rec { int kind; hipEvent_t e0, e1; };
  std::vector<hipEvent_t> free_events;
  std::vector<Rec> pending;
  double tot_ms[K_COUNT] = {};
  int launches[K_COUNT] = {};
};

namespace {

hipEvent_t get_event(acespec_ctx *c) {
  if (!c->free_events.empty()) {
    hipEvent_t e = c->free_events.back();
    c->free_events.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Runs one launch, bracketed by timing events when enabled.
template <typename F>
int run(acespec_ctx *c, int kind, hipStream_t s, F &&launch) {
  hipEvent_t e0 = nullptr, e1 = nullptr;
  const bool timed = c && c->timing && ((c->timing_mask >> kind) & 1u);
  if (timed) {
    e0 = get_event(c);
    e1 = get_event(c);
    if (!e0 || !e1) return fail(ACESPEC_EHIP, "hipEventCreate failed");
    if (hipEventRecord(e0, s) != hipSuccess) return fail(ACESPEC_EHIP, "hipEventRecord failed");
  }
  hipError_t err = launch();
  if (err != hipSuccess)
    return fail(ACESPEC_EHIP, "%s launch failed: %s", kKindNames[kind], hipGetErrorString(err));
  if (timed) {
    if (hipEventRecord(e1, s) != hipSuccess) return fail(ACESPEC_EHIP, "hipEventRecord failed");
    c->pending.push_back({kind, e0, e1});
  }
  return ACESPEC_OK;
}

#define RUN(kind, expr)                                              \
  do {                                                               \
    int rc_ = run(ctx, kind, stream, [&]() -> hipError_t { return expr; }); \
    if (rc_ != ACESPEC_OK) return rc_;                               \
  } while (0)

// The storage of the dense matrices (acespec_layout): packed needs a bf16 model and a
// vocabulary that is a multiple of 16.
int check_layout(int layout, const acespec_model_desc &d) {
  if (layout != ACESPEC_LAYOUT_ROWS && layout != ACESPEC_LAYOUT_PACKED)
    return fail(ACESPEC_EINVAL, "unknown weight layout %d", layout);
  if (layout == ACESPEC_LAYOUT_PACKED && (d.dtype != ACESPEC_BF16 || d.vocab % 16 != 0))
    return fail(ACESPEC_EUNSUPPORTED,
                "packed weights need a bf16 model with a vocabulary that is a multiple of 16");
  return ACESPEC_OK;
}

int check_params(const acespec_params *p, int V) {
  if (!p) return fail(ACESPEC_EINVAL, "params is NULL");
  if (!(p->temperature > 0.f) || !std::isfinite(p->temperature))
    return fail(ACESPEC_EINVAL, "temperature must be finite and > 0 (got %g)", p->temperature);
  if (!(p->top_p > 0.f && p->top_p <= 1.f))
    return fail(ACESPEC_EINVAL, "top_p must be in (0, 1] (got %g)", p->top_p);
  if (p->top_k < 1 || p->top_k > 256 || p->top_k > V)
    return fail(ACESPEC_EINVAL, "top_k must be in [1, min(256, vocab)] (got %d)", p->top_k);
  return ACESPEC_OK;
}

// log2(e) / T in double, handed to the vocabulary kernel as a float pair.
void set_temperature(VocabArgs &va, float T) {
  const double c = 1.4426950408889634074 / (double)T;
  va.c_hi = (float)c;
  va.c_lo = (float)(c - (double)va.c_hi);
}

int check_outputs(const acespec_outputs *o) {
  if (!o) return fail(ACESPEC_EINVAL, "outputs is NULL");
  if (!o->accept || !o->acc_prefix_len || !o->resample_token || !o->bonus_token ||
      !o->topk_ids || !o->topk_probs || !o->path || !o->path_len || !o->next_token ||
      !o->sibling_hit || !o->status)
    return fail(ACESPEC_EINVAL, "an output pointer is NULL (only logits_out may be)");
  return ACESPEC_OK;
}

template <typename T>
int verify_tree_impl(acespec_ctx *ctx, const acespec_weights *w, const acespec_kv_cache *kv,
                     const int32_t *tokens, const int32_t *parents, const float *draft_q,
                     const float *q_scalar, const float *uniforms, int B, int N,
                     const acespec_params *p, const acespec_outputs *o, hipStream_t stream) {
  typedef typename ActOf<T>::type A;
  const acespec_model_desc &d = ctx->d;
  const int n1 = N + 1, R = B * n1;
  const int L = d.n_layers, D = d.d_model, H = d.n_heads, Hkv = d.n_kv_heads, hd = d.head_dim;
  const int F = d.d_ff, V = d.vocab, QKVN = (H + 2 * Hkv) * hd;
  const int cap = kv->capacity;
  A *x_a = (A *)ctx->a, *x_attn = (A *)ctx->attn, *x_q = (A *)ctx->q, *x_h = (A *)ctx->h;
  const GemmAux aux{ctx->gpart, ctx->gpart_cap, ctx->cus,
                   w->layout == ACESPEC_LAYOUT_PACKED ? 1 : 0};
  float *logits = o->logits_out ? o->logits_out : ctx->logits;
  const TreeMeta &meta = ctx->meta;

  RUN(K_TREE, launch_tree_prep(tokens, parents, kv->prefix_len, B, n1, V, cap, meta, o->status,
                               stream));
  RUN(K_EMBED, launch_embed<T>((const T *)w->embed, meta.tok, ctx->x, R, D, stream));
  if (L > 0) RUN(K_ROPE, launch_rope_table(meta.pos, ctx->inv_freq, ctx->rot, R, hd / 2, stream));
  const size_t layer_stride = (size_t)B * Hkv * cap * hd;
  // The residual projections (O, down) also apply the RMSNorm that opens the next block
  // (the MLP's, the next layer's attention norm, the final norm).
  RUN(K_RMSNORM, (launch_rmsnorm<T, float>(
                     ctx->x, (const T *)(L > 0 ? w->layers[0].attn_norm : w->final_norm), x_a,
                     R, D, d.rms_eps, stream)));
  for (int l = 0; l < L; ++l) {
    const acespec_layer_weights &lw = w->layers[l];
    T *ck = (T *)kv->k + l * layer_stride;
    T *cv = (T *)kv->v + l * layer_stride;
    const RopeOut<T> ro{x_q, ck, cv, ctx->rot, meta.sess_S, n1, H, Hkv, hd, cap};
    RUN(K_GEMM_QKV, (launch_qkv_rope<T, A>(x_a, (const T *)lw.wqkv, R, QKVN, D, ctx->qkv, ro,
                                           meta, B, aux, stream)));
    int nsplit = 1;
    RUN(K_ATTN, launch_attention<T>(x_q, ck, cv, meta, x_attn, ctx->part_o, ctx->part_ml,
                                    ctx->part_cap, B, n1, H, Hkv, hd, cap, ctx->cus, stream,
                                    &nsplit));
    RUN(K_GEMM_O, (launch_gemm_resid_norm<T, A>(x_attn, (const T *)lw.wo, R, D, H * hd, ctx->x,
                                                (const T *)lw.mlp_norm, x_a, d.rms_eps, aux,
                                                stream)));
    RUN(K_GEMM_GATE_UP, (launch_gemm<T, A>(EPI_SWIGLU, x_a, (const T *)lw.w_gate_up, R, F, D,
                                           x_h, nullptr, aux, stream)));
    const T *next_norm = (const T *)(l + 1 < L ? w->layers[l + 1].attn_norm : w->final_norm);
    RUN(K_GEMM_DOWN, (launch_gemm_resid_norm<T, A>(x_h, (const T *)lw.w_down, R, D, F, ctx->x,
                                                   next_norm, x_a, d.rms_eps, aux, stream)));
  }
  int ntile = 0;
  RUN(K_GEMM_LM, (launch_lm_head<T, A>(x_a, (const T *)w->lm_head, R, V, D, logits,
                                       ctx->tile_max, &ntile, aux, stream)));
  VocabArgs va{};
  va.logits = logits;
  va.q = draft_q;
  va.q_scalar = q_scalar;
  va.tile_max = ntile ? ctx->tile_max : nullptr;
  va.ntile = ntile;
  va.cand = ctx->cand;
  va.cand_cap = kCandCap;
  va.rowflag = ctx->rowflag;
  va.u = uniforms;
  va.tok = meta.tok;
  va.par = meta.par;
  va.n1 = n1;
  va.tail = 0;
  va.rows = R;
  va.V = V;
  va.k = p->top_k;
  set_temperature(va, p->temperature);
  va.top_p = p->top_p;
  va.accept = o->accept;
  va.resample = o->resample_token;
  va.bonus = o->bonus_token;
  va.topk_ids = o->topk_ids;
  va.topk_probs = o->topk_probs;
  RUN(K_VOCAB, launch_vocab(va, stream));
  RUN(K_WALK, launch_walk(meta.tok, meta.par, meta.depth, o->accept, o->resample_token,
                          o->bonus_token, ctx->rowflag, B, n1, o->acc_prefix_len, o->path,
                          o->path_len, o->next_token, o->sibling_hit, o->status, stream));
  return ACESPEC_OK;
}

// Where one LM-head + verify call keeps its intermediate data.
struct TailWorkspace {
  float *logits;      // [R, V] when the caller keeps no logits_out
  float *tile_max;    // [R, ceil(V / 128)]
  uint32_t *cand;     // [R, cand_cap] or NULL (the vocabulary kernel re-reads the row)
  int cand_cap;
  int32_t *rowflag;   // [R]
  void *a;            // [R, d_model] activation type: normalised / widened hidden states
  GemmAux aux;        // split-K partials (part_cap 0: the LM head is never split)
};

// ctx only times the launches (NULL: no timing).
template <typename T>
int verify_tail_run(acespec_ctx *ctx, const acespec_model_desc &d, const TailWorkspace &ws,
                    const void *lm_head, const void *final_norm, const void *hidden,
                    const int32_t *draft, const float *draft_q, const float *uniforms, int R,
                    int chain_len, const acespec_params *p, const acespec_outputs *o,
                    hipStream_t stream) {
  typedef typename ActOf<T>::type A;
  const int D = d.d_model, V = d.vocab;
  float *logits = o->logits_out ? o->logits_out : ws.logits;
  const A *h_in = (const A *)hidden;
  if (final_norm) {
    RUN(K_RMSNORM, (launch_rmsnorm<T, T>((const T *)hidden, (const T *)final_norm, (A *)ws.a,
                                         R, D, d.rms_eps, stream)));
    h_in = (const A *)ws.a;
  } else if (sizeof(T) == 2) {  // bf16 hidden states: widen to fp16 for the f16 MFMA path
    RUN(K_RMSNORM, launch_cast_bf16_f16((const bf16 *)hidden, (f16 *)ws.a, (size_t)R * D,
                                        stream));
    h_in = (const A *)ws.a;
  }
  int ntile = 0;
  RUN(K_GEMM_LM, (launch_lm_head<T, A>(h_in, (const T *)lm_head, R, V, D, logits,
                                       ws.tile_max, &ntile, ws.aux, stream)));
  VocabArgs va{};
  va.logits = logits;
  va.q = draft_q;
  va.q_scalar = nullptr;
  va.tile_max = ntile ? ws.tile_max : nullptr;
  va.ntile = ntile;
  va.cand = ws.cand;
  va.cand_cap = ws.cand_cap;
  va.rowflag = ws.rowflag;
  va.u = uniforms;
  va.tok = draft;
  va.par = nullptr;
  va.n1 = 1;
  va.tail = 1;
  va.rows = R;
  va.V = V;
  va.k = p->top_k;
  set_temperature(va, p->temperature);
  va.top_p = p->top_p;
  va.accept = o->accept;
  va.resample = o->resample_token;
  va.bonus = o->bonus_token;
  va.topk_ids = o->topk_ids;
  va.topk_probs = o->topk_probs;
  RUN(K_VOCAB, launch_vocab(va, stream));
  RUN(K_WALK, launch_walk_tail(o->accept, o->resample_token, draft, ws.rowflag, R,
                               chain_len, V, o->acc_prefix_len, o->path, o->path_len,
                               o->next_token, o->sibling_hit, o->status, stream));
  return ACESPEC_OK;
}

template <typename T>
int verify_tail_impl(acespec_ctx *ctx, const void *lm_head, int packed, const void *final_norm,
                     const void *hidden, const int32_t *draft, const float *draft_q,
                     const float *uniforms, int R, int chain_len, const acespec_params *p,
                     const acespec_outputs *o, hipStream_t stream) {
  const TailWorkspace ws{ctx->logits, ctx->tile_max, ctx->cand, kCandCap, ctx->rowflag, ctx->a,
                         GemmAux{ctx->gpart, ctx->gpart_cap, ctx->cus, packed}};
  return verify_tail_run<T>(ctx, ctx->d, ws, lm_head, final_norm, hidden, draft, draft_q,
                            uniforms, R, chain_len, p, o, stream);
}

}  // namespace

extern "C" {

const char *acespec_last_error(void) { return g_err.c_str(); }

int acespec_create(const acespec_model_desc *desc, int max_batch, int max_nodes,
                   acespec_ctx **out) {
  g_err.clear();
  if (!desc || !out) return fail(ACESPEC_EINVAL, "desc and out must be non-NULL");
  *out = nullptr;
  const acespec_model_desc &d = *desc;
  if (d.dtype != ACESPEC_F32 && d.dtype != ACESPEC_BF16)
    return fail(ACESPEC_EINVAL, "unknown dtype %d", (int)d.dtype);
  if (max_batch < 1 || max_nodes < 0)
    return fail(ACESPEC_EINVAL, "max_batch >= 1 and max_nodes >= 0 required");
  if (max_nodes > 64) return fail(ACESPEC_EUNSUPPORTED, "max_nodes > 64 is not supported");
  if (d.n_layers < 0 || d.d_model < 64 || d.d_model % 64 || d.vocab < 1 || d.vocab % 4 ||
      d.vocab > 262144)
    return fail(ACESPEC_EUNSUPPORTED,
                "need d_model a multiple of 64, vocab a multiple of 4 and <= 262144");
  if (d.n_layers > 0) {
    if (d.head_dim != 64 && d.head_dim != 128)
      return fail(ACESPEC_EUNSUPPORTED, "head_dim must be 64 or 128 (got %d)", d.head_dim);
    if (d.n_heads < 1 || d.n_kv_heads < 1 || d.n_heads % d.n_kv_heads)
      return fail(ACESPEC_EINVAL, "n_heads must be a positive multiple of n_kv_heads");
    if (d.d_ff < 64 || d.d_ff % 64 || (d.n_heads * d.head_dim) % 64)
      return fail(ACESPEC_EUNSUPPORTED, "d_ff and n_heads*head_dim must be multiples of 64");
    if (!(d.rope_base > 0.f) || !(d.rms_eps >= 0.f))
      return fail(ACESPEC_EINVAL, "rope_base > 0 and rms_eps >= 0 required");
  }
  acespec_ctx *c = new (std::nothrow) acespec_ctx();
  if (!c) return fail(ACESPEC_ENOMEM, "host allocation failed");
  c->d = d;
  c->max_batch = max_batch;
  c->max_nodes = max_nodes;
  c->max_rows = max_batch * (max_nodes + 1);
  c->esz = d.dtype == ACESPEC_BF16 ? 2 : 4;  // bytes per activation (fp16 or fp32)
  const size_t R = c->max_rows;
  const bool layers = d.n_layers > 0;
  const int G = layers ? d.n_heads / d.n_kv_heads : 1;
  const size_t QR = (size_t)G * (max_nodes + 1);
  c->part_cap = layers ? ((long long)max_batch * d.n_kv_heads + 512) * QR * d.head_dim : 0;
  struct Part { size_t bytes; void **dst; };
  void *p_x = nullptr, *p_logits = nullptr, *p_po = nullptr, *p_pml = nullptr, *p_if = nullptr;
  void *p_qkv = nullptr, *p_gpart = nullptr, *p_rot = nullptr, *p_tmax = nullptr,
       *p_cand = nullptr, *p_rflag = nullptr;
  void *p_tok = nullptr, *p_par = nullptr, *p_pos = nullptr, *p_depth = nullptr,
       *p_anc = nullptr, *p_S = nullptr;
  std::vector<Part> parts = {
      {R * d.d_model * 4, &p_x},
      {R * d.d_model * c->esz, &c->a},
      {layers ? R * d.n_heads * d.head_dim * c->esz : 0, &c->attn},
      {layers ? R * (d.n_heads + 2 * d.n_kv_heads) * d.head_dim * 4 : 0, &p_qkv},
      {layers ? R * d.n_heads * d.head_dim * c->esz : 0, &c->q},
      {layers ? R * d.d_ff * c->esz : 0, &c->h},
      {R * (size_t)d.vocab * 4, &p_logits},
      {R * (size_t)((d.vocab + 127) / 128) * 4, &p_tmax},
      {R * (size_t)kCandCap * 4, &p_cand},
      {R * 4, &p_rflag},
      {(size_t)c->part_cap * 4, &p_po},
      {(size_t)c->part_cap / (layers ? d.head_dim : 1) * 2 * 4, &p_pml},
      {layers ? (size_t)d.head_dim / 2 * 8 : 0, &p_if},
      {layers ? R * (size_t)d.head_dim / 2 * 8 : 0, &p_rot},
      {(size_t)8 * R * d.d_model * 4, &p_gpart},
      {R * 4, &p_tok}, {R * 4, &p_par}, {R * 4, &p_pos}, {R * 4, &p_depth}, {R * 8, &p_anc},
      {(size_t)max_batch * 4, &p_S}};
  size_t total = 0;
  for (auto &pt : parts) total += align_up(pt.bytes);
  if (hipMalloc(&c->ws, total) != hipSuccess) {
    (void)hipGetLastError();
    delete c;
    return fail(ACESPEC_ENOMEM, "hipMalloc of %zu workspace bytes failed", total);
  }
  size_t off = 0;
  for (auto &pt : parts) {
    *pt.dst = pt.bytes ? (char *)c->ws + off : nullptr;
    off += align_up(pt.bytes);
  }
  c->x = (float *)p_x;
  c->qkv = (float *)p_qkv;
  c->gpart = (float *)p_gpart;
  c->gpart_cap = (long long)8 * R * d.d_model;
  {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0)
      c->cus = n;
  }
  c->logits = (float *)p_logits;
  c->part_o = (float *)p_po;
  c->part_ml = (float *)p_pml;
  c->inv_freq = (double *)p_if;
  c->rot = (float2 *)p_rot;
  c->tile_max = (float *)p_tmax;
  c->cand = (uint32_t *)p_cand;
  c->rowflag = (int32_t *)p_rflag;
  c->meta.tok = (int32_t *)p_tok;
  c->meta.par = (int32_t *)p_par;
  c->meta.pos = (int32_t *)p_pos;
  c->meta.depth = (int32_t *)p_depth;
  c->meta.anc = (uint64_t *)p_anc;
  c->meta.sess_S = (int32_t *)p_S;
  if (layers) {
    std::vector<double> f(d.head_dim / 2);
    for (int i = 0; i < d.head_dim / 2; ++i)
      f[i] = std::pow((double)d.rope_base, -2.0 * i / (double)d.head_dim);
    if (hipMemcpy(c->inv_freq, f.data(), f.size() * 8, hipMemcpyHostToDevice) != hipSuccess) {
      (void)hipFree(c->ws);
      delete c;
      return fail(ACESPEC_EHIP, "copy of the RoPE frequency table failed");
    }
  }
  *out = c;
  return ACESPEC_OK;
}

void acespec_destroy(acespec_ctx *c) {
  if (!c) return;
  (void)hipDeviceSynchronize();
  for (auto &r : c->pending) {
    (void)hipEventDestroy(r.e0);
    (void)hipEventDestroy(r.e1);
  }
  for (auto e : c->free_events) (void)hipEventDestroy(e);
  (void)hipFree(c->ws);
  delete c;
}

}  // extern "C"

namespace {

// Shared argument checks and dispatch of the two verify_tree entry points (dense draft
// distributions, or the scalar q-hat of each drafted token).
int verify_tree_checked(acespec_ctx *ctx, const acespec_weights *w, const acespec_kv_cache *kv,
                        const int32_t *tree_tokens, const int32_t *parent_idx,
                        const float *draft_q, const float *q_scalar, const float *uniforms,
                        int B, int N, const acespec_params *p, const acespec_outputs *o,
                        hipStream_t stream) {
  g_err.clear();
  if (!ctx) return fail(ACESPEC_EINVAL, "ctx is NULL");
  const acespec_model_desc &d = ctx->d;
  if (d.n_layers < 1) return fail(ACESPEC_EINVAL, "context has no layers (tail-only model)");
  if (!w || !kv || !tree_tokens || !parent_idx || !(draft_q || q_scalar) || !uniforms)
    return fail(ACESPEC_EINVAL, "a required pointer is NULL");
  if (!w->embed || !w->layers || !w->final_norm || !w->lm_head)
    return fail(ACESPEC_EINVAL, "a weight pointer is NULL");
  for (int l = 0; l < d.n_layers; ++l) {
    const acespec_layer_weights &lw = w->layers[l];
    if (!lw.attn_norm || !lw.wqkv || !lw.wo || !lw.mlp_norm || !lw.w_gate_up || !lw.w_down)
      return fail(ACESPEC_EINVAL, "layer %d has a NULL weight pointer", l);
  }
  {
    const int rc = check_layout(w->layout, d);
    if (rc) return rc;
  }
  if (!kv->k || !kv->v || !kv->prefix_len) return fail(ACESPEC_EINVAL, "kv cache pointer NULL");
  if (B < 1 || B > ctx->max_batch)
    return fail(ACESPEC_EINVAL, "B must be in [1, %d] (got %d)", ctx->max_batch, B);
  if (N < 0 || N > ctx->max_nodes)
    return fail(N > 64 ? ACESPEC_EUNSUPPORTED : ACESPEC_EINVAL,
                "N must be in [0, %d] (got %d)", ctx->max_nodes, N);
  if (kv->capacity < N + 1)
    return fail(ACESPEC_EINVAL, "kv capacity %d cannot hold the %d tree rows", kv->capacity, N + 1);
  if (kv->capacity % 64 != 0)
    return fail(ACESPEC_EINVAL, "kv capacity must be a multiple of 64 (got %d)", kv->capacity);
  int rc = check_params(p, d.vocab);
  if (rc) return rc;
  rc = check_outputs(o);
  if (rc) return rc;
  if (d.dtype == ACESPEC_BF16)
    return verify_tree_impl<bf16>(ctx, w, kv, tree_tokens, parent_idx, draft_q, q_scalar,
                                  uniforms, B, N, p, o, stream);
  return verify_tree_impl<float>(ctx, w, kv, tree_tokens, parent_idx, draft_q, q_scalar,
                                 uniforms, B, N, p, o, stream);
}

}  // namespace

namespace acespec {
// commit.hip: each of `planes` [rows][cols] matrices of elem_bytes-wide elements (2 or 4),
// written transposed as [cols][rows] to dst (no overlap).
hipError_t launch_transpose_planes(const void *src, void *dst, int elem_bytes, int planes,
                                   int rows, int cols, hipStream_t s);
}  // namespace acespec

extern "C" {

int acespec_verify_tree(acespec_ctx *ctx, const acespec_weights *w, const acespec_kv_cache *kv,
                        const int32_t *tree_tokens, const int32_t *parent_idx,
                        const float *draft_q, const float *uniforms, int B, int N,
                        const acespec_params *p, const acespec_outputs *o,
                        hipStream_t stream) {
  if (!draft_q) {
    g_err.clear();
    return fail(ACESPEC_EINVAL, "draft_q is NULL");
  }
  return verify_tree_checked(ctx, w, kv, tree_tokens, parent_idx, draft_q, nullptr, uniforms, B,
                             N, p, o, stream);
}

int acespec_verify_tree_scalar_q(acespec_ctx *ctx, const acespec_weights *w,
                                 const acespec_kv_cache *kv, const int32_t *tree_tokens,
                                 const int32_t *parent_idx, const float *q_hat,
                                 const float *uniforms, int B, int N, const acespec_params *p,
                                 const acespec_outputs *o, hipStream_t stream) {
  if (!q_hat) {
    g_err.clear();
    return fail(ACESPEC_EINVAL, "q_hat is NULL");
  }
  return verify_tree_checked(ctx, w, kv, tree_tokens, parent_idx, nullptr, q_hat, uniforms, B,
                             N, p, o, stream);
}

int acespec_pack_weight(const void *src, void *dst, int rows, int cols, hipStream_t stream) {
  g_err.clear();
  if (!src || !dst) return fail(ACESPEC_EINVAL, "src or dst is NULL");
  if (rows < 16 || cols < 32 || rows % 16 != 0 || cols % 32 != 0)
    return fail(ACESPEC_EINVAL, "rows must be a positive multiple of 16 and cols of 32 (got %d x %d)",
                rows, cols);
  const char *s0 = (const char *)src, *d0 = (const char *)dst;
  const size_t bytes = (size_t)rows * cols * 2;
  if (s0 < d0 + bytes && d0 < s0 + bytes) return fail(ACESPEC_EINVAL, "src and dst overlap");
  const hipError_t e = launch_pack_weights((const bf16 *)src, (f16 *)dst, rows, cols, stream);
  if (e != hipSuccess) return fail(ACESPEC_EHIP, "pack launch: %s", hipGetErrorString(e));
  return ACESPEC_OK;
}

int acespec_convert_v_cache(const void *src, void *dst, int planes, int capacity, int head_dim,
                            acespec_dtype dtype, acespec_v_direction direction,
                            hipStream_t stream) {
  g_err.clear();
  if (!src || !dst) return fail(ACESPEC_EINVAL, "src or dst is NULL");
  if (dtype != ACESPEC_BF16 && dtype != ACESPEC_F32)
    return fail(ACESPEC_EINVAL, "dtype must be ACESPEC_BF16 or ACESPEC_F32 (got %d)", (int)dtype);
  if (direction != ACESPEC_V_TO_HEAD_DIM_MAJOR && direction != ACESPEC_V_TO_SLOT_MAJOR)
    return fail(ACESPEC_EINVAL, "unknown direction %d", (int)direction);
  if (planes < 1 || head_dim < 1 || capacity < 64 || capacity % 64 != 0)
    return fail(ACESPEC_EINVAL,
                "planes and head_dim must be >= 1 and capacity a positive multiple of 64 "
                "(got %d, %d, %d)", planes, head_dim, capacity);
  const int eb = dtype == ACESPEC_BF16 ? 2 : 4;
  const long long tiles = (long long)planes * ((capacity + 31) / 32) * ((head_dim + 31) / 32);
  if (tiles > 0x7fffffffLL)
    return fail(ACESPEC_EINVAL, "%lld tiles of 32 x 32 exceed one launch: convert in parts", tiles);
  const size_t bytes = (size_t)planes * capacity * head_dim * eb;
  const char *s0 = (const char *)src, *d0 = (const char *)dst;
  if (s0 < d0 + bytes && d0 < s0 + bytes) return fail(ACESPEC_EINVAL, "src and dst overlap");
  const bool to_hd = direction == ACESPEC_V_TO_HEAD_DIM_MAJOR;
  const hipError_t e = acespec::launch_transpose_planes(src, dst, eb, planes, to_hd ? capacity : head_dim,
                                               to_hd ? head_dim : capacity, stream);
  if (e != hipSuccess) return fail(ACESPEC_EHIP, "convert launch: %s", hipGetErrorString(e));
  return ACESPEC_OK;
}

int acespec_verify_tail(acespec_ctx *ctx, const void *lm_head, acespec_layout lm_head_layout,
                        const void *final_norm, const void *hidden, const int32_t *draft_tokens,
                        const float *draft_q, const float *uniforms, int R, int chain_len,
                        const acespec_params *p, const acespec_outputs *o,
                        hipStream_t stream) {
  g_err.clear();
  if (!ctx) return fail(ACESPEC_EINVAL, "ctx is NULL");
  if (!lm_head || !hidden || !draft_tokens || !draft_q || !uniforms)
    return fail(ACESPEC_EINVAL, "a required pointer is NULL");
  int rc = check_layout(lm_head_layout, ctx->d);
  if (rc) return rc;
  const int packed = lm_head_layout == ACESPEC_LAYOUT_PACKED ? 1 : 0;
  if (R < 1 || R > ctx->max_rows)
    return fail(ACESPEC_EINVAL, "R must be in [1, %d] (got %d)", ctx->max_rows, R);
  if (chain_len < 1 || R % chain_len)
    return fail(ACESPEC_EINVAL, "chain_len must be >= 1 and divide R");
  rc = check_params(p, ctx->d.vocab);
  if (rc) return rc;
  rc = check_outputs(o);
  if (rc) return rc;
  if (ctx->d.dtype == ACESPEC_BF16)
    return verify_tail_impl<bf16>(ctx, lm_head, packed, final_norm, hidden, draft_tokens,
                                  draft_q, uniforms, R, chain_len, p, o, stream);
  return verify_tail_impl<float>(ctx, lm_head, packed, final_norm, hidden, draft_tokens,
                                 draft_q, uniforms, R, chain_len, p, o, stream);
}

int acespec_commit_kv(acespec_ctx *ctx, const acespec_kv_cache *kv, const int32_t *path,
                      const int32_t *path_len, const int32_t *status, int B, int N,
                      int32_t *new_prefix_len, hipStream_t stream) {
  g_err.clear();
  if (!kv || !kv->k || !kv->v || !kv->prefix_len || !path || !path_len || !new_prefix_len)
    return fail(ACESPEC_EINVAL, "a required pointer is NULL (only status may be)");
  if (B < 1) return fail(ACESPEC_EINVAL, "B must be >= 1 (got %d)", B);
  {
    // The kernel's workgroups read prefix_len[b] while one of them writes
    // new_prefix_len[b]: the two arrays must be distinct memory.
    const uintptr_t a0 = (uintptr_t)kv->prefix_len, n0 = (uintptr_t)new_prefix_len;
    const uintptr_t bytes = (uintptr_t)B * sizeof(int32_t);
    if (a0 < n0 + bytes && n0 < a0 + bytes)
      return fail(ACESPEC_EINVAL,
                  "new_prefix_len overlaps kv->prefix_len: give it its own buffer and copy "
                  "it over after the call");
  }
  if (!ctx) return fail(ACESPEC_EINVAL, "ctx is NULL");
  if (ctx->d.n_layers < 1) return fail(ACESPEC_EINVAL, "the model has no layers (no KV cache)");
  if (B > ctx->max_batch)
    return fail(ACESPEC_EINVAL, "B must be in [1, %d] (got %d)", ctx->max_batch, B);
  if (N < 0 || N > ctx->max_nodes)
    return fail(ACESPEC_EINVAL, "N must be in [0, %d] (got %d)", ctx->max_nodes, N);
  if (kv->capacity < N + 1)
    return fail(ACESPEC_EINVAL, "kv capacity %d cannot hold the %d tree rows", kv->capacity, N + 1);
  const acespec_model_desc &d = ctx->d;
  if (d.dtype == ACESPEC_BF16)
    RUN(K_COMMIT, launch_commit_kv<bf16>((bf16 *)kv->k, (bf16 *)kv->v, kv->prefix_len, path,
                                         path_len, status, d.n_layers, B, N + 1, d.n_kv_heads,
                                         d.head_dim, kv->capacity, new_prefix_len, stream));
  else
    RUN(K_COMMIT, launch_commit_kv<float>((float *)kv->k, (float *)kv->v, kv->prefix_len, path,
                                          path_len, status, d.n_layers, B, N + 1, d.n_kv_heads,
                                          d.head_dim, kv->capacity, new_prefix_len, stream));
  return ACESPEC_OK;
}

int acespec_timing_enable(acespec_ctx *ctx, int enable) {
  if (!ctx) return fail(ACESPEC_EINVAL, "ctx is NULL");
  ctx->timing = enable != 0;
  return ACESPEC_OK;
}

int acespec_timing_only(acespec_ctx *ctx, const char *kind) {
  if (!ctx) return fail(ACESPEC_EINVAL, "ctx is NULL");
  if (!kind) {
    ctx->timing_mask = ~0u;
    return ACESPEC_OK;
  }
  for (int k = 0; k < K_COUNT; ++k)
    if (std::strcmp(kind, kKindNames[k]) == 0) {
      ctx->timing_mask = 1u << k;
      return ACESPEC_OK;
    }
  return fail(ACESPEC_EINVAL, "unknown kernel kind '%s'", kind);
}

int acespec_timing_read(acespec_ctx *ctx, const char **names, double *total_ms, int *launches,
                        int max) {
  if (!ctx) return fail(ACESPEC_EINVAL, "ctx is NULL");
  for (auto &r : ctx->pending) {
    if (hipEventSynchronize(r.e1) != hipSuccess) return fail(ACESPEC_EHIP, "event wait failed");
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, r.e0, r.e1) != hipSuccess)
      return fail(ACESPEC_EHIP, "hipEventElapsedTime failed");
    ctx->tot_ms[r.kind] += ms;
    ctx->launches[r.kind] += 1;
    ctx->free_events.push_back(r.e0);
    ctx->free_events.push_back(r.e1);
  }
  ctx->pending.clear();
  int n = 0;
  for (int k = 0; k < K_COUNT && n < max; ++k) {
    if (!ctx->launches[k]) continue;
    if (names) names[n] = kKindNames[k];
    if (total_ms) total_ms[n] = ctx->tot_ms[k];
    if (launches) launches[n] = ctx->launches[k];
    ++n;
  }
  for (int k = 0; k < K_COUNT; ++k) {
    ctx->tot_ms[k] = 0.0;
    ctx->launches[k] = 0;
  }
  return n;
}

}  // extern "C"

// ------------------------------------------------------------------------------------
// Allocation-free LM-head verify (acespec_verify_tail_noalloc)
// ------------------------------------------------------------------------------------
// Its intermediate data lives in a file-scope device array, one copy per device, held
// until the process ends.  On the host the array's name is not a device address: the
// address comes from hipGetSymbolAddress, taken once per device with that device current,
// and only that address is ever handed to kernels.  Calls on one device share the array,
// so calls that overlap in time on one device race.
namespace {

constexpr size_t kScratchBytes = (size_t)48 << 20;
__device__ __align__(256) char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
char *g_scratch_ptr[kMaxDevices] = {};
int g_scratch_cus[kMaxDevices] = {};

int scratch_of_current_device(char **ptr, int *cus) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return fail(ACESPEC_EHIP, "hipGetDevice failed");
  if (dev < 0 || dev >= kMaxDevices)
    return fail(ACESPEC_EUNSUPPORTED, "device %d is beyond the %d the scratch table holds", dev,
                kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(ACESPEC_EHIP, "hipGetSymbolAddress(scratch) failed on device %d: %s", dev,
                  hipGetErrorString(e));
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        n <= 0)
      n = 256;
    g_scratch_ptr[dev] = (char *)p;
    g_scratch_cus[dev] = n;
  }
  *ptr = g_scratch_ptr[dev];
  *cus = g_scratch_cus[dev];
  return ACESPEC_OK;
}

}  // namespace

extern "C" {

int acespec_verify_tail_noalloc(const acespec_model_desc *desc, const void *lm_head,
                                acespec_layout lm_head_layout, const void *final_norm,
                                const void *hidden,
                                const int32_t *draft_tokens, const float *draft_q,
                                const float *uniforms, int R, int chain_len,
                                const acespec_params *p, const acespec_outputs *o,
                                hipStream_t stream) {
  g_err.clear();
  if (!desc) return fail(ACESPEC_EINVAL, "desc is NULL");
  const acespec_model_desc &d = *desc;
  if (d.dtype != ACESPEC_F32 && d.dtype != ACESPEC_BF16)
    return fail(ACESPEC_EINVAL, "unknown dtype %d", (int)d.dtype);
  if (d.d_model < 64 || d.d_model % 64 || d.vocab < 1 || d.vocab % 4 || d.vocab > 262144)
    return fail(ACESPEC_EUNSUPPORTED,
                "need d_model a multiple of 64, vocab a multiple of 4 and <= 262144");
  if (!lm_head || !hidden || !draft_tokens || !draft_q || !uniforms)
    return fail(ACESPEC_EINVAL, "a required pointer is NULL");
  int rc = check_layout(lm_head_layout, d);
  if (rc) return rc;
  if (R < 1) return fail(ACESPEC_EINVAL, "R must be >= 1 (got %d)", R);
  if (chain_len < 1 || R % chain_len)
    return fail(ACESPEC_EINVAL, "chain_len must be >= 1 and divide R");
  rc = check_params(p, d.vocab);
  if (rc) return rc;
  rc = check_outputs(o);
  if (rc) return rc;
  if (!o->logits_out)
    return fail(ACESPEC_EINVAL, "logits_out is required here: the logits are written there");
  // scratch layout: row flags, LM-head row maxima per 128-column tile, the hidden states
  // in the activation type (bf16 model, or any model with a final norm), and the
  // vocabulary kernel's candidate lists when they still fit
  const size_t esz = d.dtype == ACESPEC_BF16 ? 2 : 4;
  const bool need_a = d.dtype == ACESPEC_BF16 || final_norm != nullptr;
  const size_t b_flag = align_up((size_t)R * 4);
  const size_t b_tmax = align_up((size_t)R * ((d.vocab + 127) / 128) * 4);
  const size_t b_a = need_a ? align_up((size_t)R * d.d_model * esz) : 0;
  const size_t b_cand = align_up((size_t)R * kCandCap * 4);
  const size_t need = b_flag + b_tmax + b_a;
  if (need > kScratchBytes)
    return fail(ACESPEC_EINVAL,
                "R = %d rows of d_model %d and vocab %d need %zu scratch bytes; the "
                "allocation-free entry point holds %zu (use acespec_verify_tail)",
                R, d.d_model, d.vocab, need, kScratchBytes);
  char *base = nullptr;
  int cus = 256;
  rc = scratch_of_current_device(&base, &cus);
  if (rc) return rc;
  const bool cand = need + b_cand <= kScratchBytes;
  TailWorkspace ws{nullptr,
                   (float *)(base + b_flag),
                   cand ? (uint32_t *)(base + need) : nullptr,
                   cand ? kCandCap : 0,
                   (int32_t *)base,
                   need_a ? (void *)(base + b_flag + b_tmax) : nullptr,
                   GemmAux{nullptr, 0, cus, lm_head_layout == ACESPEC_LAYOUT_PACKED ? 1 : 0}};
  if (d.dtype == ACESPEC_BF16)
    return verify_tail_run<bf16>(nullptr, d, ws, lm_head, final_norm, hidden, draft_tokens,
                                 draft_q, uniforms, R, chain_len, p, o, stream);
  return verify_tail_run<float>(nullptr, d, ws, lm_head, final_norm, hidden, draft_tokens,
                                draft_q, uniforms, R, chain_len, p, o, stream);
}

}  // extern "C"
