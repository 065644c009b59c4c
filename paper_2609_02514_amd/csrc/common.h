// Shared device helpers and the internal launch interface of the verify library.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/acespec.h"

typedef __bf16 bf16;
typedef _Float16 f16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Storage of a bf16 model: weights and KV cache in bf16; activations handed from one
// kernel to the next in fp16 (same MFMA rate on gfx950, 3 more mantissa bits: the
// rounding of activations is what dominates the logit error of a deep bf16 decoder).
// An fp32 model keeps everything in fp32.
template <typename TW> struct ActOf { typedef f16 type; };
template <> struct ActOf<float> { typedef float type; };

#define AS_DEVICE __device__ __forceinline__

template <typename T> AS_DEVICE float to_f32(T v);
template <> AS_DEVICE float to_f32<float>(float v) { return v; }
template <> AS_DEVICE float to_f32<bf16>(bf16 v) { return (float)v; }
template <> AS_DEVICE float to_f32<f16>(f16 v) { return (float)v; }

template <typename T> AS_DEVICE T from_f32(float v);
template <> AS_DEVICE float from_f32<float>(float v) { return v; }
template <> AS_DEVICE bf16 from_f32<bf16>(float v) { return (bf16)v; }  // RNE
template <> AS_DEVICE f16 from_f32<f16>(float v) { return (f16)v; }     // RNE

// Exact for values in the fp16 normal range (bf16 has 8 significant bits, fp16 11).
AS_DEVICE f16x8 bf16x8_to_f16x8(bf16x8 v) {
  f16x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = (f16)(float)v[i];
  return r;
}

// Order-preserving map of an fp32 value to uint32 (larger float -> larger key).
AS_DEVICE uint32_t f32_key(float f) {
  const uint32_t u = __float_as_uint(f);
  // negative: all bits flipped; otherwise the sign bit set
  return u ^ ((uint32_t)((int32_t)u >> 31) | 0x80000000u);
}

// Running maximum that turns any non-finite value (NaN or +-inf) into +inf, so that a
// maximum over logits also reports whether one of them overflowed.
AS_DEVICE float max_or_inf(float m, float v) {
  return fabsf(v) <= 3.402823466e38f ? fmaxf(m, v) : __builtin_inff();
}

AS_DEVICE float wave_max(float v) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
// Reductions over the four lanes l, l^16, l^32, l^48 (one value per 16-lane row), with
// gfx950's row-swap permutes instead of LDS-routed shuffles: after the 16-lane swap of
// v with itself, the two results hold the even and the odd rows, so combining them
// reduces each xor-16 pair; the 32-lane swap then does the same for the halves.
AS_DEVICE float rows4_max(float v) {
  auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
  auto q = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(q[0]), __uint_as_float(q[1]));
}
AS_DEVICE float rows4_sum(float v) {
  auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(p[0]) + __uint_as_float(p[1]);
  auto q = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(q[0]) + __uint_as_float(q[1]);
}

AS_DEVICE float wave_sum(float v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
AS_DEVICE unsigned long long wave_sum_u64(unsigned long long v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
AS_DEVICE int wave_sum_i32(int v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// ------------------------------------------------------------------------------------
// Direct global -> LDS staging (gfx950)
// ------------------------------------------------------------------------------------
typedef __attribute__((address_space(3))) void *lds_ptr_t;

// A 16-byte global load with the nontemporal cache policy (last read of a stream).
typedef float f32x4v __attribute__((ext_vector_type(4)));
AS_DEVICE float4 ld_stream(const float *p) {
  const f32x4v t = __builtin_nontemporal_load((const f32x4v *)p);
  return make_float4(t.x, t.y, t.z, t.w);
}

// One wave copies 64 x 16 bytes through a buffer resource: lane i reads rsrc + voff + soff
// (soff scalar, so a moving k offset costs no vector arithmetic) and the bytes land at
// l + 16 i (l is wave-uniform); reads past the resource's size return 0.  Completion is
// counted by vmcnt like any load.
AS_DEVICE void buf_dma16(__amdgpu_buffer_rsrc_t rsrc, lds_ptr_t l, uint32_t voff, int soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, l, 16, voff, soff, 0, 0);
}
// The same with the nontemporal cache policy, for data read once per step (the KV cache):
// measured on MI355X, streaming reads with it run at about 6.4 TB/s against 5.0-5.4 TB/s
// without (they do not allocate in L2 or the MALL).  Unlike the global-address form of the
// LDS DMA, the compiler counts this one on vmcnt alone, so its waits for LDS reads issued
// after it stay exact instead of waiting for every outstanding LDS access.
AS_DEVICE void buf_dma16_stream(__amdgpu_buffer_rsrc_t rsrc, lds_ptr_t l, uint32_t voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, l, 16, voff, 0, 0, 2 /* nt */);
}
AS_DEVICE __amdgpu_buffer_rsrc_t make_rsrc(const void *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes,
                                           0x00020000);
}

// Waits until at most VM vector-memory loads of this wave are outstanding (leaves the
// LDS and export counters alone).
template <int VM> AS_DEVICE void wait_vmcnt() {
  static_assert(VM >= 0 && VM < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((VM & 0xF) | ((VM >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Waits until no LDS or scalar memory access of this wave is outstanding.  Before a loop
// it spares the loop's LDS reads a full wait on every iteration: the compiler merges the
// counter state of the code before the loop (scalar loads of kernel arguments, which
// complete out of order) into the loop head, where it then cannot count LDS reads.
AS_DEVICE void wait_lgkmcnt0() { __builtin_amdgcn_s_waitcnt((0xF) | (0x3 << 14) | (0x7 << 4)); }

// Workgroup barrier that orders LDS accesses only: unlike __syncthreads() it does not
// drain outstanding global loads, so DMA into other stages stays in flight.
AS_DEVICE void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

#define SCHED_FENCE() __builtin_amdgcn_sched_barrier(0)

// ------------------------------------------------------------------------------------
// Tree metadata produced by the tree-prep kernel (one entry per tree row)
// ------------------------------------------------------------------------------------
struct TreeMeta {
  int32_t *tok;      // [rows] token id, clamped into [0, V)
  int32_t *par;      // [rows] parent row within the session (-1 for the root); a chain
                     //        for sessions whose tree is malformed
  int32_t *pos;      // [rows] RoPE position = prefix_len + depth
  int32_t *depth;    // [rows]
  uint64_t *anc;     // [rows] bit (j-1) set iff drafted row j is r or an ancestor of r
  int32_t *sess_S;   // [B] prefix length, clamped so that S + N + 1 <= capacity
};

// Fixed-point scale for deterministic mass sums in the vocabulary kernel.
#define AS_FX_SCALE 1099511627776.0f  /* 2^40 */

// ------------------------------------------------------------------------------------
// Launchers (defined in the kernel translation units)
// ------------------------------------------------------------------------------------
namespace acespec {

hipError_t launch_tree_prep(const int32_t *tokens, const int32_t *parents,
                            const int32_t *prefix_len, int B, int n1, int V, int capacity,
                            TreeMeta meta, int32_t *status, hipStream_t s);

template <typename TW>
hipError_t launch_embed(const TW *embed, const int32_t *tok, float *x, int rows, int d,
                        hipStream_t s);

// y = x / sqrt(mean(x^2) + eps) * gain, rounded once to the activation type.
template <typename TW, typename TIN>
hipError_t launch_rmsnorm(const TIN *x, const TW *gain, typename ActOf<TW>::type *out, int rows,
                          int d, float eps, hipStream_t s);

// RoPE on q and k of the fp32 QKV projection; q goes to q_out (activation type,
// [rows, H*hd]), k and v to the cache slots of the tree rows (keys [B][Hkv][cap][hd],
// values head-dim-major [B][Hkv][hd][cap]).
// rot[row * hd/2 + i] = (cos, sin) of pos[row] * inv_freq[i], evaluated in double and
// rounded to fp32 (positions are fixed for the whole step, so one table serves all layers).
hipError_t launch_rope_table(const int32_t *pos, const double *inv_freq, float2 *rot, int rows,
                             int half, hipStream_t s);
template <typename TW>
hipError_t launch_rope_kv(const float *qkv, typename ActOf<TW>::type *q_out,
                          const TreeMeta &meta, TW *cache_k, TW *cache_v, int B, int n1, int H,
                          int Hkv, int hd, int capacity, const float2 *rot, hipStream_t s);


enum GemmEpi { EPI_STORE = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_F32 = 3, EPI_QKV_ROPE = 4,
               EPI_F32_MAX = 5 };

// C[M, N] = A[M, K] . W[N, K]^T with the epilogue:
//  EPI_STORE : out (activation type) [M, N]
//  EPI_RESID : resid (fp32) [M, N] += C
//  EPI_SWIGLU: W holds 2F rows (gate, up); out[M, F] = silu(gate) * up, N = F
//  EPI_F32   : outf (fp32) [M, N] = C
//  EPI_QKV_ROPE: C is the QKV projection; RoPE, rounding and the cache write of the tree
//              rows happen in the epilogue (see launch_qkv_rope)
//  EPI_F32_MAX: as EPI_F32, and the maximum of every row over each column tile
//              (see launch_lm_head)
// A is in the activation type.  aux.part: fp32 workspace for split-K partials
// (aux.part_cap floats), aux.cus: compute units of the device.
struct GemmAux {
  float *part;
  long long part_cap;
  int cus;
  int packed = 0;  // W is in the packed fragment order of launch_pack_weights
};
// Where the QKV projection's RoPE epilogue puts its results: rotated queries (activation
// type, [rows, H*hd]) and the tree rows' keys and values in their cache slots.
template <typename TW> struct RopeOut {
  typename ActOf<TW>::type *q;
  TW *ck, *cv;
  const float2 *rot;
  const int32_t *sess_S;
  int n1, H, Hkv, hd, capacity;
};
// The QKV projection with RoPE and the cache write fused into its epilogue when the
// product is not sliced along K; otherwise the fp32 projection goes to qkv and the RoPE
// kernel follows.  Results are identical either way.
template <typename TW, typename TA>
hipError_t launch_qkv_rope(const TA *A, const TW *W, int M, int N, int K, float *qkv,
                           const RopeOut<TW> &ro, const TreeMeta &meta, int B,
                           const GemmAux &aux, hipStream_t s);

// The LM head: fp32 logits [M, N] = A . W^T.  When the product is not sliced along K the
// epilogue also writes tile_max[row * ntile + t], the maximum of row `row` over column
// tile t, and *ntile is set (else *ntile = 0): the vocabulary kernel then takes a row's
// maximum from ntile values instead of a pass over the row.
template <typename TW, typename TA>
hipError_t launch_lm_head(const TA *A, const TW *W, int M, int N, int K, float *logits,
                          float *tile_max, int *ntile, const GemmAux &aux, hipStream_t s);

template <typename TW, typename TA>
hipError_t launch_gemm(int epi, const TA *A, const TW *W, int M, int N, int K,
                       typename ActOf<TW>::type *out, float *outf, const GemmAux &aux,
                       hipStream_t s);

// x[M, N] += A . W^T followed by out = RMSNorm(x) * gain (the residual projection and the
// norm that opens the next block).  When the product is sliced along K in every tile the
// slices are summed, added to x and normalised by one row-wise kernel (x is read and
// written once); otherwise the product's own epilogue adds to x and a separate RMSNorm
// follows.  Results are identical either way.
template <typename TW, typename TA>
hipError_t launch_gemm_resid_norm(const TA *A, const TW *W, int M, int N, int K, float *x,
                                  const TW *gain, typename ActOf<TW>::type *out, float eps,
                                  const GemmAux &aux, hipStream_t s);

// The fp16-activation MFMA GEMM (weights TB = bf16, widened to fp16 in registers) with
// an explicit tiling (var >= 0) and split count (splits_override > 0); var < 0 /
// splits_override <= 0 choose automatically.
template <typename TB>
hipError_t launch_f16w_variant(int var, int splits_override, int epi, const f16 *A,
                               const TB *W, int M, int N, int K, f16 *out, float *outf,
                               float *part, long long part_cap, int cus, hipStream_t s,
                               int packed = 0);

// Packs a row-major bf16 weight matrix [rows, K] (rows % 16 == 0, K % 32 == 0) into the
// fp16 MFMA-fragment order the packed GEMM path reads (same byte size).
hipError_t launch_pack_weights(const bf16 *W, f16 *P, int rows, int K, hipStream_t s);

// Exact widening of a bf16 tensor to fp16 (in range), n elements.
hipError_t launch_cast_bf16_f16(const bf16 *in, f16 *out, size_t n, hipStream_t s);

template <typename TW>
hipError_t launch_attention(const typename ActOf<TW>::type *q, const TW *cache_k,
                            const TW *cache_v, const TreeMeta &meta,
                            typename ActOf<TW>::type *out, float *part_o, float *part_ml,
                            long long part_capacity, int B, int n1, int H, int Hkv, int hd,
                            int capacity, int cus, hipStream_t s, int *nsplit_used);

struct VocabArgs {
  const float *logits;      // [rows, V]
  const float *q;           // [rows, V] dense draft distributions (NULL in scalar mode)
  const float *q_scalar;    // [rows] q-hat of each row's own token, or NULL (dense mode)
  const float *tile_max;    // [rows, ntile] row maxima over column tiles, or NULL
  int ntile;
  uint32_t *cand;           // [rows, cand_cap] scratch for threshold-bin candidates, or NULL
  int cand_cap;
  int32_t *rowflag;         // [rows] out: 0, ACESPEC_EBADDRAFT or ACESPEC_ENONFINITE
  const float *u;           // [rows, 3]
  const int32_t *tok;       // [rows] token of each row (children look theirs up here)
  const int32_t *par;       // [rows] parent row within the session, -1 for the root
  int n1;                   // rows per session (1 for the tail)
  int tail;                 // 1: each row is the parent of one drafted token tok[row]
  int rows, V, k;
  // log2(e) / T as an unevaluated pair of floats (c_hi + c_lo, from double on the host):
  // a single fp32 factor would tilt every weight exp2(x c) by x times its rounding error,
  // a systematic shift of the cumulative masses the inverse CDFs read
  float c_hi, c_lo;
  float top_p;
  uint8_t *accept;
  int32_t *resample;
  int32_t *bonus;
  int32_t *topk_ids;
  float *topk_probs;
};
hipError_t launch_vocab(const VocabArgs &a, hipStream_t s);

// The walk also folds the rows' data-error codes (rowflag) into status[b] of sessions
// whose tree was valid.
hipError_t launch_walk(const int32_t *tok, const int32_t *par, const int32_t *depth,
                       const uint8_t *accept, const int32_t *resample, const int32_t *bonus,
                       const int32_t *rowflag, int B, int n1, int32_t *acc_prefix_len,
                       int32_t *path, int32_t *path_len, int32_t *next_token,
                       uint8_t *sibling_hit, int32_t *status, hipStream_t s);

// Algorithm 1 COMPACT_KV: moves the root and kept rows of each session to the slots
// following its prefix; new_len[b] = prefix_len[b] + 1 + path_len[b], or -1 (nothing moved)
// if the session's status or path data is not valid.
template <typename T>
hipError_t launch_commit_kv(T *ck, T *cv, const int32_t *prefix_len, const int32_t *path,
                            const int32_t *path_len, const int32_t *status, int L, int B,
                            int n1, int Hkv, int hd, int capacity, int32_t *new_len,
                            hipStream_t s);

hipError_t launch_walk_tail(const uint8_t *accept, const int32_t *resample,
                            const int32_t *draft, const int32_t *rowflag, int R,
                            int chain_len, int V,
                            int32_t *acc_prefix_len, int32_t *path,
                            int32_t *path_len, int32_t *next_token, uint8_t *sibling_hit,
                            int32_t *status, hipStream_t s);

}  // namespace acespec
