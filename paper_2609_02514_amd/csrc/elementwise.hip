// Embedding gather, RMSNorm, and RoPE with the tree K/V write into the cache.
//
// RMSNorm: y = x / sqrt(mean(x^2) + eps) * gain, fp32 math, rounded once to the
// activation type.  The residual stream x stays fp32 between layers.
// RoPE (rotate-half): the pair (i, i + hd/2) of every query and key head is rotated by
// pos * base^(-2i/hd); the angle and its sine/cosine are evaluated in double so that
// large positions (16k-token prefixes) keep full fp32 accuracy, once per step into a
// (cos, sin) table of fp32 pairs per tree row.  The rotation itself normally runs in the
// QKV projection's epilogue; the kernel here serves the fp32 model and products sliced
// along K.  The projection is rounded once: q to the activation type, k and v to the
// cache dtype.  Tree row r of session b sits at position prefix_len + depth(r) and its
// key/value go to slot prefix_len + r.
#include "common.h"

namespace {

// Four consecutive elements as float4 (the row bases are 16-byte aligned: d % 64 == 0).
AS_DEVICE float4 load4(const float *p, int c) { return *(const float4 *)(p + 4 * c); }
AS_DEVICE float4 load4(const bf16 *p, int c) {
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
  const bf16x4 v = *(const bf16x4 *)(p + 4 * c);
  return make_float4((float)v[0], (float)v[1], (float)v[2], (float)v[3]);
}
AS_DEVICE void store4(float *p, int c, float4 v) { *(float4 *)(p + 4 * c) = v; }
AS_DEVICE void store4(f16 *p, int c, float4 v) {
  typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
  *(f16x4 *)(p + 4 * c) = f16x4{(f16)v.x, (f16)v.y, (f16)v.z, (f16)v.w};
}

// One row per block, four elements a thread per step (d % 64 == 0).
template <typename T>
__global__ void embed_kernel(const T *__restrict__ embed, const int32_t *__restrict__ tok,
                             float *__restrict__ x, int d) {
  const int row = blockIdx.x;
  const T *src = embed + (size_t)tok[row] * d;
  float *dst = x + (size_t)row * d;
  for (int c = threadIdx.x; c < (d >> 2); c += blockDim.x) store4(dst, c, load4(src, c));
}

// One 256-thread block per row; d is a multiple of 64.  A row of up to 8192 values is read
// once (float4 per thread and step, kept in registers), longer rows are read twice.
template <typename Tin, typename TG, typename Tout>
__global__ __launch_bounds__(256) void rmsnorm_kernel(const Tin *__restrict__ x,
                                                      const TG *__restrict__ gain,
                                                      Tout *__restrict__ out, int d, float eps) {
  constexpr int MAXJ = 8;
  const int row = blockIdx.x, tid = threadIdx.x;
  const int d4 = d >> 2;
  const Tin *xr = x + (size_t)row * d;
  float4 v[MAXJ];
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < MAXJ; ++j) {
    const int c = tid + 256 * j;
    if (c < d4) {
      v[j] = load4(xr, c);
      ss += v[j].x * v[j].x + v[j].y * v[j].y + v[j].z * v[j].z + v[j].w * v[j].w;
    }
  }
  for (int c = tid + 256 * MAXJ; c < d4; c += 256) {
    const float4 t = load4(xr, c);
    ss += t.x * t.x + t.y * t.y + t.z * t.z + t.w * t.w;
  }
  __shared__ float red[4];
  ss = wave_sum(ss);
  if ((tid & 63) == 0) red[tid >> 6] = ss;
  __syncthreads();
  const float tot = (red[0] + red[1]) + (red[2] + red[3]);
  const float scale = 1.0f / sqrtf(tot / (float)d + eps);
  Tout *o = out + (size_t)row * d;
#pragma unroll
  for (int j = 0; j < MAXJ; ++j) {
    const int c = tid + 256 * j;
    if (c < d4) {
      const float4 g = load4(gain, c);
      store4(o, c, make_float4(v[j].x * scale * g.x, v[j].y * scale * g.y,
                               v[j].z * scale * g.z, v[j].w * scale * g.w));
    }
  }
  for (int c = tid + 256 * MAXJ; c < d4; c += 256) {
    const float4 t = load4(xr, c), g = load4(gain, c);
    store4(o, c, make_float4(t.x * scale * g.x, t.y * scale * g.y, t.z * scale * g.z,
                             t.w * scale * g.w));
  }
}

__global__ void rope_table_kernel(const int32_t *__restrict__ pos,
                                  const double *__restrict__ inv_freq, float2 *__restrict__ rot,
                                  int rows, int half) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= rows * half) return;
  const int row = idx / half, i = idx - row * half;
  double sd, cd;
  sincos((double)pos[row] * inv_freq[i], &sd, &cd);
  rot[idx] = make_float2((float)cd, (float)sd);
}

// grid: (kv heads, sessions, chunks of ROPE_ROWS tree rows); block: 256 threads.  One block
// rotates ROPE_ROWS tree rows of one session for one kv head and the G query heads that
// share it, so that its value columns land as runs of consecutive slots in the
// head-dim-major value cache.
constexpr int ROPE_ROWS = 16, ROPE_MAX_HALF = 64, ROPE_THREADS = 256;
template <typename TW, typename TA>
__global__ __launch_bounds__(ROPE_THREADS) void rope_kv_kernel(const float *__restrict__ qkv,
                                                      TA *__restrict__ q_out, TreeMeta meta,
                                                      TW *__restrict__ ck, TW *__restrict__ cv,
                                                      int n1, int H, int Hkv, int hd,
                                                      int capacity,
                                                      const float2 *__restrict__ rot) {
  __shared__ float vs[ROPE_ROWS * (2 * ROPE_MAX_HALF + 1)];
  const int g = blockIdx.x, b = blockIdx.y, r0 = blockIdx.z * ROPE_ROWS, tid = threadIdx.x;
  const int nr = min(ROPE_ROWS, n1 - r0);  // rows of this block
  const int half = hd >> 1, G = H / Hkv;
  // item e of a row-major [nr][half] walk -> (row, frequency); shifts when half is a power
  // of two (every bf16 model: head_dim 64 or 128)
  const bool pow2 = (half & (half - 1)) == 0;
  const int lh = __builtin_ctz(half);
  auto split = [&](int e, int &r, int &i) {
    if (pow2) { r = e >> lh; i = e & (half - 1); }
    else { r = e / half; i = e - r * half; }
  };
  const size_t W = (size_t)(H + 2 * Hkv) * hd;  // qkv row width
  const float *base = qkv + ((size_t)b * n1 + r0) * W;
  const float2 *rt = rot + ((size_t)b * n1 + r0) * half;
  for (int e = tid; e < nr * hd; e += ROPE_THREADS) {  // this head's values, row-major
    int r, i;
    split(e >> 1, r, i);                 // (two items of a row per frequency)
    const int dd = e - r * hd;
    vs[r * (hd + 1) + dd] = base[r * W + (size_t)(H + Hkv + g) * hd + dd];
  }
  __syncthreads();
  for (int hh = 0; hh < G; ++hh) {  // queries, one head of the group at a time
    const int h = g * G + hh;
    for (int e = tid; e < nr * half; e += ROPE_THREADS) {
      int r, i;
      split(e, r, i);
      const float *x = base + r * W + (size_t)h * hd;
      const float2 cs = rt[e];
      const float x1 = x[i], x2 = x[i + half];
      TA *qo = q_out + ((size_t)b * n1 + r0 + r) * H * hd + (size_t)h * hd;
      qo[i] = from_f32<TA>(x1 * cs.x - x2 * cs.y);
      qo[i + half] = from_f32<TA>(x2 * cs.x + x1 * cs.y);
    }
  }
  const int S = meta.sess_S[b];
  for (int e = tid; e < nr * half; e += ROPE_THREADS) {  // keys
    int r, i;
    split(e, r, i);
    const float *k = base + r * W + (size_t)(H + g) * hd;
    const float2 cs = rt[e];
    const float x1 = k[i], x2 = k[i + half];
    const size_t kdst = (((size_t)b * Hkv + g) * capacity + S + r0 + r) * hd;
    ck[kdst + i] = from_f32<TW>(x1 * cs.x - x2 * cs.y);
    ck[kdst + i + half] = from_f32<TW>(x2 * cs.x + x1 * cs.y);
  }
  // values: runs of ROPE_ROWS consecutive slots per head dim (consecutive threads,
  // consecutive slots)
  for (int e = tid; e < hd * ROPE_ROWS; e += ROPE_THREADS) {
    const int dd = e / ROPE_ROWS, r = e % ROPE_ROWS;
    if (r < nr)
      cv[(((size_t)b * Hkv + g) * hd + dd) * capacity + S + r0 + r] =
          from_f32<TW>(vs[r * (hd + 1) + dd]);
  }
}

__global__ void cast_bf16_f16_kernel(const bf16x8 *__restrict__ in, f16x8 *__restrict__ out,
                                     size_t n8) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n8) out[i] = bf16x8_to_f16x8(in[i]);
}

}  // namespace

namespace acespec {

hipError_t launch_rope_table(const int32_t *pos, const double *inv_freq, float2 *rot, int rows,
                             int half, hipStream_t s) {
  const int n = rows * half;
  hipLaunchKernelGGL(rope_table_kernel, dim3((n + 255) / 256), dim3(256), 0, s, pos, inv_freq,
                     rot, rows, half);
  return hipGetLastError();
}

hipError_t launch_cast_bf16_f16(const bf16 *in, f16 *out, size_t n, hipStream_t s) {
  const size_t n8 = n / 8;  // n is a multiple of 64 (rows x d_model)
  hipLaunchKernelGGL(cast_bf16_f16_kernel, dim3((n8 + 255) / 256), dim3(256), 0, s,
                     (const bf16x8 *)in, (f16x8 *)out, n8);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_embed(const T *embed, const int32_t *tok, float *x, int rows, int d,
                        hipStream_t s) {
  hipLaunchKernelGGL(embed_kernel<T>, dim3(rows), dim3(256), 0, s, embed, tok, x, d);
  return hipGetLastError();
}

template <typename TW, typename TIN>
hipError_t launch_rmsnorm(const TIN *x, const TW *gain, typename ActOf<TW>::type *out, int rows,
                          int d, float eps, hipStream_t s) {
  hipLaunchKernelGGL((rmsnorm_kernel<TIN, TW, typename ActOf<TW>::type>), dim3(rows), dim3(256),
                     0, s, x, gain, out, d, eps);
  return hipGetLastError();
}

template <typename TW>
hipError_t launch_rope_kv(const float *qkv, typename ActOf<TW>::type *q_out,
                          const TreeMeta &meta, TW *cache_k, TW *cache_v, int B, int n1, int H,
                          int Hkv, int hd, int capacity, const float2 *rot, hipStream_t s) {
  if (hd > 2 * ROPE_MAX_HALF || H % Hkv) return hipErrorInvalidValue;
  hipLaunchKernelGGL((rope_kv_kernel<TW, typename ActOf<TW>::type>),
                     dim3(Hkv, B, (n1 + ROPE_ROWS - 1) / ROPE_ROWS), dim3(ROPE_THREADS),
                     0, s, qkv, q_out, meta, cache_k, cache_v, n1, H, Hkv, hd, capacity, rot);
  return hipGetLastError();
}

template hipError_t launch_embed<float>(const float *, const int32_t *, float *, int, int,
                                        hipStream_t);
template hipError_t launch_embed<bf16>(const bf16 *, const int32_t *, float *, int, int,
                                       hipStream_t);
template hipError_t launch_rmsnorm<float, float>(const float *, const float *, float *, int, int,
                                                 float, hipStream_t);
template hipError_t launch_rmsnorm<bf16, float>(const float *, const bf16 *, f16 *, int, int,
                                                float, hipStream_t);
template hipError_t launch_rmsnorm<bf16, bf16>(const bf16 *, const bf16 *, f16 *, int, int,
                                               float, hipStream_t);
template hipError_t launch_rope_kv<float>(const float *, float *, const TreeMeta &, float *,
                                          float *, int, int, int, int, int, int, const float2 *,
                                          hipStream_t);
template hipError_t launch_rope_kv<bf16>(const float *, f16 *, const TreeMeta &, bf16 *, bf16 *,
                                         int, int, int, int, int, int, const float2 *,
                                         hipStream_t);

}  // namespace acespec
