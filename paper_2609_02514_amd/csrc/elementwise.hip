// Embedding gather, RMSNorm, and RoPE with the tree K/V write into the cache.
//
// RMSNorm: y = x / sqrt(mean(x^2) + eps) * gain, fp32 math, rounded once to the
// activation type.  The residual stream x stays fp32 between layers.
// RoPE (rotate-half): the pair (i, i + hd/2) of every query and key head is rotated by
// pos * base^(-2i/hd); the angle and its sine/cosine are evaluated in double so that
// large positions (16k-token prefixes) keep full fp32 accuracy.  The QKV projection
// arrives in fp32 and is rounded once: q to the activation type, k and v to the cache
// dtype.  Tree row r of session b sits at position prefix_len + depth(r) and its
// key/value go to slot prefix_len + r.
#include "common.h"

namespace {

template <typename T>
__global__ void embed_kernel(const T *__restrict__ embed, const int32_t *__restrict__ tok,
                             float *__restrict__ x, int d) {
  const int row = blockIdx.x;
  const T *src = embed + (size_t)tok[row] * d;
  float *dst = x + (size_t)row * d;
  for (int i = threadIdx.x; i < d; i += blockDim.x) dst[i] = to_f32(src[i]);
}

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

// grid: (rows); block: 256 threads.  Thread t owns rotation frequency i = t % (hd/2) for
// every head it visits, so one sine/cosine pair per thread serves all its heads.
template <typename TW, typename TA>
__global__ __launch_bounds__(256) void rope_kv_kernel(const float *__restrict__ qkv,
                                                      TA *__restrict__ q_out, TreeMeta meta,
                                                      TW *__restrict__ ck, TW *__restrict__ cv,
                                                      int n1, int H, int Hkv, int hd,
                                                      int capacity,
                                                      const double *__restrict__ inv_freq) {
  const int row = blockIdx.x, tid = threadIdx.x;
  const int half = hd >> 1;
  const int i = tid % half;
  const int b = row / n1, r = row - b * n1;
  const double ang = (double)meta.pos[row] * inv_freq[i];
  double sd, cd;
  sincos(ang, &sd, &cd);
  const float c = (float)cd, s = (float)sd;
  const float *base = qkv + (size_t)row * (H + 2 * Hkv) * hd;
  TA *qo = q_out + (size_t)row * H * hd;
  for (int p = tid; p < H * half; p += 256) {
    const int h = p / half;
    const float x1 = base[h * hd + i], x2 = base[h * hd + i + half];
    qo[h * hd + i] = from_f32<TA>(x1 * c - x2 * s);
    qo[h * hd + i + half] = from_f32<TA>(x2 * c + x1 * s);
  }
  const int slot = meta.sess_S[b] + r;
  for (int p = tid; p < Hkv * half; p += 256) {
    const int g = p / half;
    const float *k = base + (H + g) * hd;
    const float x1 = k[i], x2 = k[i + half];
    const size_t kdst = (((size_t)b * Hkv + g) * capacity + slot) * hd;
    ck[kdst + i] = from_f32<TW>(x1 * c - x2 * s);
    ck[kdst + i + half] = from_f32<TW>(x2 * c + x1 * s);
  }
  for (int e = tid; e < Hkv * hd; e += 256) {   // values: head-dim-major cache
    const int g = e / hd, dd = e - g * hd;
    cv[(((size_t)b * Hkv + g) * hd + dd) * capacity + slot] =
        from_f32<TW>(base[(H + Hkv) * hd + e]);
  }
}

__global__ void cast_bf16_f16_kernel(const bf16x8 *__restrict__ in, f16x8 *__restrict__ out,
                                     size_t n8) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n8) out[i] = bf16x8_to_f16x8(in[i]);
}

}  // namespace

namespace acespec {

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
                          int Hkv, int hd, int capacity, const double *inv_freq, hipStream_t s) {
  hipLaunchKernelGGL((rope_kv_kernel<TW, typename ActOf<TW>::type>), dim3(B * n1), dim3(256),
                     0, s, qkv, q_out, meta, cache_k, cache_v, n1, H, Hkv, hd, capacity,
                     inv_freq);
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
                                          float *, int, int, int, int, int, int, const double *,
                                          hipStream_t);
template hipError_t launch_rope_kv<bf16>(const float *, f16 *, const TreeMeta &, bf16 *, bf16 *,
                                         int, int, int, int, int, int, const double *,
                                         hipStream_t);

}  // namespace acespec
