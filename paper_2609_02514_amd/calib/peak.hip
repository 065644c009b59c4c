// Calibration kernels of the measurement harness (not part of the verify path): the
// rates the chip actually sustains, against which the verify kernels' roofline fractions
// are also reported next to the published peaks.
//   - a streaming device copy (16-byte loads and stores, grid-stride), the achievable
//     HBM rate;
//   - the MFMA pipe on random fp16 operands: every wave keeps 16 independent
//     v_mfma_f32_16x16x32_f16 accumulators busy, cycling through 4 A and 4 B fragments of
//     pseudo-random values generated in registers, so consecutive instructions see
//     different operand bits (the switching, and so the power draw, of real data), with
//     no memory traffic at all.
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
#define AS_CALIB __device__ __forceinline__

namespace {

__global__ __launch_bounds__(256) void copy_kernel(const float4 *__restrict__ src,
                                                   float4 *__restrict__ dst, size_t n4) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride)
    dst[i] = src[i];
}

// Pseudo-random fp16 operand: random sign and mantissa, magnitude in [0.5, 1).
AS_CALIB uint32_t mix(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7feb352du;
  x ^= x >> 15;
  x *= 0x846ca68bu;
  return x ^ (x >> 16);
}
AS_CALIB f16x8 random_fragment(uint32_t seed) {
  f16x8 v;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const uint16_t bits = (uint16_t)((mix(seed * 8u + e) & 0x83FFu) | 0x3800u);
    v[e] = __builtin_bit_cast(_Float16, bits);
  }
  return v;
}

// Operands are generated in registers (no memory traffic at all); out: one float per
// thread, so the accumulators stay live.
__global__ __launch_bounds__(256) void mfma_loop_kernel(uint32_t seed, float *__restrict__ out,
                                                        int iters) {
  const int gtid = blockIdx.x * blockDim.x + threadIdx.x;
  f16x8 a[4], b[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    a[i] = random_fragment(seed ^ ((uint32_t)gtid * 8u + i));
    b[i] = random_fragment(seed ^ ((uint32_t)gtid * 8u + 4u + i));
  }
  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)  // a new (A, B) pair every instruction
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a[i], b[j], acc[i][j], 0, 0, 0);
  }
  float r = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) r += acc[i][j][0] + acc[i][j][1] + acc[i][j][2] + acc[i][j][3];
  out[gtid] = r;
}

}  // namespace

extern "C" {

// Copies n_bytes (a multiple of 16; both pointers 16-byte aligned) from src to dst.
int acespec_calib_copy(const void *src, void *dst, size_t n_bytes, int blocks,
                       hipStream_t stream) {
  if (!src || !dst || n_bytes % 16 || blocks < 1) return -1;
  hipLaunchKernelGGL(copy_kernel, dim3(blocks), dim3(256), 0, stream, (const float4 *)src,
                     (float4 *)dst, n_bytes / 16);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

// blocks workgroups of 4 waves, each wave iters x 16 MFMAs of 16x16x32 (16384 flops each)
// on operands drawn from seed; out: >= blocks * 256 floats.
int acespec_calib_mfma(uint32_t seed, float *out, int blocks, int iters, hipStream_t stream) {
  if (!out || blocks < 1 || iters < 1) return -1;
  hipLaunchKernelGGL(mfma_loop_kernel, dim3(blocks), dim3(256), 0, stream, seed, out, iters);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

}  // extern "C"
