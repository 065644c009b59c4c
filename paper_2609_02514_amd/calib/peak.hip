// Calibration kernels of the measurement harness (not part of the verify path): the
// rates the chip actually sustains, against which the verify kernels' roofline fractions
// are also reported next to the published peaks.
//   - a streaming device copy (16-byte loads and stores, grid-stride), the achievable
//     HBM rate;
//   - the MFMA pipe on random fp16 operands: every wave keeps 16 independent
//     v_mfma_f32_16x16x32_f16 accumulators busy, cycling through 4 A and 4 B fragments
//     loaded from a random buffer, so consecutive instructions see different operand bits
//     (the switching, and so the power draw, of real data), with no memory traffic in the
//     loop.
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

namespace {

__global__ __launch_bounds__(256) void copy_kernel(const float4 *__restrict__ src,
                                                   float4 *__restrict__ dst, size_t n4) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride)
    dst[i] = src[i];
}

// operands: random fp16 values, at least (gridDim.x * 4 waves * 64 lanes * 8 fragments *
// 8 halves) elements; out: one float per thread.
__global__ __launch_bounds__(256) void mfma_loop_kernel(const _Float16 *__restrict__ operands,
                                                        float *__restrict__ out, int iters) {
  const int gtid = blockIdx.x * blockDim.x + threadIdx.x;
  const f16x8 *src = (const f16x8 *)operands + (size_t)gtid * 8;
  f16x8 a[4], b[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    a[i] = src[i];
    b[i] = src[4 + i];
  }
  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int j = (i + s) & 3;  // a new (A, B) pair every instruction
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a[i], b[j], acc[i][j], 0, 0, 0);
      }
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

// blocks workgroups of 4 waves, each wave iters x 16 MFMAs of 16x16x32 (16384 flops each).
// operands: >= blocks * 256 * 64 fp16 values; out: >= blocks * 256 floats.
int acespec_calib_mfma(const void *operands, float *out, int blocks, int iters,
                       hipStream_t stream) {
  if (!operands || !out || blocks < 1 || iters < 1) return -1;
  hipLaunchKernelGGL(mfma_loop_kernel, dim3(blocks), dim3(256), 0, stream,
                     (const _Float16 *)operands, out, iters);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

}  // extern "C"
