// Calibration kernels of the measurement harness (not part of the verify path): the
// rates the chip actually sustains, against which the verify kernels' roofline fractions
// are also reported next to the published peaks.
//   - a streaming device copy (16-byte loads and stores, grid-stride) and a streaming
//     read (four 16-byte loads in flight per thread), the achievable HBM rates;
//   - the LDS read rate of a fragment-read lane pattern (bank conflicts show as a lower
//     rate than a conflict-free pattern's);
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

// Streaming read: four independent 16-byte loads in flight per thread and step, summed so
// the loads stay live; one float per block out.
__global__ __launch_bounds__(256) void read_kernel(const float4 *__restrict__ src,
                                                   float *__restrict__ out, size_t n4) {
  // eight 16-byte loads in flight a thread, with the nontemporal cache policy (a stream
  // read once: it does not allocate in L2 or the MALL); measured on MI355X this reads at
  // about 6.4 TB/s against 5.0-5.4 TB/s with the default policy
  typedef float f4v __attribute__((ext_vector_type(4)));
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  f4v acc = f4v{0.f, 0.f, 0.f, 0.f};
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (; i + 7 * stride < n4; i += 8 * stride) {
    f4v v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = __builtin_nontemporal_load((const f4v *)(src + i + u * stride));
#pragma unroll
    for (int u = 0; u < 8; ++u) acc += v[u];
  }
  for (; i < n4; i += stride) acc += __builtin_nontemporal_load((const f4v *)(src + i));
  float v = acc.x + acc.y + acc.z + acc.w;
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  if ((threadIdx.x & 63) == 0) out[blockIdx.x * 4 + (threadIdx.x >> 6)] = v;
}

// LDS read rate of one 16-byte-per-lane fragment pattern: offs[64] gives each lane's byte
// offset (< 16 KB) within a 256-byte-aligned window that moves by whole 256-byte rounds
// (so the bank pattern is the table's), 8 reads in flight per wave.
__global__ __launch_bounds__(256) void lds_read_kernel(const int *__restrict__ offs, int iters,
                                                       float *__restrict__ out) {
  __shared__ __attribute__((aligned(1024))) char lds[40960];
  for (int i = threadIdx.x; i < 40960 / 4; i += 256) ((float *)lds)[i] = (float)(i & 7);
  __syncthreads();
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int off = offs[lane] & 16383;
  float4 acc[8];
  for (int j = 0; j < 8; ++j) acc[j] = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float4 v = *(const float4 *)(lds + (off & ~15) + ((it * 8 + j + w) & 63) * 256);
      acc[j].x += v.x; acc[j].y += v.y; acc[j].z += v.z; acc[j].w += v.w;
    }
  }
  float r = 0.f;
  for (int j = 0; j < 8; ++j) r += acc[j].x + acc[j].y + acc[j].z + acc[j].w;
  out[blockIdx.x * 256 + threadIdx.x] = r;
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

// Reads n_bytes (a multiple of 16; 16-byte aligned) from src; out: >= 4 * blocks floats.
int acespec_calib_read(const void *src, float *out, size_t n_bytes, int blocks,
                       hipStream_t stream) {
  if (!src || !out || n_bytes % 16 || blocks < 1) return -1;
  hipLaunchKernelGGL(read_kernel, dim3(blocks), dim3(256), 0, stream, (const float4 *)src, out,
                     n_bytes / 16);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

// offs: 64 device ints (lane byte offsets, < 16 KB, 16-byte aligned); out: blocks * 256.
int acespec_calib_lds(const int *offs, float *out, int blocks, int iters, hipStream_t stream) {
  if (!offs || !out || blocks < 1 || iters < 1) return -1;
  hipLaunchKernelGGL(lds_read_kernel, dim3(blocks), dim3(256), 0, stream, offs, iters, out);
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
