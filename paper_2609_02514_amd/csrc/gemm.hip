// Dense contractions of the verify forward pass: C[M, N] = A[M, K] . W[N, K]^T.
//
// bf16 model: weights are bf16, activations arrive in fp16; both operands are staged
//   into LDS as fp16 (weights converted exactly while staging) and multiplied with
//   gfx950's v_mfma_f32_16x16x32_f16 (same rate as the bf16 form), fp32 accumulation.
//   block tile 128 x 128 x 64, 256 threads = 4 waves in a 2 x 2 grid, each wave owning a
//   64 x 64 sub-tile (4 x 4 MFMA blocks of 16 x 16).  A and W tiles are staged through
//   LDS, double buffered, with an XOR swizzle of the 16-byte chunks inside each 128-byte
//   row so that both the stores and the per-lane 16-byte fragment reads are free of
//   bank conflicts.  The next tile's global loads are in flight while the current tile
//   is multiplied.  Tiles are ordered so that the row tiles of one weight panel land on
//   the same XCD (workgroups are dealt round-robin over the 8 XCDs), which keeps that
//   panel in one L2.
// fp32 path (small models only): LDS-tiled FMA kernel with the same epilogues.
//
// Epilogues fuse the elementwise work that follows each product: fp32 store (QKV, LM head),
// fp32 residual add (attention output and MLP down projections), SwiGLU (gate/up
// projection: each tile holds matching gate and up columns), activation-type store.
#include "common.h"

namespace {

constexpr int BM = 128, BN = 128, BK = 64;

AS_DEVICE int swz(int row, int chunk) { return row * BK + (((chunk ^ (row & 7))) << 3); }

AS_DEVICE float silu_mul(float g, float u) { return g / (1.0f + __expf(-g)) * u; }

// Maps a workgroup id onto a tile id so that consecutive tile ids share an XCD.
AS_DEVICE int xcd_tile(int bid, int total) {
  const int x = bid & 7, local = bid >> 3;
  const int q = total >> 3, rem = total & 7;
  const int before = x * q + (x < rem ? x : rem);
  return before + local;
}

AS_DEVICE f16x8 to_f16x8(f16x8 v) { return v; }
AS_DEVICE f16x8 to_f16x8(bf16x8 v) { return bf16x8_to_f16x8(v); }

template <typename TA> struct Vec8;
template <> struct Vec8<f16> { typedef f16x8 type; };
template <> struct Vec8<bf16> { typedef bf16x8 type; };

template <int EPI, typename TA>
__global__ __launch_bounds__(256, 2) void gemm_mfma_kernel(
    const TA *__restrict__ A, const bf16 *__restrict__ W, int M, int N, int K,
    f16 *__restrict__ out, float *__restrict__ outf, int mt, int nt) {
  typedef typename Vec8<TA>::type va_t;
  __shared__ __attribute__((aligned(16))) f16 sA[2][BM * BK];
  __shared__ __attribute__((aligned(16))) f16 sB[2][BN * BK];

  const int tile = xcd_tile(blockIdx.x, mt * nt);
  const int tn = tile / mt, tm = tile - tn * mt;
  const int m0 = tm * BM;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // Global source rows of the 4 chunks this thread stages per operand.
  const TA *ga[4];
  const bf16 *gb[4];
  int lds_off[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = tid + 256 * i, row = c >> 3, kc = c & 7;
    int am = m0 + row;
    am = am < M ? am : M - 1;
    ga[i] = A + (size_t)am * K + kc * 8;
    int wr;
    if (EPI == acespec::EPI_SWIGLU) {
      const int j0 = tn * 64;  // N is the SwiGLU output width F here
      wr = row < 64 ? j0 + row : N + j0 + (row - 64);
    } else {
      wr = tn * BN + row;
      wr = wr < N ? wr : N - 1;
    }
    gb[i] = W + (size_t)wr * K + kc * 8;
    lds_off[i] = swz(row, kc);
  }

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  va_t ra[4];
  bf16x8 rb[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    ra[i] = *(const va_t *)(ga[i]);
    rb[i] = *(const bf16x8 *)(gb[i]);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    *(f16x8 *)(&sA[0][lds_off[i]]) = to_f16x8(ra[i]);
    *(f16x8 *)(&sB[0][lds_off[i]]) = to_f16x8(rb[i]);
  }
  __syncthreads();

  // Fragment rows for this lane.
  const int lr = lane & 15, lk = lane >> 4;
  int arow[4], brow[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) arow[i] = wm * 64 + i * 16 + lr;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    if (EPI == acespec::EPI_SWIGLU)
      brow[j] = (j < 2 ? wn * 32 + j * 16 : 64 + wn * 32 + (j - 2) * 16) + lr;
    else
      brow[j] = wn * 64 + j * 16 + lr;
  }

  const int KT = K / BK;
  for (int kt = 0; kt < KT; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < KT;
    if (more) {
      const int koff = (kt + 1) * BK;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        ra[i] = *(const va_t *)(ga[i] + koff);
        rb[i] = *(const bf16x8 *)(gb[i] + koff);
      }
    }
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      f16x8 fa[4], fb[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) fa[i] = *(const f16x8 *)(&sA[cur][swz(arow[i], s * 4 + lk)]);
#pragma unroll
      for (int j = 0; j < 4; ++j) fb[j] = *(const f16x8 *)(&sB[cur][swz(brow[j], s * 4 + lk)]);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(fa[i], fb[j], acc[i][j], 0, 0, 0);
    }
    if (more) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        *(f16x8 *)(&sA[cur ^ 1][lds_off[i]]) = to_f16x8(ra[i]);
        *(f16x8 *)(&sB[cur ^ 1][lds_off[i]]) = to_f16x8(rb[i]);
      }
    }
    __syncthreads();
  }

  // Epilogue.  acc[i][j][e] is C[row = .. + lk*4 + e][col = .. + lr].
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int row = m0 + wm * 64 + i * 16 + lk * 4 + e;
      if (row >= M) continue;
      if (EPI == acespec::EPI_SWIGLU) {
#pragma unroll
        for (int jj = 0; jj < 2; ++jj) {
          const int col = tn * 64 + wn * 32 + jj * 16 + lr;
          out[(size_t)row * N + col] = (f16)silu_mul(acc[i][jj][e], acc[i][jj + 2][e]);
        }
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int col = tn * BN + wn * 64 + j * 16 + lr;
          if (col >= N) continue;
          const size_t o = (size_t)row * N + col;
          if (EPI == acespec::EPI_STORE) out[o] = (f16)acc[i][j][e];
          else if (EPI == acespec::EPI_RESID) outf[o] += acc[i][j][e];
          else outf[o] = acc[i][j][e];
        }
      }
    }
  }
}

// ------------------------------------------------------------------------------------
// fp32 reference-precision path (tiny models): 64 x 64 tiles, 4 x 4 outputs per thread.
// ------------------------------------------------------------------------------------
template <int EPI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(const float *__restrict__ A,
                                                       const float *__restrict__ W, int M,
                                                       int N, int K, float *__restrict__ out,
                                                       float *__restrict__ outf) {
  constexpr int T = 64, KS = 16;
  __shared__ float sA[KS][T + 1];
  __shared__ float sW[KS][2 * T + 1];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int m0 = blockIdx.y * T, n0 = blockIdx.x * T;
  const int wcols = EPI == acespec::EPI_SWIGLU ? 2 * T : T;
  float acc[4][8];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = 0.f;
  for (int k0 = 0; k0 < K; k0 += KS) {
    for (int idx = tid; idx < T * KS; idx += 256) {
      const int r = idx / KS, kk = idx % KS;
      const int m = m0 + r;
      sA[kk][r] = (m < M && k0 + kk < K) ? A[(size_t)m * K + k0 + kk] : 0.f;
    }
    for (int idx = tid; idx < wcols * KS; idx += 256) {
      const int r = idx / KS, kk = idx % KS;
      int wr;
      bool ok;
      if (EPI == acespec::EPI_SWIGLU) {
        wr = r < T ? n0 + r : N + n0 + (r - T);
        ok = (n0 + (r % T)) < N;
      } else {
        wr = n0 + r;
        ok = wr < N;
      }
      sW[kk][r] = (ok && k0 + kk < K) ? W[(size_t)wr * K + k0 + kk] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      float a[4], w[8];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = sA[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) w[j] = sW[kk][tx * 4 + j];
      if (EPI == acespec::EPI_SWIGLU) {
#pragma unroll
        for (int j = 0; j < 4; ++j) w[4 + j] = sW[kk][T + tx * 4 + j];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[i][j] = fmaf(a[i], w[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = m0 + ty * 4 + i;
    if (row >= M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = n0 + tx * 4 + j;
      if (col >= N) continue;
      const size_t o = (size_t)row * N + col;
      if (EPI == acespec::EPI_SWIGLU) out[o] = silu_mul(acc[i][j], acc[i][4 + j]);
      else if (EPI == acespec::EPI_STORE) out[o] = acc[i][j];
      else if (EPI == acespec::EPI_RESID) outf[o] += acc[i][j];
      else outf[o] = acc[i][j];
    }
  }
}

}  // namespace

namespace acespec {

template <typename TA>
hipError_t launch_mfma(int epi, const TA *A, const bf16 *W, int M, int N, int K, f16 *out,
                       float *outf, hipStream_t s) {
  const int mt = (M + BM - 1) / BM;
  const int nt = epi == EPI_SWIGLU ? N / 64 : (N + BN - 1) / BN;
  const dim3 grid(mt * nt), block(256);
  switch (epi) {
    case EPI_STORE:
      hipLaunchKernelGGL((gemm_mfma_kernel<EPI_STORE, TA>), grid, block, 0, s, A, W, M, N, K,
                         out, outf, mt, nt);
      break;
    case EPI_RESID:
      hipLaunchKernelGGL((gemm_mfma_kernel<EPI_RESID, TA>), grid, block, 0, s, A, W, M, N, K,
                         out, outf, mt, nt);
      break;
    case EPI_SWIGLU:
      hipLaunchKernelGGL((gemm_mfma_kernel<EPI_SWIGLU, TA>), grid, block, 0, s, A, W, M, N, K,
                         out, outf, mt, nt);
      break;
    default:
      hipLaunchKernelGGL((gemm_mfma_kernel<EPI_F32, TA>), grid, block, 0, s, A, W, M, N, K,
                         out, outf, mt, nt);
  }
  return hipGetLastError();
}

template <>
hipError_t launch_gemm<bf16, f16>(int epi, const f16 *A, const bf16 *W, int M, int N, int K,
                                  f16 *out, float *outf, hipStream_t s) {
  return launch_mfma<f16>(epi, A, W, M, N, K, out, outf, s);
}

template <>
hipError_t launch_gemm<bf16, bf16>(int epi, const bf16 *A, const bf16 *W, int M, int N, int K,
                                   f16 *out, float *outf, hipStream_t s) {
  return launch_mfma<bf16>(epi, A, W, M, N, K, out, outf, s);
}

template <>
hipError_t launch_gemm<float, float>(int epi, const float *A, const float *W, int M, int N,
                                     int K, float *out, float *outf, hipStream_t s) {
  const dim3 grid((N + 63) / 64, (M + 63) / 64), block(256);
  switch (epi) {
    case EPI_STORE:
      hipLaunchKernelGGL(gemm_f32_kernel<EPI_STORE>, grid, block, 0, s, A, W, M, N, K, out,
                         outf);
      break;
    case EPI_RESID:
      hipLaunchKernelGGL(gemm_f32_kernel<EPI_RESID>, grid, block, 0, s, A, W, M, N, K, out,
                         outf);
      break;
    case EPI_SWIGLU:
      hipLaunchKernelGGL(gemm_f32_kernel<EPI_SWIGLU>, grid, block, 0, s, A, W, M, N, K, out,
                         outf);
      break;
    default:
      hipLaunchKernelGGL(gemm_f32_kernel<EPI_F32>, grid, block, 0, s, A, W, M, N, K, out,
                         outf);
  }
  return hipGetLastError();
}

}  // namespace acespec
