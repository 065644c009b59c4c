// Dense contractions of the verify forward pass: C[M, N] = A[M, K] . W[N, K]^T.
//
// bf16 model: weights are bf16, activations arrive in fp16; both operands are staged
//   into LDS and the weight fragments are converted to fp16 (exactly) as they are read,
//   then multiplied with gfx950's v_mfma_f32_16x16x32_f16 (same rate as the bf16 form),
//   fp32 accumulation.  See the kernel comment below for the tiling and pipeline; tiles
//   are ordered so that the row tiles of one weight panel land on the same XCD
//   (workgroups are dealt round-robin over the 8 XCDs), which keeps that panel in one
//   L2.  GEMMs whose tile count cannot fill the chip split K; the fp32 partials are
//   summed in a fixed order (deterministic) by a small reduction kernel.
// fp32 model (small models only): LDS-tiled FMA kernel with the same epilogues.
//
// Epilogues fuse the elementwise work that follows each product: fp32 store (QKV, LM
// head), fp32 residual add (attention output and MLP down projections), SwiGLU
// (gate/up projection: each tile holds matching gate and up columns), activation-type
// store.
#include <cmath>

#include "common.h"

namespace {

AS_DEVICE float silu_mul(float g, float u) { return g / (1.0f + __expf(-g)) * u; }

// Maps a workgroup id onto a tile id so that consecutive tile ids share an XCD.
AS_DEVICE int xcd_tile(int bid, int total) {
  const int x = bid & 7, local = bid >> 3;
  const int q = total >> 3, rem = total & 7;
  const int before = x * q + (x < rem ? x : rem);
  return before + local;
}

// ------------------------------------------------------------------------------------
// fp16 x bf16 MFMA kernel, templated on the tiling.
//   WMN x WNN waves; each owns a (WTM*16) x (WTN*16) output sub-tile made of 16 x 16 MFMA
//   blocks, fp32 accumulators in AGPRs.  Block tile TBM x TBN, k-step 32 (64-byte rows).
//   Operands move HBM -> LDS with gfx950's direct loads (global_load_lds_dwordx4: 64
//   lanes x 16 bytes land contiguously at a wave-uniform LDS address) through a ring of
//   NST stages, NST - 2 of them in flight.  The four 16-byte chunks of each 64-byte row
//   are XOR-swizzled by ((row >> 1) & 3) so that the 16-byte fragment reads of 8
//   consecutive rows hit 32 distinct banks; since the DMA fixes where each lane's bytes
//   land, the swizzle is applied to the global source address.
//   One barrier per stage, placed mid-stage: it certifies that the NEXT stage has landed
//   for every wave and that the stage loaded NST - 1 ahead is free, so each wave reads
//   the next stage's first fragments while its last MFMAs of the current stage run.  The
//   loop body is branch-free (past the end of K the last k-tile is loaded again into a
//   free stage; next-stage fragments are always read) so the compiler counts
//   outstanding LDS reads exactly, and fragment reads are fenced against the MFMAs.
// ------------------------------------------------------------------------------------
constexpr int KS = 32;  // k per stage

// 64-byte rows, 16-byte chunks swizzled by (row >> 1) & 3; returns an element offset.
AS_DEVICE int swz32(int row, int chunk) { return row * KS + ((chunk ^ ((row >> 1) & 3)) << 3); }


template <int EPI, int WMN, int WNN, int WTM, int WTN, int NST, int OCC>
__global__ __launch_bounds__(WMN * WNN * 64, OCC) void gemm_f16w_kernel(
    const f16 *__restrict__ A, const bf16 *__restrict__ W, int M, int N, int K,
    f16 *__restrict__ out, float *__restrict__ outf, float *__restrict__ part, int mt, int nt,
    int splits) {
  constexpr int NW = WMN * WNN;
  constexpr int TBM = WMN * WTM * 16, TBN = WNN * WTN * 16;
  constexpr int A_BYTES = TBM * KS * 2, B_BYTES = TBN * KS * 2;
  constexpr int STAGE_BYTES = A_BYTES + B_BYTES;
  constexpr int A_DMA = A_BYTES / 1024 / NW, B_DMA = B_BYTES / 1024 / NW;
  constexpr int L_DMA = A_DMA + B_DMA;
  static_assert(A_DMA * 1024 * NW == A_BYTES && B_DMA * 1024 * NW == B_BYTES, "DMA split");
  static_assert(WTM >= 4 && NST >= 3, "pipeline shape");
  constexpr int HALF = WTN / 2;  // SwiGLU: gate blocks, then the matching up blocks
  __shared__ __attribute__((aligned(16))) char smem[NST * STAGE_BYTES];

  const int units = mt * nt * splits;
  const int unit = xcd_tile(blockIdx.x, units);
  const int tn = unit / (mt * splits);
  const int rem = unit - tn * (mt * splits);
  const int tm = rem / splits, sp = rem - tm * splits;
  const int m0 = tm * TBM;
  const int KT = K / KS;
  const int kt0 = (int)((long long)KT * sp / splits), kt1 = (int)((long long)KT * (sp + 1) / splits);
  const int nk = kt1 - kt0;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wm = w / WNN, wn = w - wm * WNN;
  const int lr = lane & 15, lk = lane >> 4;

  // DMA sources: block j covers tile rows 16j..16j+15; lane l lands at row 16j + l/4,
  // physical chunk l%4, which holds logical chunk (l%4) ^ ((row >> 1) & 3).
  const int drow = lane >> 2, dchunk = (lane & 3) ^ ((lane >> 3) & 3);
  const f16 *ga[A_DMA];
  const bf16 *gb[B_DMA];
#pragma unroll
  for (int t = 0; t < A_DMA; ++t) {
    int r = m0 + (w * A_DMA + t) * 16 + drow;
    r = r < M ? r : M - 1;
    ga[t] = A + (size_t)r * K + dchunk * 8;
  }
#pragma unroll
  for (int t = 0; t < B_DMA; ++t) {
    const int row = (w * B_DMA + t) * 16 + drow;  // W-tile row
    int wr;
    if (EPI == acespec::EPI_SWIGLU) {
      const int j = tn * (TBN / 2) + (row % (TBN / 2));
      const int jc = j < N ? j : N - 1;
      wr = row < TBN / 2 ? jc : N + jc;
    } else {
      wr = tn * TBN + row;
      wr = wr < N ? wr : N - 1;
    }
    gb[t] = W + (size_t)wr * K + dchunk * 8;
  }
  auto issue = [&](int kt, int stage) {
    char *base = smem + stage * STAGE_BYTES;
    const int koff = kt * KS;
#pragma unroll
    for (int t = 0; t < A_DMA; ++t)
      dma16(ga[t] + koff, (lds_ptr_t)(base + (w * A_DMA + t) * 1024));
#pragma unroll
    for (int t = 0; t < B_DMA; ++t)
      dma16(gb[t] + koff, (lds_ptr_t)(base + A_BYTES + (w * B_DMA + t) * 1024));
  };

  int boff[WTN], aoff[WTM];
#pragma unroll
  for (int j = 0; j < WTN; ++j) {
    const int brow = (EPI == acespec::EPI_SWIGLU)
                         ? (j < HALF ? wn * HALF * 16 + j * 16
                                     : TBN / 2 + wn * HALF * 16 + (j - HALF) * 16) + lr
                         : wn * WTN * 16 + j * 16 + lr;
    boff[j] = swz32(brow, lk);
  }
#pragma unroll
  for (int ii = 0; ii < WTM; ++ii) aoff[ii] = swz32(wm * WTM * 16 + ii * 16 + lr, lk);

  f32x4 acc[WTM][WTN];
#pragma unroll
  for (int i = 0; i < WTM; ++i)
#pragma unroll
    for (int j = 0; j < WTN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int p = 0; p < NST - 1; ++p) issue(kt0 + (p < nk ? p : nk - 1), p);
  wait_vmcnt<(NST - 2) * L_DMA>();  // stage 0 landed for this wave
  __builtin_amdgcn_s_barrier();
  f16x8 fb[WTN], fa[WTM];
  bf16x8 rbn[WTN];
  {
    const bf16 *sB = (const bf16 *)(smem + A_BYTES);
    const f16 *sA = (const f16 *)smem;
#pragma unroll
    for (int j = 0; j < WTN; ++j) fb[j] = bf16x8_to_f16x8(*(const bf16x8 *)(&sB[boff[j]]));
    fa[0] = *(const f16x8 *)(&sA[aoff[0]]);
    fa[1] = *(const f16x8 *)(&sA[aoff[1]]);
  }

  for (int i = 0; i < nk; ++i) {
    const int cur = i % NST, nxt = (i + 1) % NST;
    const f16 *sA = (const f16 *)(smem + cur * STAGE_BYTES);
    const f16 *sAn = (const f16 *)(smem + nxt * STAGE_BYTES);
    const bf16 *sBn = (const bf16 *)(smem + nxt * STAGE_BYTES + A_BYTES);
    const int knext = i + NST - 1 < nk ? i + NST - 1 : nk - 1;
#pragma unroll
    for (int ii = 0; ii < WTM; ++ii) {
      if (ii + 2 < WTM) fa[ii + 2] = *(const f16x8 *)(&sA[aoff[ii + 2]]);
      if (ii == WTM / 2) {
        // stage i+1 has landed for this wave (NST-3 newer stages may be outstanding);
        // after the barrier it has landed for every wave and stage i-1 is free
        wait_vmcnt<(NST - 3) * L_DMA>();
        __builtin_amdgcn_s_barrier();
        issue(kt0 + knext, (i + NST - 1) % NST);
#pragma unroll
        for (int j = 0; j < WTN; ++j) rbn[j] = *(const bf16x8 *)(&sBn[boff[j]]);
      }
      SCHED_FENCE();
#pragma unroll
      for (int j = 0; j < WTN; ++j)
        acc[ii][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(fa[ii], fb[j], acc[ii][j], 0, 0, 0);
      SCHED_FENCE();
      if (ii == WTM - 2) fa[0] = *(const f16x8 *)(&sAn[aoff[0]]);
      if (ii == WTM - 1) {
        fa[1] = *(const f16x8 *)(&sAn[aoff[1]]);
#pragma unroll
        for (int j = 0; j < WTN; ++j) fb[j] = bf16x8_to_f16x8(rbn[j]);
      }
    }
  }
  // No LDS DMA may still be writing when the workgroup's LDS is released.
  wait_vmcnt<0>();

  // Epilogue.  acc[i][j][e] is C[row = m0 + wm*WTM*16 + i*16 + lk*4 + e][col = .. + lr].
  const size_t MN = (size_t)M * N;
#pragma unroll
  for (int ii = 0; ii < WTM; ++ii) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int row = m0 + wm * WTM * 16 + ii * 16 + lk * 4 + e;
      if (row >= M) continue;
      if (EPI == acespec::EPI_SWIGLU) {
#pragma unroll
        for (int jj = 0; jj < HALF; ++jj) {
          const int col = tn * (TBN / 2) + wn * HALF * 16 + jj * 16 + lr;
          if (col < N)
            out[(size_t)row * N + col] = (f16)silu_mul(acc[ii][jj][e], acc[ii][jj + HALF][e]);
        }
      } else {
#pragma unroll
        for (int j = 0; j < WTN; ++j) {
          const int col = tn * TBN + wn * WTN * 16 + j * 16 + lr;
          if (col >= N) continue;
          const size_t o = (size_t)row * N + col;
          if (splits > 1) part[sp * MN + o] = acc[ii][j][e];
          else if (EPI == acespec::EPI_STORE) out[o] = (f16)acc[ii][j][e];
          else if (EPI == acespec::EPI_RESID) outf[o] += acc[ii][j][e];
          else outf[o] = acc[ii][j][e];
        }
      }
    }
  }
}

// Split-K reduction in a fixed order (deterministic): dst (+)= sum_s part[s].
template <bool RESID>
__global__ void splitk_reduce_kernel(const float4 *__restrict__ part, float4 *__restrict__ dst,
                                     size_t n4, int splits) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n4) return;
  float4 acc = RESID ? dst[i] : make_float4(0.f, 0.f, 0.f, 0.f);
  for (int s = 0; s < splits; ++s) {
    const float4 v = part[s * n4 + i];
    acc.x += v.x;
    acc.y += v.y;
    acc.z += v.z;
    acc.w += v.w;
  }
  dst[i] = acc;
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

using acespec::EPI_STORE;
using acespec::EPI_RESID;
using acespec::EPI_SWIGLU;
using acespec::EPI_F32;

// Tilings: {waves M, waves N, wave tile M / 16, wave tile N / 16, stages, WGs per CU}.
// Measured on MI355X against the verify-step shapes (other tilings tried: 32 x 32 MFMA
// blocks with one wave per SIMD, 64-wide k stages, weights loaded straight to VGPRs,
// deeper rings at one workgroup per CU; none was faster than these two).
struct GemmVariant {
  int wmn, wnn, wtm, wtn, nst, occ;
};
constexpr GemmVariant kVariants[] = {
    {1, 4, 8, 4, 3, 2},  // 0: 128 x 256, wave 128 x 64, 72 KB LDS, 2 workgroups per CU
    {2, 2, 4, 4, 4, 2},  // 1: 128 x 128, wave 64 x 64, 64 KB LDS, 2 workgroups per CU
};
constexpr int kNumVariants = sizeof(kVariants) / sizeof(kVariants[0]);

// Chooses the number of K splits: enough units to fill the chip, weighed against the
// cost of re-reading fp32 partials.  Only residual / fp32 epilogues split.
int choose_splits(int epi, int M, int N, int K, int tiles, int cus, int occ) {
  if (epi == EPI_SWIGLU || epi == EPI_STORE || (N % 4) != 0) return 1;
  const int KT = K / 64;
  const double part_cost = (double)M * N * 4 / 10e12 / 0.43e-6;  // per split, in 64-k units
  int best = 1;
  double best_t = 1e30;
  for (int s = 1; s <= 8; ++s) {
    if (KT / s < 4) break;
    const double rounds = std::ceil((double)tiles * s / ((double)cus * occ));
    const double t = rounds * std::ceil((double)KT / s) + (s > 1 ? part_cost * s : 0.0);
    if (t < best_t * 0.97) { best_t = t; best = s; }
  }
  return best;
}

template <int EPI, int V>
void launch_variant(dim3 grid, hipStream_t s, const f16 *A, const bf16 *W, int M, int N, int K,
                    f16 *out, float *outf, float *part, int mt, int nt, int splits) {
  constexpr GemmVariant v = kVariants[V];
  hipLaunchKernelGGL((gemm_f16w_kernel<EPI, v.wmn, v.wnn, v.wtm, v.wtn, v.nst, v.occ>), grid,
                     dim3(v.wmn * v.wnn * 64), 0, s, A, W, M, N, K, out, outf, part, mt, nt,
                     splits);
}

template <int EPI>
void launch_epi(int var, dim3 grid, hipStream_t s, const f16 *A, const bf16 *W, int M, int N,
                int K, f16 *out, float *outf, float *part, int mt, int nt, int splits) {
  switch (var) {
#define CASE(V) case V: launch_variant<EPI, V>(grid, s, A, W, M, N, K, out, outf, part, mt, nt, splits); break;
    CASE(0) CASE(1)
#undef CASE
    default: break;
  }
}

// Default tiling per shape (measured on MI355X): 128 x 128 tiles for few rows (more
// tiles to spread over 256 CUs) and for QKV-sized fp32 outputs, 128 x 256 otherwise.
int pick_variant(int epi, int M, int N, int K) {
  (void)K;
  if (M <= 384) return 1;
  if (epi == EPI_F32 && N <= 8192) return 1;
  return 0;
}

}  // namespace

namespace acespec {

hipError_t launch_f16w_variant(int var, int splits_override, int epi, const f16 *A,
                               const bf16 *W, int M, int N, int K, f16 *out, float *outf,
                               float *part, long long part_cap, int cus, hipStream_t s) {
  if (var < 0) var = pick_variant(epi, M, N, K);
  if (var >= kNumVariants) return hipErrorInvalidValue;
  const GemmVariant v = kVariants[var];
  const int tbm = v.wmn * v.wtm * 16, tbn = v.wnn * v.wtn * 16;
  const int mt = (M + tbm - 1) / tbm;
  const int nt = epi == EPI_SWIGLU ? (N + tbn / 2 - 1) / (tbn / 2) : (N + tbn - 1) / tbn;
  int splits = splits_override > 0 ? splits_override
                                   : choose_splits(epi, M, N, K, mt * nt, cus, v.occ);
  if (epi == EPI_SWIGLU || epi == EPI_STORE || (N % 4) != 0) splits = 1;
  while (splits > 1 && (long long)splits * M * N > part_cap) --splits;
  const dim3 grid(mt * nt * splits);
  switch (epi) {
    case EPI_STORE: launch_epi<EPI_STORE>(var, grid, s, A, W, M, N, K, out, outf, part, mt, nt, splits); break;
    case EPI_RESID: launch_epi<EPI_RESID>(var, grid, s, A, W, M, N, K, out, outf, part, mt, nt, splits); break;
    case EPI_SWIGLU: launch_epi<EPI_SWIGLU>(var, grid, s, A, W, M, N, K, out, outf, part, mt, nt, splits); break;
    default: launch_epi<EPI_F32>(var, grid, s, A, W, M, N, K, out, outf, part, mt, nt, splits);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || splits == 1) return e;
  const size_t n4 = (size_t)M * N / 4;
  if (epi == EPI_RESID)
    hipLaunchKernelGGL(splitk_reduce_kernel<true>, dim3((n4 + 255) / 256), dim3(256), 0, s,
                       (const float4 *)part, (float4 *)outf, n4, splits);
  else
    hipLaunchKernelGGL(splitk_reduce_kernel<false>, dim3((n4 + 255) / 256), dim3(256), 0, s,
                       (const float4 *)part, (float4 *)outf, n4, splits);
  return hipGetLastError();
}

template <>
hipError_t launch_gemm<bf16, f16>(int epi, const f16 *A, const bf16 *W, int M, int N, int K,
                                  f16 *out, float *outf, const GemmAux &aux, hipStream_t s) {
  return launch_f16w_variant(-1, 0, epi, A, W, M, N, K, out, outf, aux.part, aux.part_cap,
                             aux.cus, s);
}

template <>
hipError_t launch_gemm<float, float>(int epi, const float *A, const float *W, int M, int N,
                                     int K, float *out, float *outf, const GemmAux &,
                                     hipStream_t s) {
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
