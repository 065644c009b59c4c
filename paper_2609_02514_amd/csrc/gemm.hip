// Dense contractions of the verify forward pass: C[M, N] = A[M, K] . W[N, K]^T.
//
// bf16 model: weights are bf16, activations arrive in fp16; both operands are staged
//   into LDS and the weight fragments are converted to fp16 (exactly) as they are read,
//   then multiplied with gfx950's v_mfma_f32_16x16x32_f16 (same rate as the bf16 form),
//   fp32 accumulation.  See the kernel comment below for the tiling and pipeline; tiles
//   are ordered so that the row tiles of one weight panel land on the same XCD
//   (workgroups are dealt round-robin over the 8 XCDs), which keeps that panel in one
//   L2.  Tiles of a last, partly empty round of workgroups (or every tile, when there
//   are fewer tiles than workgroup slots) are sliced along K; the fp32 slices are summed
//   in a fixed order (deterministic) by a fixup kernel that also applies the epilogue.
// fp32 model (small models only): LDS-tiled FMA kernel with the same epilogues.
//
// Epilogues fuse the elementwise work that follows each product: fp32 store (LM head,
// with per-tile row maxima for the vocabulary kernel), RoPE + q store + cache write of
// the tree K/V (QKV projection), fp32 residual add followed by the next block's RMSNorm
// (attention output and MLP down projections), SwiGLU (gate/up projection: each tile
// holds matching gate and up columns), activation-type store.
#include <cmath>

#include "common.h"

namespace {

AS_DEVICE float silu_mul(float g, float u) { return g / (1.0f + __expf(-g)) * u; }

// Weight fragments: fp16 weights are used as loaded, bf16 weights are widened to fp16.
template <typename TB> struct Vec8;
template <> struct Vec8<f16> { typedef f16x8 type; };
template <> struct Vec8<bf16> { typedef bf16x8 type; };
AS_DEVICE f16x8 to_f16(f16x8 v) { return v; }
AS_DEVICE f16x8 to_f16(bf16x8 v) { return bf16x8_to_f16x8(v); }

// Maps a workgroup id onto a tile id so that consecutive tile ids share an XCD.
AS_DEVICE int xcd_tile(int bid, int total) {
  const int x = bid & 7, local = bid >> 3;
  const int q = total >> 3, rem = total & 7;
  const int before = x * q + (x < rem ? x : rem);
  return before + local;
}

// ------------------------------------------------------------------------------------
// fp16-activation MFMA kernel, templated on the tiling.
//   WMN x WNN waves; each owns a (WTM*16) x (WTN*16) output sub-tile made of 16 x 16 MFMA
//   blocks (v_mfma_f32_16x16x32_f16), fp32 accumulators.  Block tile TBM x TBN, KSS
//   k-values per stage (rows of 2*KSS bytes).  Operands move HBM -> LDS by direct
//   buffer loads (buffer_load_dwordx4 ... lds: 64 lanes x 16 bytes land contiguously at a
//   wave-uniform LDS address; the k offset of a stage is a scalar) through a ring of NST
//   stages, NST - 2 of them in flight.  Full 128-byte rows (KSS = 64) move twice the bytes
//   per cycle of 64-byte rows through the L2 -> LDS path.  The 16-byte pieces of every row
//   are XOR-swizzled so that the 16 rows read by one 16-lane group of a fragment load
//   hit 16 distinct bank groups; since the DMA fixes where each lane's bytes land, the
//   swizzle is applied to the global source addresses.
//   One barrier per stage, placed mid-stage: it certifies that the NEXT stage has landed
//   for every wave and that the stage loaded NST - 1 ahead is free, so each wave reads
//   the next stage's first fragments while its last MFMAs of the current stage run.  The
//   loop body is branch-free (past the end of K the last k-tile is loaded again into a
//   free stage; next-stage fragments are always read) so the compiler counts
//   outstanding LDS reads exactly, and fragment reads are fenced against the MFMAs.
// ------------------------------------------------------------------------------------
// Byte offset of 16-byte piece `pc` of row `row` in rows of ROWB bytes.  The piece index
// is XORed with (row / 2): measured on gfx950, a 16-lane fragment read (16 rows, one
// logical piece each) then runs at the LDS's full rate for 64- and 128-byte rows alike,
// where XORing with the row's 256-byte bank round (row / 4 for 64-byte rows) halves it.
template <int ROWB> AS_DEVICE int piece_off(int row, int pc) {
  const int sw = (row >> 1) & (ROWB / 16 - 1);
  return row * ROWB + ((pc ^ sw) << 4);
}

// Epilogue LDS needs beyond the operand ring: the QKV RoPE epilogue stages 64-row parts
// of the fp32 tile (plus a row table), the row-maximum epilogue one float per (wave
// column, tile row).
constexpr int epi_smem(int epi, int tbm, int tbn, int wnn) {
  return epi == acespec::EPI_QKV_ROPE ? 64 * (tbn + 4) * 4 + 64 * 8
         : epi == acespec::EPI_F32_MAX ? wnn * tbm * 4
                                        : 0;
}

// PK = 0: W is row-major [N, K] and staged through LDS with the activations.
// PK = 1: W is pre-packed fp16 in MFMA fragment order (pack_frag_kernel): each wave loads
//   its own weight fragments straight into registers, NST - 1 k-steps ahead, and only the
//   activations go through LDS.  A packed fragment is 1 KB of contiguous memory, so these
//   loads are as cheap for the address unit as the row-contiguous DMA, while LDS carries a
//   third of the bytes (no weight rows written, no weight fragments read) and no widening
//   instructions run.  KSS = 32.
// PK = 2: as PK = 1 with twice the waves, the tile's k-steps split between two wave
//   groups (even and odd 32-wide steps of each 64-wide stage, 128-byte activation rows),
//   whose accumulators are summed through LDS before the epilogue: two waves a SIMD for
//   a product with fewer tiles than CUs, without fp32 partials in memory (QKV + RoPE
//   epilogue only).  KSS = 64.
template <int EPI, typename TB, int WMN, int WNN, int WTM, int WTN, int NST, int OCC, int KSS,
          int PK>
__global__ __launch_bounds__(WMN * WNN * (PK == 2 ? 2 : 1) * 64, OCC) void gemm_f16w_kernel(
    const f16 *__restrict__ A, const void *__restrict__ W, int M, int N, int K,
    f16 *__restrict__ out, float *__restrict__ outf, float *__restrict__ part, int mt, int nt,
    int full, int tsplit, acespec::RopeOut<TB> ro, float *__restrict__ tmax) {
  constexpr int KG = PK == 2 ? 2 : 1;  // wave groups splitting each stage's k-steps
  constexpr int NW = WMN * WNN * KG;
  constexpr int TBM = WMN * WTM * 16, TBN = WNN * WTN * 16;
  constexpr int ROWB = KSS * 2, PIECES = KSS / 8, ROWS_PER_BLK = 1024 / ROWB;
  constexpr int A_BYTES = TBM * ROWB, B_BYTES = PK ? 0 : TBN * ROWB;
  constexpr int STAGE_BYTES = A_BYTES + B_BYTES;
  // 1 KB DMA blocks of the A tile per wave (rounded up: a wave past the last block loads
  // the last block again, the same bytes to the same place, so every wave issues the same
  // number of loads and the vmcnt arithmetic below holds for all of them)
  constexpr int A_BLKS = A_BYTES / 1024, A_DMA = (A_BLKS + NW - 1) / NW;
  constexpr int B_DMA = B_BYTES / 1024 / NW;
  constexpr int L_DMA = A_DMA + B_DMA;
  constexpr int KSUB = KSS / 32;            // 32-wide MFMA k steps per stage
  constexpr int F = KSUB * WTM;             // A fragments per stage, in use order
  static_assert(A_BLKS * 1024 == A_BYTES && B_DMA * 1024 * NW == B_BYTES, "DMA split");
  static_assert(F >= 4 && NST >= 3, "pipeline shape");
  static_assert(!PK || KSS == 32 * KG, "packed weights come in 32-wide k steps, one a group");
  static_assert(KG == 1 || EPI == acespec::EPI_QKV_ROPE, "split wave groups: QKV epilogue only");
  constexpr int HALF = WTN / 2;  // SwiGLU: gate blocks, then the matching up blocks
  constexpr int RING = NST * STAGE_BYTES, EPI_SM = epi_smem(EPI, TBM, TBN, WNN);
  constexpr int RED = KG > 1 ? WMN * WNN * WTM * WTN * 4 * 64 * 4 : 0;  // group-sum buffer
  constexpr int SM1 = RING > EPI_SM ? RING : EPI_SM;
  __shared__ __attribute__((aligned(1024))) char smem[SM1 > RED ? SM1 : RED];
  typedef typename Vec8<TB>::type tbx8;

  // Units: `full` whole tiles, then tsplit k-slices of each remaining tile (their partial
  // sums go to `part`, summed by tile_fixup_kernel).  Each group is dealt over the XCDs on
  // its own (full is a multiple of 8), so the slices spread over the whole chip.  Slices
  // are numbered k-slice first: an XCD's run of units then covers one k-slice (two at a
  // boundary) of a band of weight panels, so it fetches its k-columns of the activations
  // once for all its panels, instead of the whole activation matrix once per XCD.
  const int tiles = mt * nt;
  int tile, sp, ns;
  if ((int)blockIdx.x < full) {
    tile = xcd_tile(blockIdx.x, full);
    sp = 0;
    ns = 1;
  } else {
    const int ntl = tiles - full;
    const int u = xcd_tile(blockIdx.x - full, ntl * tsplit);
    sp = u / ntl;
    tile = full + (u - sp * ntl);
    ns = tsplit;
  }
  const int tn = tile / mt, tm = tile - tn * mt;
  const int m0 = tm * TBM;
  const int KT = K / KSS;
  const int kt0 = (int)((long long)KT * sp / ns), kt1 = (int)((long long)KT * (sp + 1) / ns);
  const int nk = kt1 - kt0;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int kg = w / (WMN * WNN), wl = w - kg * (WMN * WNN);  // k group, wave in the group
  const int wm = wl / WNN, wn = wl - wm * WNN;
  const int lr = lane & 15, lk = lane >> 4;

  // DMA sources: block j of an operand covers tile rows ROWS_PER_BLK*j ..; lane l lands at
  // row ROWS_PER_BLK*j + l / PIECES, physical piece l % PIECES.  Rows of A past M get an
  // offset past the end of A's buffer range, which the buffer load's range check turns
  // into zeros (no fetch, and zero MFMA operands draw less power); rows of W past N are
  // clamped to the last row.  Neither product is ever stored.
  const __amdgpu_buffer_rsrc_t rsa = make_rsrc(A, (uint32_t)((size_t)M * K * 2));
  const int wrows = EPI == acespec::EPI_SWIGLU ? 2 * N : N;
  const __amdgpu_buffer_rsrc_t rsb = make_rsrc(W, (uint32_t)((size_t)wrows * K * 2));
  const int drow = lane / PIECES, dpc = lane % PIECES;
  uint32_t va[A_DMA], vb[B_DMA > 0 ? B_DMA : 1];
#pragma unroll
  for (int t = 0; t < A_DMA; ++t) {
    const int blk = w * A_DMA + t < A_BLKS ? w * A_DMA + t : A_BLKS - 1;
    const int lrow = blk * ROWS_PER_BLK + drow;
    const int r = m0 + lrow;
    va[t] = r < M ? (uint32_t)r * K * 2 + (piece_off<ROWB>(lrow, dpc) - lrow * ROWB)
                  : (uint32_t)M * K * 2;
  }
#pragma unroll
  for (int t = 0; t < B_DMA; ++t) {
    const int row = (w * B_DMA + t) * ROWS_PER_BLK + drow;  // W-tile row
    int wr;
    if (EPI == acespec::EPI_SWIGLU) {
      const int j = tn * (TBN / 2) + (row % (TBN / 2));
      const int jc = j < N ? j : N - 1;
      wr = row < TBN / 2 ? jc : N + jc;
    } else {
      wr = tn * TBN + row;
      wr = wr < N ? wr : N - 1;
    }
    vb[t] = (uint32_t)wr * K * 2 + (piece_off<ROWB>(row, dpc) - row * ROWB);
  }
  // Packed weights: fragment (16-row block nb, k step kt) at ((nb * KT + kt) * 64 + lane)
  // 16-byte units; the wave's WTN column blocks, SwiGLU-paired like the LDS path's rows.
  const f16x8 *pkw[PK ? WTN : 1];
  if constexpr (PK) {
#pragma unroll
    for (int j = 0; j < WTN; ++j) {
      int c, base;
      if (EPI == acespec::EPI_SWIGLU) {
        c = tn * (TBN / 2) + wn * HALF * 16 + (j < HALF ? j : j - HALF) * 16;
        c = c < N ? c : N - 16;
        base = j < HALF ? c : N + c;
      } else {
        c = tn * TBN + wn * WTN * 16 + j * 16;
        base = c < N ? c : N - 16;
      }
      pkw[j] = (const f16x8 *)W + (size_t)(base >> 4) * (K / 32) * 64 + lane;
    }
  }
  auto issue = [&](int kt, int stage) {
    char *base = smem + stage * STAGE_BYTES;
    const int soff = kt * ROWB;
#pragma unroll
    for (int t = 0; t < A_DMA; ++t) {
      const int blk = w * A_DMA + t < A_BLKS ? w * A_DMA + t : A_BLKS - 1;
      buf_dma16(rsa, (lds_ptr_t)(base + blk * 1024), va[t], soff);
    }
#pragma unroll
    for (int t = 0; t < B_DMA; ++t)
      buf_dma16(rsb, (lds_ptr_t)(base + A_BYTES + (w * B_DMA + t) * 1024), vb[t], soff);
  };

  // Fragment byte offsets within a stage: A fragment f = (k step f / WTM, row block
  // f % WTM); B fragment (k step s2, column block j).
  int aoff[F], boff[KSUB][WTN];
#pragma unroll
  for (int f = 0; f < F; ++f)
    aoff[f] = piece_off<ROWB>(wm * WTM * 16 + (f % WTM) * 16 + lr, (f / WTM) * 4 + lk);
#pragma unroll
  for (int j = 0; j < WTN; ++j) {
    const int brow = (EPI == acespec::EPI_SWIGLU)
                         ? (j < HALF ? wn * HALF * 16 + j * 16
                                     : TBN / 2 + wn * HALF * 16 + (j - HALF) * 16) + lr
                         : wn * WTN * 16 + j * 16 + lr;
#pragma unroll
    for (int s2 = 0; s2 < KSUB; ++s2) boff[s2][j] = A_BYTES + piece_off<ROWB>(brow, s2 * 4 + lk);
  }

  f32x4 acc[WTM][WTN];
#pragma unroll
  for (int i = 0; i < WTM; ++i)
#pragma unroll
    for (int j = 0; j < WTN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  if constexpr (PK) {
    // Step i: A k-tile i sits in ring slot i % NST, its weight fragments in register set
    // i % NST (the loop is unrolled NST times so the set index is static).  At the top of
    // a step this wave's loads of step i have landed (NST - 2 newer steps may be out);
    // after the barrier every wave's have, and every wave is done with slot i - 1, which
    // the loads of step i + NST - 1 then refill.
    constexpr int L_VM = A_DMA + WTN;
    constexpr int FW = WTM;  // A fragments of this wave's k-step
    f16x8 rb[NST][WTN], fa[FW];
    int aok[FW];  // this group's 16-byte pieces of the stage's rows
#pragma unroll
    for (int f = 0; f < FW; ++f)
      aok[f] = piece_off<ROWB>(wm * WTM * 16 + f * 16 + lr, kg * 4 + lk);
#pragma unroll
    for (int p = 0; p < NST - 1; ++p) {
      const int kt = kt0 + (p < nk ? p : nk - 1);
      issue(kt, p);
#pragma unroll
      for (int j = 0; j < WTN; ++j) rb[p][j] = pkw[j][(size_t)(kt * KG + kg) * 64];
    }
    // One k-step (i = the step, u = i % NST, a constant once the callers are unrolled).
    auto step = [&](int i, int u) {
      wait_vmcnt<(NST - 2) * L_VM>();
      __builtin_amdgcn_s_barrier();
      const int kn = kt0 + (i + NST - 1 < nk ? i + NST - 1 : nk - 1);
      const char *sc = smem + u * STAGE_BYTES;
      fa[0] = *(const f16x8 *)(sc + aok[0]);
      fa[1] = *(const f16x8 *)(sc + aok[1]);
      fa[2] = *(const f16x8 *)(sc + aok[2]);
#pragma unroll
      for (int f = 0; f < FW; ++f) {
        if (f + 3 < FW) fa[f + 3] = *(const f16x8 *)(sc + aok[f + 3]);
        SCHED_FENCE();
#pragma unroll
        for (int j = 0; j < WTN; ++j)
          acc[f][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(fa[f], rb[u][j], acc[f][j], 0, 0, 0);
        SCHED_FENCE();
        if (f == 0) {
          issue(kn, (u + NST - 1) % NST);
#pragma unroll
          for (int j = 0; j < WTN; ++j)
            rb[(u + NST - 1) % NST][j] = pkw[j][(size_t)(kn * KG + kg) * 64];
        }
      }
    };
    // Whole rounds of NST steps run as straight-line code: with a conditional exit between
    // the steps the compiler moves each step's weight loads down to the step that reads
    // them, so their latency is no longer covered by the NST - 1 steps in between.
    int i0 = 0;
    wait_lgkmcnt0();
    for (; i0 + NST <= nk; i0 += NST) {
#pragma unroll
      for (int u = 0; u < NST; ++u) step(i0 + u, u);
    }
#pragma unroll
    for (int u = 0; u < NST - 1; ++u)
      if (i0 + u < nk) step(i0 + u, u);
  } else {
  for (int p = 0; p < NST - 1; ++p) issue(kt0 + (p < nk ? p : nk - 1), p);
  wait_vmcnt<(NST - 2) * L_DMA>();  // stage 0 landed for this wave
  __builtin_amdgcn_s_barrier();
  f16x8 fb[KSUB][WTN], fa[F];
  tbx8 rbn[KSUB][WTN];
#pragma unroll
  for (int s2 = 0; s2 < KSUB; ++s2)
#pragma unroll
    for (int j = 0; j < WTN; ++j) fb[s2][j] = to_f16(*(const tbx8 *)(smem + boff[s2][j]));
  fa[0] = *(const f16x8 *)(smem + aoff[0]);
  fa[1] = *(const f16x8 *)(smem + aoff[1]);

  for (int i = 0; i < nk; ++i) {
    const int cur = i % NST, nxt = (i + 1) % NST;
    const char *sc = smem + cur * STAGE_BYTES;
    const char *sn = smem + nxt * STAGE_BYTES;
    const int knext = i + NST - 1 < nk ? i + NST - 1 : nk - 1;
#pragma unroll
    for (int f = 0; f < F; ++f) {
      if (f + 2 < F) fa[f + 2] = *(const f16x8 *)(sc + aoff[f + 2]);
      if (f == F / 2) {
        // stage i+1 has landed for this wave (NST-3 newer stages may be outstanding);
        // after the barrier it has landed for every wave and stage i-1 is free
        wait_vmcnt<(NST - 3) * L_DMA>();
        __builtin_amdgcn_s_barrier();
        issue(kt0 + knext, (i + NST - 1) % NST);
#pragma unroll
        for (int s2 = 0; s2 < KSUB; ++s2)
#pragma unroll
          for (int j = 0; j < WTN; ++j) rbn[s2][j] = *(const tbx8 *)(sn + boff[s2][j]);
      }
      SCHED_FENCE();
#pragma unroll
      for (int j = 0; j < WTN; ++j)
        acc[f % WTM][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(fa[f], fb[f / WTM][j],
                                                                 acc[f % WTM][j], 0, 0, 0);
      SCHED_FENCE();
      if (f == F - 2) fa[0] = *(const f16x8 *)(sn + aoff[0]);
      if (f == F - 1) {
        fa[1] = *(const f16x8 *)(sn + aoff[1]);
#pragma unroll
        for (int s2 = 0; s2 < KSUB; ++s2)
#pragma unroll
          for (int j = 0; j < WTN; ++j) fb[s2][j] = to_f16(rbn[s2][j]);
      }
    }
  }
  }
  // No LDS DMA may still be writing when the workgroup's LDS is released.
  wait_vmcnt<0>();
  if constexpr (KG > 1) {
    // the wave groups' sums of their k-steps: group 1 hands its blocks to group 0
    __syncthreads();  // every wave is past the ring
    float *red = (float *)smem;
    if (kg == 1) {
#pragma unroll
      for (int ii = 0; ii < WTM; ++ii)
#pragma unroll
        for (int j = 0; j < WTN; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            red[(((wl * WTM + ii) * WTN + j) * 4 + e) * 64 + lane] = acc[ii][j][e];
    }
    __syncthreads();
    if (kg == 0) {
#pragma unroll
      for (int ii = 0; ii < WTM; ++ii)
#pragma unroll
        for (int j = 0; j < WTN; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            acc[ii][j][e] += red[(((wl * WTM + ii) * WTN + j) * 4 + e) * 64 + lane];
    }
  }

  if constexpr (EPI == acespec::EPI_QKV_ROPE) {
    // QKV projection (never sliced along K here): the fp32 tile goes through LDS in
    // 64-row parts so that each head's rotation pairs (i, i + hd/2) and each value
    // column's run of consecutive tree slots can be read across waves.
    constexpr int CR = 64, SP = TBN + 4;  // rows per part, row pitch in floats
    static_assert(CR * SP * 4 + CR * 8 <= sizeof(smem),
                  "a part of the tile and its row table fit the workgroup's LDS");
    float *st = (float *)smem;
    int *rsess = (int *)(st + CR * SP);  // per row of the part: its session,
    int *rslot = rsess + CR;             // and the cache slot of its tree row
    const int hd = ro.hd, half = hd >> 1, nheads = ro.H + 2 * ro.Hkv;
    const int lq4 = hd == 128 ? 4 : 3;  // log2 of the 4-frequency items per row (hd 64 or 128)
    for (int c0 = 0; c0 < TBM; c0 += CR) {
      const int nr = TBM - c0 < CR ? TBM - c0 : CR;  // rows of this part (tiles of 112 rows)
      __syncthreads();  // every wave is past the ring / the previous part
      if (tid < CR) {
        const int row = m0 + c0 + tid;
        if (row < M) {
          const int b = row / ro.n1;
          rsess[tid] = b;
          rslot[tid] = ro.sess_S[b] + row - b * ro.n1;
        }
      }
#pragma unroll
      for (int ii = 0; ii < WTM; ++ii)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int lrow = wm * WTM * 16 + ii * 16 + lk * 4 + e - c0;
          if (lrow < 0 || lrow >= CR || kg != 0) continue;  // group 0 holds the sums
#pragma unroll
          for (int j = 0; j < WTN; ++j) st[lrow * SP + wn * WTN * 16 + j * 16 + lr] = acc[ii][j][e];
        }
      __syncthreads();
      for (int hb = 0; hb < TBN / hd; ++hb) {
        const int gh = tn * (TBN / hd) + hb;  // head of the projection: q, k, then v heads
        if (gh >= nheads) break;
        const float *sb = st + hb * hd;
        if (gh < ro.H + ro.Hkv) {  // query or key head: rotate-half, 4 frequencies a thread
          for (int it = tid; it < (nr << lq4); it += NW * 64) {
            const int r = it >> lq4, i = (it & ((1 << lq4) - 1)) * 4, row = m0 + c0 + r;
            if (row >= M) continue;
            const float4 a1 = *(const float4 *)(sb + r * SP + i);
            const float4 a2 = *(const float4 *)(sb + r * SP + i + half);
            const float4 c01 = *(const float4 *)(ro.rot + (size_t)row * half + i);
            const float4 c23 = *(const float4 *)(ro.rot + (size_t)row * half + i + 2);
            const float x1[4] = {a1.x, a1.y, a1.z, a1.w}, x2[4] = {a2.x, a2.y, a2.z, a2.w};
            const float cc[4] = {c01.x, c01.z, c23.x, c23.z}, sn[4] = {c01.y, c01.w, c23.y, c23.w};
            float y1[4], y2[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              y1[e] = x1[e] * cc[e] - x2[e] * sn[e];
              y2[e] = x2[e] * cc[e] + x1[e] * sn[e];
            }
            if (gh < ro.H) {
              typedef _Float16 h4 __attribute__((ext_vector_type(4)));
              f16 *qo = ro.q + (size_t)row * ro.H * hd + (size_t)gh * hd;
              *(h4 *)(qo + i) = h4{(f16)y1[0], (f16)y1[1], (f16)y1[2], (f16)y1[3]};
              *(h4 *)(qo + i + half) = h4{(f16)y2[0], (f16)y2[1], (f16)y2[2], (f16)y2[3]};
            } else {
              typedef TB t4 __attribute__((ext_vector_type(4)));
              TB *kd = ro.ck + (((size_t)rsess[r] * ro.Hkv + (gh - ro.H)) * ro.capacity +
                                rslot[r]) * hd;
              *(t4 *)(kd + i) = t4{from_f32<TB>(y1[0]), from_f32<TB>(y1[1]),
                                   from_f32<TB>(y1[2]), from_f32<TB>(y1[3])};
              *(t4 *)(kd + i + half) = t4{from_f32<TB>(y2[0]), from_f32<TB>(y2[1]),
                                          from_f32<TB>(y2[2]), from_f32<TB>(y2[3])};
            }
          }
        } else {  // value head: head-dim-major cache, consecutive rows -> consecutive slots
          const int g = gh - ro.H - ro.Hkv;
          for (int it = tid; it < CR * hd; it += NW * 64) {
            const int dd = it / CR, r = it - dd * CR, row = m0 + c0 + r;
            if (r >= nr || row >= M) continue;
            ro.cv[(((size_t)rsess[r] * ro.Hkv + g) * hd + dd) * ro.capacity + rslot[r]] =
                from_f32<TB>(sb[r * SP + dd]);
          }
        }
      }
    }
    return;
  }

  // Epilogue.  acc[i][j][e] is C[row = m0 + wm*WTM*16 + i*16 + lk*4 + e][col = .. + lr].
  if (ns > 1) {  // k-slice of a split tile: raw sums at [slice][tile row][W-tile row]
    // (rows past M are never read back)
    float *pt = part + ((size_t)(tile - full) * ns + sp) * (TBM * TBN);
#pragma unroll
    for (int ii = 0; ii < WTM; ++ii)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int lrow = wm * WTM * 16 + ii * 16 + lk * 4 + e;
        if (m0 + lrow >= M) continue;
#pragma unroll
        for (int j = 0; j < WTN; ++j) {
          const int tc = (EPI == acespec::EPI_SWIGLU)
                             ? (j < HALF ? wn * HALF * 16 + j * 16
                                         : TBN / 2 + wn * HALF * 16 + (j - HALF) * 16) + lr
                             : wn * WTN * 16 + j * 16 + lr;
          pt[lrow * TBN + tc] = acc[ii][j][e];
        }
      }
    return;
  }
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
          if (EPI == acespec::EPI_STORE) out[o] = (f16)acc[ii][j][e];
          else if (EPI == acespec::EPI_RESID) outf[o] += acc[ii][j][e];
          else outf[o] = acc[ii][j][e];
        }
      }
    }
  }
  if constexpr (EPI == acespec::EPI_F32_MAX) {
    // row maxima over this tile's columns (padding columns repeat the last real one):
    // over the wave's blocks in registers, its 16 column lanes by shuffles, then the
    // WNN waves of a row through LDS; tmax holds [M][nt].  A non-finite logit makes its
    // tile's maximum +inf, which the vocabulary kernel reports.
    __syncthreads();  // every wave is past the ring
    float *red = (float *)smem;  // [WNN][TBM]
#pragma unroll
    for (int ii = 0; ii < WTM; ++ii)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float m = -INFINITY;
#pragma unroll
        for (int j = 0; j < WTN; ++j) m = max_or_inf(m, acc[ii][j][e]);
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) m = fmaxf(m, __shfl_xor(m, o));
        if (lr == 0) red[wn * TBM + wm * WTM * 16 + ii * 16 + lk * 4 + e] = m;
      }
    __syncthreads();
    for (int r = tid; r < TBM; r += NW * 64) {
      if (m0 + r >= M) break;
      float m = red[r];
#pragma unroll
      for (int q = 1; q < WNN; ++q) m = fmaxf(m, red[q * TBM + r]);
      tmax[(size_t)(m0 + r) * nt + tn] = m;
    }
  }
}

// Sums the k-slices of the split tiles in a fixed order (deterministic) and applies the
// epilogue.  One thread per 4 adjacent tile columns of one tile row (SwiGLU: 4 gate
// columns and the matching 4 up columns).
template <int EPI, int TBM, int TBN>
__global__ __launch_bounds__(256) void tile_fixup_kernel(const float *__restrict__ part,
                                                         f16 *__restrict__ out,
                                                         float *__restrict__ outf, int M, int N,
                                                         int mt, int full, int nsplit_tiles,
                                                         int tsplit, float *__restrict__ tmax,
                                                         int nt) {
  constexpr int CW = (EPI == acespec::EPI_SWIGLU ? TBN / 2 : TBN) / 4;  // threads per row
  const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (gid >= (long long)nsplit_tiles * TBM * CW) return;
  const int t = (int)(gid / (TBM * CW));
  const int rem = (int)(gid - (long long)t * TBM * CW);
  const int lrow = rem / CW, c4 = (rem - lrow * CW) * 4;
  const int tile = full + t, tn = tile / mt, tm = tile - tn * mt;
  const int row = tm * TBM + lrow;
  // rows past M have no partials; with the row maxima their lanes still join the shuffles
  if (EPI != acespec::EPI_F32_MAX && row >= M) return;
  const float *pt = part + (size_t)t * tsplit * (TBM * TBN) + (size_t)lrow * TBN + c4;
  float4 a = make_float4(0.f, 0.f, 0.f, 0.f), g = a;
  for (int sp = 0; sp < (row < M ? tsplit : 0); ++sp) {
    const float4 v = *(const float4 *)(pt + (size_t)sp * (TBM * TBN));
    a.x += v.x; a.y += v.y; a.z += v.z; a.w += v.w;
    if (EPI == acespec::EPI_SWIGLU) {
      const float4 u = *(const float4 *)(pt + (size_t)sp * (TBM * TBN) + TBN / 2);
      g.x += u.x; g.y += u.y; g.z += u.z; g.w += u.w;
    }
  }
  if constexpr (EPI == acespec::EPI_F32_MAX) {
    // the CW threads of a tile row are CW consecutive lanes of one wave (CW divides 64)
    float m = max_or_inf(max_or_inf(max_or_inf(max_or_inf(-INFINITY, a.x), a.y), a.z), a.w);
#pragma unroll
    for (int o = 1; o < CW; o <<= 1) m = fmaxf(m, __shfl_xor(m, o));
    if (row >= M) return;
    if (c4 == 0) tmax[(size_t)row * nt + tn] = m;
  }
  const float av[4] = {a.x, a.y, a.z, a.w}, uv[4] = {g.x, g.y, g.z, g.w};
  const int col0 = tn * (EPI == acespec::EPI_SWIGLU ? TBN / 2 : TBN) + c4;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int col = col0 + q;
    if (col >= N) continue;
    const size_t o = (size_t)row * N + col;
    if (EPI == acespec::EPI_SWIGLU) out[o] = (f16)silu_mul(av[q], uv[q]);
    else if (EPI == acespec::EPI_STORE) out[o] = (f16)av[q];
    else if (EPI == acespec::EPI_RESID) outf[o] += av[q];
    else outf[o] = av[q];
  }
}

// Residual projection fixup fused with the following RMSNorm: one 256-thread block per
// row sums the row's k-slices (every tile sliced), adds them to the fp32 residual x,
// writes x back and emits RMSNorm(x) * gain.  Thread t owns the float4 columns
// t, t + 256, ... (at most 8, N <= 8192) in the same order as the RMSNorm kernel, so the
// result is bit-identical to the unfused path.
template <typename TG, int TBM, int TBN>
__global__ __launch_bounds__(256) void fixup_resid_norm_kernel(
    const float *__restrict__ part, float *__restrict__ x, const TG *__restrict__ gain,
    f16 *__restrict__ out, int N, int mt, int tsplit, float eps) {
  constexpr int MAXJ = 8;
  const int row = blockIdx.x, tid = threadIdx.x;
  const int tm = row / TBM, lrow = row - tm * TBM;
  const int n4 = N >> 2;
  float4 v[MAXJ];
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < MAXJ; ++j) {
    const int c = tid + 256 * j;
    if (c < n4) {
      const int col = 4 * c, tn = col / TBN, tc = col - tn * TBN;
      const float *pt = part + (size_t)(tn * mt + tm) * tsplit * (TBM * TBN) +
                        (size_t)lrow * TBN + tc;
      float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int sp = 0; sp < tsplit; ++sp) {
        const float4 w = *(const float4 *)(pt + (size_t)sp * (TBM * TBN));
        a.x += w.x; a.y += w.y; a.z += w.z; a.w += w.w;
      }
      float4 *xp = (float4 *)(x + (size_t)row * N) + c;
      float4 t = *xp;
      t.x += a.x; t.y += a.y; t.z += a.z; t.w += a.w;
      *xp = t;
      v[j] = t;
      ss += t.x * t.x + t.y * t.y + t.z * t.z + t.w * t.w;
    }
  }
  __shared__ float red[4];
  ss = wave_sum(ss);
  if ((tid & 63) == 0) red[tid >> 6] = ss;
  __syncthreads();
  const float tot = (red[0] + red[1]) + (red[2] + red[3]);
  const float scale = 1.0f / sqrtf(tot / (float)N + eps);
  f16 *o = out + (size_t)row * N;
#pragma unroll
  for (int j = 0; j < MAXJ; ++j) {
    const int c = tid + 256 * j;
    if (c < n4) {
      float g[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) g[e] = (float)gain[4 * c + e];
      typedef _Float16 h4 __attribute__((ext_vector_type(4)));
      *(h4 *)(o + 4 * c) = h4{(f16)(v[j].x * scale * g[0]), (f16)(v[j].y * scale * g[1]),
                              (f16)(v[j].z * scale * g[2]), (f16)(v[j].w * scale * g[3])};
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

// Packs a row-major bf16 weight matrix [rows, K] into the fp16 fragment order the packed
// GEMM path loads: 16-byte unit u = (nb * (K / 32) + kt) * 64 + l holds row nb * 16 + l % 16,
// columns kt * 32 + (l / 16) * 8 .. + 8 (the B operand of one v_mfma_f32_16x16x32_f16 per
// 64 units).  The widening is exact in the fp16 normal range (the same conversion the
// row-major path applies in registers), so both layouts give identical products.
__global__ __launch_bounds__(256) void pack_frag_kernel(const bf16 *__restrict__ W,
                                                        f16 *__restrict__ P, int rows, int K) {
  const long long u = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  const int KT = K >> 5;
  if (u >= (long long)(rows >> 4) * KT * 64) return;
  const int l = (int)(u & 63);
  const long long fr = u >> 6;
  const int kt = (int)(fr % KT), nb = (int)(fr / KT);
  const bf16x8 v = *(const bf16x8 *)(W + (size_t)(nb * 16 + (l & 15)) * K + kt * 32 + (l >> 4) * 8);
  *(f16x8 *)(P + u * 8) = bf16x8_to_f16x8(v);
}

using acespec::EPI_STORE;
using acespec::EPI_RESID;
using acespec::EPI_SWIGLU;
using acespec::EPI_F32;
using acespec::EPI_F32_MAX;

// Tilings: {waves M, waves N, wave tile M / 16, wave tile N / 16, stages, WGs per CU,
// k per stage, weight layout}.  Measured on MI355X against the verify-step shapes.  Tried
// and slower on every shape here with row-major weights: ping-pong pairs of waves per SIMD
// (one issuing 32 x 32 MFMAs while the other loads), deeper rings (5-8 stages) at one
// workgroup per CU, with 64 x 64 wave tiles or 128 x 512 block tiles (with packed weights
// 128 x 512 tiles are the fastest), 128 x 128 tiles with 64-wide k stages, fp16 weights
// (which only removes the in-register widening, worth 3-8 %), and weights and
// activations pre-packed into 1 KB tile blocks (contiguous DMA; 2-9 %), 256 x 128 tiles,
// and 256 x 256 tiles on 32 x 32 MFMAs with one wave per SIMD (128 x 128 wave tiles: the
// single wave cannot cover the barrier and DMA waits).
struct GemmVariant {
  int wmn, wnn, wtm, wtn, nst, occ, kss, pk;
};
constexpr GemmVariant kVariants[] = {
    {1, 4, 8, 4, 3, 2, 32, 0},  // 0: 128 x 256, 4 waves of 128 x 64, 72 KB LDS, 2 WGs per CU
    {2, 2, 4, 4, 4, 2, 32, 0},  // 1: 128 x 128, 4 waves of 64 x 64, 64 KB LDS, 2 WGs per CU
    {2, 4, 4, 4, 3, 1, 64, 0},  // 2: 128 x 256, 8 waves of 64 x 64, k 64, 144 KB LDS, 1 WG per CU
    {2, 4, 8, 4, 4, 1, 32, 0},  // 3: 256 x 256, 8 waves of 128 x 64, 128 KB LDS, 1 WG per CU
    {2, 2, 9, 2, 3, 1, 64, 0},  // 4: 288 x 64, 4 waves of 144 x 32, k 64, 132 KB LDS, 1 WG per CU
    // packed weights (registers fed straight from the fragment-ordered copy):
    {1, 4, 8, 4, 4, 2, 32, 1},  // 5: 128 x 256, 4 waves of 128 x 64, 32 KB ring, 2 WGs per CU
    {2, 4, 8, 4, 4, 1, 32, 1},  // 6: 256 x 256, 8 waves of 128 x 64, 64 KB ring, 1 WG per CU
    {2, 2, 4, 4, 4, 2, 32, 1},  // 7: 128 x 128, 4 waves of 64 x 64, 32 KB ring, 2 WGs per CU
    {2, 2, 9, 2, 4, 1, 32, 1},  // 8: 288 x 64, 4 waves of 144 x 32, 72 KB ring, 1 WG per CU
    {1, 4, 8, 4, 4, 1, 64, 2},  // 9: 128 x 256, two groups of 4 waves of 128 x 64 splitting k
    {2, 2, 4, 4, 4, 1, 64, 2},  // 10: 128 x 128, two groups of 4 waves of 64 x 64 splitting k
    {1, 8, 8, 4, 4, 1, 32, 1},  // 11: 128 x 512, 8 waves of 128 x 64, 32 KB ring, 1 WG per CU
    {1, 8, 4, 4, 4, 1, 32, 1},  // 12: 64 x 512, 8 waves of 64 x 64, 16 KB ring, 1 WG per CU
    {1, 4, 7, 4, 4, 1, 64, 2},  // 13: 112 x 256, two groups of 4 waves of 112 x 64 splitting k
};
constexpr int kNumVariants = sizeof(kVariants) / sizeof(kVariants[0]);

// Work split of a product: `full` whole tiles, then `tsplit` k-slices of each of the
// remaining tiles.  With at least one round of whole tiles, only the tiles of the last,
// partly empty round are sliced (enough slices to fill it); with fewer tiles than
// workgroup slots every tile is sliced, weighing the fill against the cost of the fp32
// partials.
struct SplitPlan {
  int full, tsplit;
};
SplitPlan plan_split(int M, int N, int K, int kss, int tbm, int tbn, int tiles, int cus, int occ,
                     long long part_cap) {
  const int slots = cus * occ;
  const int KT = K / kss;
  SplitPlan p{tiles, 1};
  if (tiles >= slots) {
    const int full = tiles / slots * slots, rest = tiles - full;
    if (rest == 0) return p;
    int sl = slots / rest;
    if (sl > 8) sl = 8;
    while (sl > 1 && KT / sl < 8) --sl;
    while (sl > 1 && (long long)rest * sl * tbm * tbn > part_cap) --sl;
    if (sl > 1) p = SplitPlan{full, sl};
    return p;
  }
  const double part_cost = (double)M * N * 4 / 10e12 / 0.43e-6 * (64.0 / kss);  // per slice
  int best = 1;
  double best_t = 1e30;
  for (int sl = 1; sl <= 8; ++sl) {
    if (KT / sl < 4) break;
    if ((long long)tiles * sl * tbm * tbn > part_cap) break;
    const double rounds = std::ceil((double)tiles * sl / slots);
    const double t = rounds * std::ceil((double)KT / sl) + (sl > 1 ? part_cost * sl : 0.0);
    if (t < best_t * 0.97) { best_t = t; best = sl; }
  }
  if (best > 1) p = SplitPlan{0, best};
  return p;
}

template <int EPI, int V, typename TB>
void launch_variant(hipStream_t s, const f16 *A, const TB *W, int M, int N, int K, f16 *out,
                    float *outf, float *part, int mt, int nt, SplitPlan sp,
                    const acespec::RopeOut<TB> &ro, float *tmax) {
  constexpr GemmVariant v = kVariants[V];
  constexpr int TBM = v.wmn * v.wtm * 16, TBN = v.wnn * v.wtn * 16;
  const int tiles = mt * nt;
  const int units = sp.full + (tiles - sp.full) * sp.tsplit;
  hipLaunchKernelGGL(
        (gemm_f16w_kernel<EPI, TB, v.wmn, v.wnn, v.wtm, v.wtn, v.nst, v.occ, v.kss, v.pk>),
        dim3(units), dim3(v.wmn * v.wnn * (v.pk == 2 ? 2 : 1) * 64), 0, s, A, W, M, N, K, out, outf, part, mt, nt,
        sp.full, sp.tsplit, ro, tmax);
  if (sp.tsplit > 1) {
    const int nsplit_tiles = tiles - sp.full;
    const long long threads =
        (long long)nsplit_tiles * TBM * ((EPI == EPI_SWIGLU ? TBN / 2 : TBN) / 4);
    hipLaunchKernelGGL((tile_fixup_kernel<EPI, TBM, TBN>), dim3((threads + 255) / 256),
                       dim3(256), 0, s, part, out, outf, M, N, mt, sp.full, nsplit_tiles,
                       sp.tsplit, tmax, nt);
  }
}

template <int EPI, typename TB>
void launch_epi(int var, hipStream_t s, const f16 *A, const TB *W, int M, int N, int K,
                f16 *out, float *outf, float *part, int mt, int nt, SplitPlan sp,
                const acespec::RopeOut<TB> &ro = acespec::RopeOut<TB>{},
                float *tmax = nullptr) {
  switch (var) {
#define CASE(V)                                                                             \
  case V:                                                                                   \
    if constexpr (kVariants[V].pk != 2 || EPI == acespec::EPI_QKV_ROPE)                     \
      launch_variant<EPI, V, TB>(s, A, W, M, N, K, out, outf, part, mt, nt, sp, ro, tmax);  \
    break;
    CASE(0) CASE(1) CASE(2) CASE(3) CASE(4) CASE(5) CASE(6) CASE(7) CASE(8) CASE(9) CASE(10) CASE(11) CASE(12) CASE(13)
#undef CASE
    default: break;
  }
}

// Default tiling per shape (measured on MI355X): 128 x 128 tiles for few rows (more
// tiles to spread over 256 CUs), the 8-wave 64-wide-k tiling for QKV-sized fp32
// outputs, 256 x 256 tiles (a third fewer operand bytes per flop, two stages in flight)
// for the residual and LM-head products once there are enough rows, 128 x 256 otherwise
// (for the gate/up product at ~1k rows both tilings measure the same, the 256 x 256 one
// only with its last round sliced).
int pick_variant(int epi, int M, int N, int K, int packed) {
  if (packed) {
    // measured on MI355X in the verify steps (272 - 4096 rows).  What sets these products'
    // rate is the bytes each CU's address unit moves per k-step: one 512-column tile of
    // eight waves shares its activation rows across twice the columns of a 256-column
    // one (40 instead of 48 KB a CU per k-step at 128 rows), so from ~500 rows the
    // products take 128 x 512 tiles (64 x 512 for the residual product with a short K
    // at ~520 rows, where 128-row tiles leave most of a last round empty); few-row
    // batches keep 288 x 64 tiles for the gate/up product and 128 x 128 ones otherwise
    if (epi == EPI_SWIGLU) return M <= 288 ? 8 : 11;
    if (M <= 384) return 7;
    if (epi == EPI_RESID) return K < 8192 && M <= 640 ? 12 : 11;
    if (M >= 512 && N >= 16384) return 11;
    if (M >= 2048) return 6;
    return 5;
  }
  // gate/up with up to 288 rows (a 16-session 1B-class batch: 272): one tile spans every
  // row, so each weight panel is read once and the product is one tile per CU (10 % faster
  // there; for the residual products, which are sliced along K, it measured slower)
  if (M <= 288 && epi == EPI_SWIGLU) return 4;
  if (M <= 384) return 1;
  if (epi == EPI_F32 && N <= 8192) return 2;
  if (M >= 1024 && epi != EPI_SWIGLU) return 3;
  return 0;
}

}  // namespace

namespace acespec {

template <typename TB>
hipError_t launch_f16w_variant(int var, int splits_override, int epi, const f16 *A,
                               const TB *W, int M, int N, int K, f16 *out, float *outf,
                               float *part, long long part_cap, int cus, hipStream_t s,
                               int packed) {
  if (var < 0) var = pick_variant(epi, M, N, K, packed);
  if (var >= kNumVariants || kVariants[var].pk != (packed ? 1 : 0)) return hipErrorInvalidValue;
  const GemmVariant v = kVariants[var];
  const int tbm = v.wmn * v.wtm * 16, tbn = v.wnn * v.wtn * 16;
  const int mt = (M + tbm - 1) / tbm;
  const int nt = epi == EPI_SWIGLU ? (N + tbn / 2 - 1) / (tbn / 2) : (N + tbn - 1) / tbn;
  const int tiles = mt * nt;
  SplitPlan sp = plan_split(M, N, K, v.kss, tbm, tbn, tiles, cus, v.occ, part_cap);
  if (splits_override == 1) sp = SplitPlan{tiles, 1};
  else if (splits_override > 1 &&
           (long long)tiles * splits_override * tbm * tbn <= part_cap)
    sp = SplitPlan{0, splits_override};
  switch (epi) {
    case EPI_STORE: launch_epi<EPI_STORE, TB>(var, s, A, W, M, N, K, out, outf, part, mt, nt, sp); break;
    case EPI_RESID: launch_epi<EPI_RESID, TB>(var, s, A, W, M, N, K, out, outf, part, mt, nt, sp); break;
    case EPI_SWIGLU: launch_epi<EPI_SWIGLU, TB>(var, s, A, W, M, N, K, out, outf, part, mt, nt, sp); break;
    default: launch_epi<EPI_F32, TB>(var, s, A, W, M, N, K, out, outf, part, mt, nt, sp);
  }
  return hipGetLastError();
}

template <int V, typename TB>
void launch_resid_norm_fixup(hipStream_t s, const float *part, float *x, const TB *gain,
                             f16 *out, int M, int N, int mt, int tsplit, float eps) {
  constexpr GemmVariant v = kVariants[V];
  constexpr int TBM = v.wmn * v.wtm * 16, TBN = v.wnn * v.wtn * 16;
  hipLaunchKernelGGL((fixup_resid_norm_kernel<TB, TBM, TBN>), dim3(M), dim3(256), 0, s, part,
                     x, gain, out, N, mt, tsplit, eps);
}

template <>
hipError_t launch_gemm_resid_norm<bf16, f16>(const f16 *A, const bf16 *W, int M, int N, int K,
                                             float *x, const bf16 *gain, f16 *out, float eps,
                                             const GemmAux &aux, hipStream_t s) {
  const int var = pick_variant(EPI_RESID, M, N, K, aux.packed);
  const GemmVariant v = kVariants[var];
  const int tbm = v.wmn * v.wtm * 16, tbn = v.wnn * v.wtn * 16;
  const int mt = (M + tbm - 1) / tbm, nt = (N + tbn - 1) / tbn;
  const SplitPlan sp =
      plan_split(M, N, K, v.kss, tbm, tbn, mt * nt, aux.cus, v.occ, aux.part_cap);
  if (sp.full != 0 || sp.tsplit < 2 || N % tbn != 0 || N > 8 * 4 * 256) {
    hipError_t e = launch_f16w_variant<bf16>(var, 0, EPI_RESID, A, W, M, N, K, nullptr, x,
                                             aux.part, aux.part_cap, aux.cus, s, aux.packed);
    if (e != hipSuccess) return e;
    return launch_rmsnorm<bf16, float>(x, gain, out, M, N, eps, s);
  }
  // every tile sliced: the GEMM writes only partials, the row kernel does the rest
  switch (var) {
#define CASE(VV)                                                                            \
  case VV: {                                                                                \
    constexpr GemmVariant g = kVariants[VV];                                                \
    hipLaunchKernelGGL(                                                                     \
        (gemm_f16w_kernel<EPI_RESID, bf16, g.wmn, g.wnn, g.wtm, g.wtn, g.nst, g.occ, g.kss,  \
                          g.pk>),                                                           \
        dim3(mt * nt * sp.tsplit), dim3(g.wmn * g.wnn * 64), 0, s, A, W, M, N, K, nullptr,   \
        x, aux.part, mt, nt, 0, sp.tsplit, RopeOut<bf16>{}, nullptr);                       \
    launch_resid_norm_fixup<VV, bf16>(s, aux.part, x, gain, out, M, N, mt, sp.tsplit, eps); \
    break;                                                                                  \
  }
    CASE(0) CASE(1) CASE(2) CASE(3) CASE(4) CASE(5) CASE(6) CASE(7) CASE(8) CASE(11) CASE(12)
#undef CASE
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template hipError_t launch_f16w_variant<bf16>(int, int, int, const f16 *, const bf16 *, int, int,
                                              int, f16 *, float *, float *, long long, int,
                                              hipStream_t, int);

hipError_t launch_pack_weights(const bf16 *W, f16 *P, int rows, int K, hipStream_t s) {
  if (rows <= 0 || K <= 0 || rows % 16 != 0 || K % 32 != 0) return hipErrorInvalidValue;
  const long long units = (long long)(rows / 16) * (K / 32) * 64;
  hipLaunchKernelGGL(pack_frag_kernel, dim3((unsigned)((units + 255) / 256)), dim3(256), 0, s, W,
                     P, rows, K);
  return hipGetLastError();
}

template <>
hipError_t launch_gemm<bf16, f16>(int epi, const f16 *A, const bf16 *W, int M, int N, int K,
                                  f16 *out, float *outf, const GemmAux &aux, hipStream_t s) {
  return launch_f16w_variant<bf16>(-1, 0, epi, A, W, M, N, K, out, outf, aux.part,
                                   aux.part_cap, aux.cus, s, aux.packed);
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

template <>
hipError_t launch_gemm_resid_norm<float, float>(const float *A, const float *W, int M, int N,
                                                int K, float *x, const float *gain, float *out,
                                                float eps, const GemmAux &aux, hipStream_t s) {
  hipError_t e = launch_gemm<float, float>(EPI_RESID, A, W, M, N, K, nullptr, x, aux, s);
  if (e != hipSuccess) return e;
  return launch_rmsnorm<float, float>(x, gain, out, M, N, eps, s);
}

template <>
hipError_t launch_qkv_rope<bf16, f16>(const f16 *A, const bf16 *W, int M, int N, int K,
                                      float *qkv, const RopeOut<bf16> &ro, const TreeMeta &meta,
                                      int B, const GemmAux &aux, hipStream_t s) {
  // packed weights: 128 x 256 tiles kept whole when they fill most CUs, so the RoPE and
  // cache write stay in the epilogue (measured level with the separate RoPE kernel after
  // a split product, and with eight 64 x 64 waves a tile)
  const bool fusable = N == (ro.H + 2 * ro.Hkv) * ro.hd;
  if (aux.packed && M > 384 && fusable && 128 % ro.hd == 0) {
    // tiles kept whole, each with two wave groups splitting its k-steps (two waves a SIMD
    // with about one tile a CU), RoPE and cache write in the epilogue: 112 x 256 tiles from
    // ~1k rows (1088 rows: 240 tiles for 256 CUs and 32 padding rows, against 216 tiles and
    // 64 rows at 128 x 256), 128 x 128 below
    const int gv = M >= 1024 ? 13 : 10;
    const GemmVariant g = kVariants[gv];
    const int mt = (M + g.wtm * 16 * g.wmn - 1) / (g.wtm * 16 * g.wmn);
    const int nt = (N + g.wtn * 16 * g.wnn - 1) / (g.wtn * 16 * g.wnn);
    if (4 * mt * nt >= 3 * aux.cus) {
      launch_epi<EPI_QKV_ROPE, bf16>(gv, s, A, W, M, N, K, nullptr, nullptr, aux.part, mt, nt,
                                     SplitPlan{mt * nt, 1}, ro);
      return hipGetLastError();
    }
  }
  const int var = aux.packed ? (M <= 384 ? 7 : 5) : pick_variant(EPI_F32, M, N, K, 0);
  const GemmVariant v = kVariants[var];
  const int tbm = v.wmn * v.wtm * 16, tbn = v.wnn * v.wtn * 16;
  const int mt = (M + tbm - 1) / tbm, nt = (N + tbn - 1) / tbn;
  SplitPlan sp = plan_split(M, N, K, v.kss, tbm, tbn, mt * nt, aux.cus, v.occ, aux.part_cap);
  if (aux.packed && 4 * mt * nt >= 3 * aux.cus) sp = SplitPlan{mt * nt, 1};
  if (sp.tsplit == 1 && tbn % ro.hd == 0 && fusable) {
    launch_epi<EPI_QKV_ROPE, bf16>(var, s, A, W, M, N, K, nullptr, nullptr, aux.part, mt, nt,
                                   sp, ro);
    return hipGetLastError();
  }
  hipError_t e = launch_f16w_variant<bf16>(var, 0, EPI_F32, A, W, M, N, K, nullptr, qkv,
                                           aux.part, aux.part_cap, aux.cus, s, aux.packed);
  if (e != hipSuccess) return e;
  return launch_rope_kv<bf16>(qkv, ro.q, meta, ro.ck, ro.cv, B, ro.n1, ro.H, ro.Hkv, ro.hd,
                              ro.capacity, ro.rot, s);
}

template <>
hipError_t launch_qkv_rope<float, float>(const float *A, const float *W, int M, int N, int K,
                                         float *qkv, const RopeOut<float> &ro,
                                         const TreeMeta &meta, int B, const GemmAux &aux,
                                         hipStream_t s) {
  hipError_t e = launch_gemm<float, float>(EPI_F32, A, W, M, N, K, nullptr, qkv, aux, s);
  if (e != hipSuccess) return e;
  return launch_rope_kv<float>(qkv, ro.q, meta, ro.ck, ro.cv, B, ro.n1, ro.H, ro.Hkv, ro.hd,
                               ro.capacity, ro.rot, s);
}

template <>
hipError_t launch_lm_head<bf16, f16>(const f16 *A, const bf16 *W, int M, int N, int K,
                                     float *logits, float *tile_max, int *ntile,
                                     const GemmAux &aux, hipStream_t s) {
  *ntile = 0;
  const int var = pick_variant(EPI_F32, M, N, K, aux.packed);
  const GemmVariant v = kVariants[var];
  const int tbm = v.wmn * v.wtm * 16, tbn = v.wnn * v.wtn * 16;
  const int mt = (M + tbm - 1) / tbm, nt = (N + tbn - 1) / tbn;
  SplitPlan sp = plan_split(M, N, K, v.kss, tbm, tbn, mt * nt, aux.cus, v.occ, aux.part_cap);
  if (tile_max == nullptr)
    return launch_f16w_variant<bf16>(var, 0, EPI_F32, A, W, M, N, K, nullptr, logits, aux.part,
                                     aux.part_cap, aux.cus, s, aux.packed);
  // the row maxima of sliced tiles are reduced by tbn / 4 lanes of one wave: wider tiles
  // stay whole (at most part of a last round idles)
  if (sp.tsplit > 1 && tbn / 4 > 64) sp = SplitPlan{mt * nt, 1};
  launch_epi<EPI_F32_MAX, bf16>(var, s, A, W, M, N, K, nullptr, logits, aux.part, mt, nt, sp,
                                RopeOut<bf16>{}, tile_max);
  *ntile = nt;
  return hipGetLastError();
}

template <>
hipError_t launch_lm_head<float, float>(const float *A, const float *W, int M, int N, int K,
                                        float *logits, float *, int *ntile, const GemmAux &aux,
                                        hipStream_t s) {
  *ntile = 0;
  return launch_gemm<float, float>(EPI_F32, A, W, M, N, K, nullptr, logits, aux, s);
}

}  // namespace acespec
