// Tree-masked grouped-query attention of the verify pass.
//
// Every drafted node of a session is verified in one forward pass (Section III-C): a
// node attends to the whole verified context (the KV prefix) and, among the tree's own
// slots, only to its ancestors and itself; the root is every node's ancestor.  Keys and
// values of tree row j sit in cache slot prefix_len + j, so one contiguous key range
// [0, prefix_len + N + 1) covers everything and the mask applies to its tail only.
//
// bf16 model.  One workgroup of 16 waves (8 with more than 16 tiles) per (key split, kv
// head, session).  Query rows are the G query heads of the kv head times the N+1 tree rows
// (row = tree_row * G + head), in 16-row tiles dealt round-robin to the waves; with several
// tiles per wave, a last round of at most NW/4 tiles is split into quarter units (one
// 16-key block of every chunk each) on the waves that would otherwise idle, merged at the
// end through LDS.  The key range of the split streams through LDS in chunks of 64 slots:
//  * HBM -> LDS by direct DMA (buffer loads to LDS, 16 bytes a lane, nontemporal: the
//    cache is read once per step, and streaming it past L2 and the MALL measured 15 %
//    faster at the 8B shape) into a ring of NST stages.  The buffer form rather than the
//    global one: the compiler counts it on vmcnt alone, so its waits for the fragment
//    reads stay exact (1-3 % faster).  A stage holds the chunk's keys as [64 slots][head_dim] and its values,
//    read from the head-dim-major value cache, as [head_dim][64 slots].  The 16-byte
//    pieces of every row are XOR-swizzled so that the fragment reads below hit distinct
//    banks; the DMA fixes where each lane's bytes land, so the swizzle is applied to the
//    global source addresses.
//  * One chunk ahead of its use, the stage is widened from bf16 to fp16 in place (exact
//    in the fp16 normal range), so the MFMAs run on fp16 operands like the rest of the
//    pass, and the value columns past the last tree slot are zeroed (their probability
//    is 0, but 0 * NaN would not be).  Waves without a query tile do the widening when
//    there are any, which keeps it off the SIMD that holds two tile waves.
//  * Scores are computed transposed, S^T = K Q^T with v_mfma_f32_16x16x32_f16 (16 keys
//    as rows, 16 queries as columns), so each lane holds 16 scores of ONE query.  The
//    tree mask, the running max (reduced over the query's 4 lanes by two row swaps) and
//    exp2 stay in the lane, and the lane's probabilities, rounded to fp16, are exactly
//    its B operand of O^T = V^T P^T (the keys are assigned to MFMA rows so that a lane's
//    8 probabilities are 8 consecutive keys, whose V^T fragment is one 16-byte read).  The O^T
//    accumulator lane holds 4 head dims of its query, so the online-softmax rescale is
//    lane-local (and skipped when no running max moved).
//  * Barrier protocol at chunk c: a wave waits for its own DMA of chunk c+1; one LDS
//    barrier then certifies that chunk c+1 landed for every wave, that every wave
//    widened its share of chunk c, and that chunk c-1 is consumed, so its stage takes the
//    DMA of chunk c+NST-1.  NST-2 chunks are in flight while chunk c is computed.
//  With several splits, unnormalised partial outputs and (max, sum) pairs are merged by
//  a small combine kernel.
//
// fp32 kernel (tiny models): one wave per (tree row, query head), keys in sequence.
#include "common.h"

namespace {

constexpr int KC = 64;            // slots per chunk
// Opens the tree-mask branch of a chunk loop: an empty volatile asm cannot be executed
// speculatively, so the mask stays a branch taken only by the chunks that hold tree
// slots instead of being if-converted into selects that every chunk pays for.
#define MASK_BRANCH() __asm__ volatile("")

// The chunk barrier: this wave's LDS accesses (the widening's stores, the fragment reads)
// complete, then every wave of the workgroup arrives.  The DMA is not waited for here:
// each stage's DMA is waited for explicitly, NST - 2 chunks ahead.  (Written out rather
// than as an LDS release fence, with which the compiler drains every outstanding load,
// the DMA of the chunks in flight included, at every barrier of some of these kernels.)
// Online softmax with a lazy reference: the exponent's reference m moves to a new block
// maximum only when that maximum exceeds m by more than LAZY_LOG2 in base 2 (or m is
// unset), so the accumulators are rescaled a few times per query instead of at most
// blocks; the probabilities stay below 2^LAZY_LOG2, far inside fp16, and o / l is
// unchanged because numerator and denominator share the reference.
constexpr float LAZY_LOG2 = 8.f;
AS_DEVICE float lazy_ref(float m, float mx, float lazy) { return mx > m + lazy ? mx : m; }

AS_DEVICE void chunk_barrier() { __asm__ volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }
constexpr float LOG2E = 1.4426950408889634f;
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));

AS_DEVICE bool tree_visible(int slot, int S, int n1, uint64_t anc) {
  if (slot < S) return true;
  const int j = slot - S;
  if (j >= n1) return false;
  return j == 0 || ((anc >> (j - 1)) & 1ull);
}

// Order of the keys inside each 32-key group of a chunk: A row m of key block kk (16
// rows) holds key (kk/2)*32 + (m/4)*8 + (kk%2)*4 + m%4.  The score block's output row
// lg*4 + e is then key (kk/2)*32 + lg*8 + (kk%2)*4 + e, so the lane with row group lg
// holds the 8 consecutive keys (kk/2)*32 + lg*8 .. + 7 of its query -- one contiguous
// 16-byte read of a V^T row gives its A operand of O^T = V^T P^T.
AS_DEVICE int key_of_row(int kk, int m) { return (kk >> 1) * 32 + (m >> 2) * 8 + (kk & 1) * 4 + (m & 3); }
AS_DEVICE int key_of_score(int kk, int lg, int e) { return (kk >> 1) * 32 + lg * 8 + (kk & 1) * 4 + e; }

// XOR swizzles of the 16-byte pieces of a row, chosen so that each fragment read -- 16
// lanes at one logical piece of 16 rows (keys m = 0..15 of a block above, or 16
// consecutive V^T rows) -- runs at the LDS's full rate; measured on gfx950 with the
// kernel's own lane patterns (256-byte K rows: about 200 B/clk/CU with this key swizzle;
// 128-byte V^T rows: 210 B/clk/CU with row / 2, where row ^ (row / 8) halved it).
// K rows are 2*HD bytes.
template <int HD> AS_DEVICE int ksw(int key) {
  if (HD == 128) return (((key >> 3) & 3) << 2) | (key & 3);
  return ((key & 1) ^ ((key >> 4) & 1)) | (((key >> 1) & 1) << 1) | (((key >> 3) & 1) << 2);
}
AS_DEVICE int vsw(int row) { return (row >> 1) & 7; }
// K swizzle of the 32-row-tile kernel: its 16-lane fragment groups read 16 consecutive
// keys (bits 0-3 vary) in the main tiles and keys with bits 0, 1, 3, 4 varying in the
// remainder tile's quarter units; the XOR value below takes 16 (head_dim 128: 256-byte
// rows, one bank round each) or 2 x 8 (head_dim 64: rows alternate between the two
// halves of a bank round) distinct values on both sets.
template <int HD> AS_DEVICE int ksw32(int key) {
  const int b24 = ((key >> 2) ^ (key >> 4)) & 1;
  if (HD == 128) return (key & 0xB) | (b24 << 2);
  return ((key >> 1) & 1) | (b24 << 1) | (((key >> 3) & 1) << 2);
}
template <int HD, bool T32> AS_DEVICE int kswz(int key) {
  return T32 ? ksw32<HD>(key) : ksw<HD>(key);
}

// Element offset of piece `piece` of key row `key` in a stage's K part.
template <int HD> AS_DEVICE int k_off(int key, int piece) {
  return key * HD + ((piece ^ ksw<HD>(key)) << 3);
}
// Element offset of piece `piece` (8 slots) of head-dim row `row` in a stage's V^T part
// (rows of 64 slots = 128 bytes).
AS_DEVICE int v_off(int row, int piece) { return row * KC + ((piece ^ vsw(row)) << 3); }

// DMA of one chunk (keys key0 .. key0 + 63) into a stage: HD/8 blocks of 1 KB for K and
// as many for V^T, dealt to the NW waves in turn.
template <int HD, int NW, bool T32 = false>
AS_DEVICE void issue_chunk(uint16_t *stage, __amdgpu_buffer_rsrc_t kr,
                           __amdgpu_buffer_rsrc_t vr, int key0,
                           int capacity, int wave, int lane) {
  constexpr int BLOCKS = HD / 8;
  static_assert((2 * BLOCKS) % NW == 0, "DMA blocks per wave");
#pragma unroll
  for (int j = 0; j < 2 * BLOCKS / NW; ++j) {
    const int blk = wave + NW * j;
    if (blk < BLOCKS) {
      const int e = blk * 512 + lane * 8;          // element offset this lane's bytes land at
      const int key = e / HD, piece = (e % HD) >> 3;
      buf_dma16_stream(kr, (lds_ptr_t)(stage + blk * 512),
                       (uint32_t)((key0 + key) * HD + ((piece ^ kswz<HD, T32>(key)) << 3)) * 2u);
    } else {
      const int i = blk - BLOCKS;
      const int row = i * 8 + (lane >> 3), piece = lane & 7;
      buf_dma16_stream(vr, (lds_ptr_t)(stage + KC * HD + i * 512),
                       (uint32_t)(row * capacity + key0 + ((piece ^ vsw(row)) << 3)) * 2u);
    }
  }
}

// bf16 -> fp16 in place for pieces t, t + stride, ... of a stage (t: the thread's index
// among the widening threads); value slots >= total are zeroed.
template <int HD>
AS_DEVICE void widen_chunk(uint16_t *stage, int t, int stride, int key0, int total) {
  constexpr int KPIECES = KC * HD / 8;
  const bool tail = key0 + KC > total;
  for (int pc = t; pc < 2 * KPIECES; pc += stride) {
    uint16_t *p = stage + pc * 8;
    f16x8 h = bf16x8_to_f16x8(*(const bf16x8 *)p);
    if (tail && pc >= KPIECES) {
      const int vp = pc - KPIECES, row = vp >> 3;
      const int s0 = key0 + (((vp & 7) ^ vsw(row)) << 3);
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (s0 + e >= total) h[e] = (f16)0.f;
    }
    *(f16x8 *)p = h;
  }
}

template <int HD, int NW, int UPW, int NST>
__global__ __launch_bounds__(NW * 64) void tree_attn_mfma_kernel(
    const f16 *__restrict__ qin, const bf16 *__restrict__ ck, const bf16 *__restrict__ cv,
    TreeMeta meta, f16 *__restrict__ out, float *__restrict__ part_o,
    float *__restrict__ part_ml, int n1, int H, int Hkv, int capacity, int nsplit, int tpg) {
  constexpr int KSTEPS = HD / 32, NB = HD / 16;
  constexpr int STAGE = 2 * KC * HD;     // elements: K [KC][HD], then V^T [HD][KC]
  constexpr int L_DMA = HD / 4 / NW;     // DMA instructions per wave per chunk
  static_assert(NST >= 3, "the widening runs one stage ahead of the MFMAs");
  __shared__ __attribute__((aligned(1024))) uint16_t smem[NST * STAGE];

  const int g = blockIdx.y, b = blockIdx.z;
  const int G = H / Hkv, QR = G * n1;
  // Query groups: when the query rows of a kv head need more tiles than one workgroup
  // holds, consecutive groups of tpg tiles go to separate workgroups (each streams the
  // key range once); tbase is this group's first tile.
  const int all_tiles = (QR + 15) / 16, nqg = (all_tiles + tpg - 1) / tpg;
  const int split = blockIdx.x / nqg, tbase = (blockIdx.x - split * nqg) * tpg;
  const int ntiles = min(tpg, all_tiles - tbase);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  // With several tiles per wave, a last round of only a few tiles would leave the waves
  // that hold one waiting at every chunk barrier for the waves that hold one more; each of
  // those last rlast tiles is then split into 4 quarter units (one 16-key block of every
  // chunk each), run in slot QS by the last 4 * rlast waves and merged through LDS.
  constexpr int QS = UPW - 1;
  const int rlast = ntiles - NW * QS;
  const bool split_last = UPW > 1 && rlast >= 1 && 4 * rlast <= NW;
  const int qbase = NW - 4 * rlast;  // first wave holding a quarter unit
  const bool quarter = split_last && wave >= qbase;
  const int qk = (wave - qbase) & 3;  // a quarter unit's key block within each chunk
  const int S = meta.sess_S[b];
  const int total = S + n1;
  const int nchunks = (total + KC - 1) / KC;
  const int cps = (nchunks + nsplit - 1) / nsplit;
  const int c0 = split * cps;
  const int c1 = min(nchunks, c0 + cps);
  const bf16 *kb = ck + ((size_t)b * Hkv + g) * capacity * HD;
  const bf16 *vb = cv + ((size_t)b * Hkv + g) * HD * capacity;
  const __amdgpu_buffer_rsrc_t kr = make_rsrc(kb, (uint32_t)((size_t)capacity * HD * 2));
  const __amdgpu_buffer_rsrc_t vr = make_rsrc(vb, (uint32_t)((size_t)capacity * HD * 2));
  const size_t row0 = (size_t)b * n1;
  const int q_stride = H * HD;
  const float sscale = LOG2E / sqrtf((float)HD);   // scores -> base-2 exponent
  const float lazy = LAZY_LOG2 / sscale;           // reference threshold in score units

  // Query tile t of this wave: wave + NW t.  Per tile: query fragments (B operand of
  // S^T = K Q^T), ancestor mask, running softmax state.
  f16x8 qf[UPW][KSTEPS];
  uint64_t anc[UPW];
  float m_run[UPW], l_run[UPW];
  f32x4 o[UPW][NB];
#pragma unroll
  for (int t = 0; t < UPW; ++t) {
    const int tile = (split_last && t == QS) ? NW * QS + ((wave - qbase) >> 2) : wave + NW * t;
    int qi = (tbase + tile) * 16 + lr;   // (slot QS of a wave without a quarter unit: unused)
    qi = qi < 0 ? 0 : (qi < QR ? qi : QR - 1);
    const int r = qi / G, h = g * G + (qi - r * G);
    const f16 *qp = qin + (row0 + r) * q_stride + h * HD;
    // padding rows of the last tile multiply zeros (their outputs are dropped; zero
    // operands keep the MFMA's switching, and so its power draw, down)
    const bool pad = (tbase + tile) * 16 + lr >= QR;
#pragma unroll
    for (int s = 0; s < KSTEPS; ++s) {
      const f16x8 v = *(const f16x8 *)(qp + s * 32 + lg * 8);
      qf[t][s] = pad ? f16x8{} : v;
    }
    anc[t] = meta.anc[row0 + r];
    m_run[t] = -INFINITY;
    l_run[t] = 0.f;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) o[t][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  wait_vmcnt<0>();   // the loop's vmcnt accounting covers the DMA only

  auto stage_of = [&](int c) { return smem + ((c - c0) % NST) * STAGE; };
  // The widening goes to the waves without a tile when there are any (one SIMD then
  // holds no more than its share of tile work plus widening), else to every wave.
  const int wbeg = ntiles < NW ? ntiles : 0;
  const int wt = (wave - wbeg) * 64 + lane, wstride = (NW - wbeg) * 64;
  const bool widener = wave >= wbeg;

  // Prologue: chunks c0 .. c0+NST-2 in flight, chunk c0 widened.
#pragma unroll
  for (int i = 0; i < NST - 1; ++i)
    if (c0 + i < c1) issue_chunk<HD, NW>(stage_of(c0 + i), kr, vr, (c0 + i) * KC, capacity, wave, lane);
  if (c0 < c1) {
    if (c0 + NST - 2 < c1) wait_vmcnt<(NST - 2) * L_DMA>(); else wait_vmcnt<0>();
    lds_barrier();
    if (widener) widen_chunk<HD>(stage_of(c0), wt, wstride, c0 * KC, total);
  }

  // Fragment offsets: the swizzles depend on the lane only, so the read of K block kk at
  // k-step s is koff[s] + key_of_row(kk, 0) * HD and that of V^T block nb at key step ks is
  // voff[ks] + nb * 16 * KC -- a few lane registers plus compile-time constants.
  const int ksw_l = ksw<HD>(key_of_row(0, lr));
  int koff[KSTEPS], voff[2];
#pragma unroll
  for (int s = 0; s < KSTEPS; ++s)
    koff[s] = key_of_row(0, lr) * HD + (((s * 4 + lg) ^ ksw_l) << 3);
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) voff[ks] = v_off(lr, ks * 4 + lg);
  const int qkoff = key_of_row(qk, 0) * HD;                   // quarter: its key block
  const int qvoff = (qk & 2 ? voff[1] : voff[0]) + (qk & 1) * 4;  // and its V^T half-piece

  for (int c = c0; c < c1; ++c) {
    if (c + 1 < c1) {
      if (c + NST - 2 < c1) wait_vmcnt<(NST - 3) * L_DMA>(); else wait_vmcnt<0>();
    }
    chunk_barrier();
    if (c + NST - 1 < c1)
      issue_chunk<HD, NW>(stage_of(c + NST - 1), kr, vr, (c + NST - 1) * KC, capacity, wave, lane);
    if (c + 1 < c1 && widener) widen_chunk<HD>(stage_of(c + 1), wt, wstride, (c + 1) * KC, total);

    const uint16_t *st = stage_of(c);
    const f16 *sk = (const f16 *)st;
    const f16 *sv = (const f16 *)(st + KC * HD);
    const int key0 = c * KC;
    const bool tree_chunk = key0 + KC > S;
#pragma unroll
    for (int t = 0; t < UPW; ++t) {
      if (wave + NW * t >= ntiles || (split_last && t == QS)) break;
      // S^T for 4 blocks of 16 keys: sc[kk][e] is the score of slot
      // key0 + key_of_score(kk, lg, e) against this lane's query.
      f32x4 sc[4];
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) sc[kk] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < KSTEPS; ++s)
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          const f16x8 kf = *(const f16x8 *)(sk + koff[s] + key_of_row(kk, 0) * HD);
          sc[kk] = __builtin_amdgcn_mfma_f32_16x16x32_f16(kf, qf[t][s], sc[kk], 0, 0, 0);
        }
      if (tree_chunk) {
        MASK_BRANCH();
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            // the slot is tree row j (a prefix slot if j < 0)
            const int j = key0 + key_of_score(kk, lg, e) - S;
            const int sh = min(max(j - 1, 0), 63);
            const bool vis = (j < 0) | ((j < n1) & ((j == 0) | (bool)((anc[t] >> sh) & 1ull)));
            sc[kk][e] = vis ? sc[kk][e] : -INFINITY;
          }
      }
      float mx = -INFINITY;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
#pragma unroll
        for (int e = 0; e < 4; ++e) mx = fmaxf(mx, sc[kk][e]);
      mx = rows4_max(mx);
      const float m_new = lazy_ref(m_run[t], mx, lazy);
      const float m_use = m_new == -INFINITY ? 0.f : m_new;
      // raw v_exp_f32: results below 2^-126 flush to zero, which a softmax weight can spare
      const float alpha = __builtin_amdgcn_exp2f((m_run[t] - m_use) * sscale);
      m_run[t] = m_new;
      const float mb = m_use * sscale;
      f16x8 pb[2];
      float rs = 0.f;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float p = __builtin_amdgcn_exp2f(fmaf(sc[kk][e], sscale, -mb));
          rs += p;
          pb[kk >> 1][(kk & 1) * 4 + e] = (f16)p;
        }
      l_run[t] = l_run[t] * alpha + rs;
      if (__ballot(alpha < 1.f)) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int e = 0; e < 4; ++e) o[t][nb][e] *= alpha;
      }
      // O^T += V^T P^T over two k-steps of 32 keys.
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          const f16x8 va = *(const f16x8 *)(sv + voff[ks] + nb * 16 * KC);
          o[t][nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(va, pb[ks], o[t][nb], 0, 0, 0);
        }
    }
    if (quarter) {
      // One 16-key block (key block qk of the chunk) of the split tile: 4 scores a lane.
      f32x4 sq = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < KSTEPS; ++s) {
        const f16x8 kf = *(const f16x8 *)(sk + koff[s] + qkoff);
        sq = __builtin_amdgcn_mfma_f32_16x16x32_f16(kf, qf[QS][s], sq, 0, 0, 0);
      }
      if (tree_chunk) {
        MASK_BRANCH();
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int j = key0 + key_of_score(qk, lg, e) - S;
          const int sh = min(max(j - 1, 0), 63);
          const bool vis = (j < 0) | ((j < n1) & ((j == 0) | (bool)((anc[QS] >> sh) & 1ull)));
          sq[e] = vis ? sq[e] : -INFINITY;
        }
      }
      float mx = fmaxf(fmaxf(sq[0], sq[1]), fmaxf(sq[2], sq[3]));
      mx = rows4_max(mx);
      const float m_new = lazy_ref(m_run[QS], mx, lazy);
      const float m_use = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = __builtin_amdgcn_exp2f((m_run[QS] - m_use) * sscale);
      m_run[QS] = m_new;
      const float mb = m_use * sscale;
      f16x4 pq;
      float rs = 0.f;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float p = __builtin_amdgcn_exp2f(fmaf(sq[e], sscale, -mb));
        rs += p;
        pq[e] = (f16)p;
      }
      l_run[QS] = l_run[QS] * alpha + rs;
      if (__ballot(alpha < 1.f)) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int e = 0; e < 4; ++e) o[QS][nb][e] *= alpha;
      }
      // O^T += V^T P^T over the block's 16 keys: the lane's 4 probabilities are keys
      // (qk/2)*32 + lg*8 + (qk%2)*4 + 0..3, half of one 16-byte V^T piece.
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const f16x4 va = *(const f16x4 *)(sv + qvoff + nb * 16 * KC);
        o[QS][nb] = __builtin_amdgcn_mfma_f32_16x16x16f16(va, pq, o[QS][nb], 0, 0, 0);
      }
    }
  }
  wait_vmcnt<0>();

  if (split_last) {
    // Merge the quarter units of each split tile (the ring is free once every wave is
    // past its last chunk); each of a tile's 4 quarter waves finalises NB/4 head-dim blocks.
    __syncthreads();
    const int nquart = 4 * rlast;
    f32x4 *mo = (f32x4 *)smem;                                  // [quarter][NB][64 lanes]
    float *mml = (float *)smem + (size_t)nquart * NB * 64 * 4;  // [quarter][16 queries][2]
    const int qu = wave - qbase;
    if (quarter) {
      const float l = rows4_sum(l_run[QS]);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) mo[(qu * NB + nb) * 64 + lane] = o[QS][nb];
      if (lg == 0) {
        mml[(qu * 16 + lr) * 2 + 0] = m_run[QS] == -INFINITY ? -INFINITY : m_run[QS] * sscale;
        mml[(qu * 16 + lr) * 2 + 1] = l;
      }
    }
    __syncthreads();
    if (quarter) {
      const int q0 = qu & ~3, tile = NW * QS + (qu >> 2);
      float mj[4], wj[4];
      float M = -INFINITY;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        mj[j] = mml[((q0 + j) * 16 + lr) * 2];
        M = fmaxf(M, mj[j]);
      }
      float L = 0.f;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        wj[j] = mj[j] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mj[j] - M);
        L += wj[j] * mml[((q0 + j) * 16 + lr) * 2 + 1];
      }
      const int qi = (tbase + tile) * 16 + lr;
      if (qi < QR) {
        const int r = qi / G, h = g * G + (qi - r * G);
#pragma unroll
        for (int i = 0; i < NB / 4; ++i) {
          const int nb = qk * (NB / 4) + i;
          f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const f32x4 v = mo[((q0 + j) * NB + nb) * 64 + lane];
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[e] += wj[j] * v[e];
          }
          if (nsplit == 1) {
            const float inv = L > 0.f ? 1.0f / L : 0.f;
            f16x4 v;
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = (f16)(acc[e] * inv);
            *(f16x4 *)(out + (row0 + r) * (size_t)q_stride + h * HD + nb * 16 + lg * 4) = v;
          } else {
            const size_t item = ((size_t)b * Hkv + g) * nsplit + split;
            *(f32x4 *)(part_o + (item * QR + qi) * HD + nb * 16 + lg * 4) = acc;
          }
        }
        if (nsplit > 1 && qk == 0 && lg == 0) {
          const size_t item = ((size_t)b * Hkv + g) * nsplit + split;
          part_ml[(item * QR + qi) * 2 + 0] = M;
          part_ml[(item * QR + qi) * 2 + 1] = L;
        }
      }
    }
  }

  // o[t][nb][e] is head dim nb*16 + lg*4 + e of query tile*16 + lr.
#pragma unroll
  for (int t = 0; t < UPW; ++t) {
    const int tile = wave + NW * t;
    if (tile >= ntiles || (split_last && t == QS)) break;
    const float l = rows4_sum(l_run[t]);
    const int qi = (tbase + tile) * 16 + lr;
    if (qi >= QR) continue;
    const int r = qi / G, h = g * G + (qi - r * G);
    if (nsplit == 1) {
      const float inv = l > 0.f ? 1.0f / l : 0.f;
      f16 *op = out + (row0 + r) * (size_t)q_stride + h * HD + lg * 4;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        f16x4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = (f16)(o[t][nb][e] * inv);
        *(f16x4 *)(op + nb * 16) = v;
      }
    } else {
      const size_t item = ((size_t)b * Hkv + g) * nsplit + split;
      float *po = part_o + (item * QR + qi) * HD + lg * 4;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) *(f32x4 *)(po + nb * 16) = o[t][nb];
      if (lg == 0) {
        part_ml[(item * QR + qi) * 2 + 0] = m_run[t] == -INFINITY ? -INFINITY : m_run[t] * sscale;
        part_ml[(item * QR + qi) * 2 + 1] = l;
      }
    }
  }
}

// ------------------------------------------------------------------------------------
// 32-row query tiles, for kv heads whose query rows exceed 16 tiles of 16 (a 64-node tree
// under 4 or more query heads per kv head).  Eight waves, one 32-row tile each, on
// v_mfma_f32_32x32x16_f16: every 16-byte K or V^T fragment read now feeds 32 queries
// instead of 16, which halves the LDS fragment traffic per query, and each wave's chains
// are twice as long.  A remainder of at most 16 rows is one 16-row tile split into four
// quarter units (one 16-key block of every chunk each) on waves 4-7, which share SIMDs
// with waves 0-3, merged through LDS at the end.  At most 8 x 32 + 16 rows per workgroup;
// more rows are dealt to query groups of equal size.
//  * S^T = K Q^T per 32-key block: A row r holds key p32(r) of the block, B holds the 32
//    queries, so a lane holds 16 scores of one query (lane % 32) for keys
//    key32_of_score(i, lane / 32).  The two lanes of a query reduce their running max with
//    one 32-lane swap.
//  * O^T = V^T P^T per 16-key step: lane half h needs keys 8h .. 8h+7 of the step as its
//    B operand, which is exactly what p32 put in its scores; the matching V^T fragment is
//    one contiguous 16-byte read of a head-dim row.
// ------------------------------------------------------------------------------------
typedef float f32x16 __attribute__((ext_vector_type(16)));

// key (within a 32-key block) held by A row r of a 32 x 32 score block
AS_DEVICE int p32(int r) {
  return ((r >> 4) & 1) * 16 + ((r >> 2) & 1) * 8 + ((r >> 3) & 1) * 4 + (r & 3);
}
// key (within the block) of score i = 4 j + e of a lane in half h: output row 8 j + 4 h + e
AS_DEVICE int key32_of_score(int i, int h) {
  const int j = i >> 2, e = i & 3;
  return (j >> 1) * 16 + h * 8 + (j & 1) * 4 + e;
}
AS_DEVICE float halves_max(float v) {
  auto q = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(q[0]), __uint_as_float(q[1]));
}
AS_DEVICE float halves_sum(float v) {
  auto q = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(q[0]) + __uint_as_float(q[1]);
}

template <int HD, int NST>
__global__ __launch_bounds__(512) void tree_attn_t32_kernel(
    const f16 *__restrict__ qin, const bf16 *__restrict__ ck, const bf16 *__restrict__ cv,
    TreeMeta meta, f16 *__restrict__ out, float *__restrict__ part_o,
    float *__restrict__ part_ml, int n1, int H, int Hkv, int capacity, int nsplit, int rpg) {
  constexpr int NW = 8;
  constexpr int KS16 = HD / 16;   // 16-dim k-steps of a 32-row tile's S^T
  constexpr int NDB = HD / 32;    // 32-dim blocks of its O^T
  constexpr int KS32 = HD / 32;   // 32-dim k-steps of the remainder tile's S^T
  constexpr int NB16 = HD / 16;   // 16-dim blocks of the remainder tile's O^T
  constexpr int STAGE = 2 * KC * HD;
  constexpr int L_DMA = HD / 4 / NW;
  static_assert(NST >= 3, "the widening runs one stage ahead of the MFMAs");
  __shared__ __attribute__((aligned(1024))) uint16_t smem[NST * STAGE];

  const int g = blockIdx.y, b = blockIdx.z;
  const int G = H / Hkv, QR = G * n1;
  const int nqg = (QR + rpg - 1) / rpg;
  const int split = blockIdx.x / nqg, grp = blockIdx.x - split * nqg;
  const int rlo = grp * rpg, rows = min(rpg, QR - rlo);
  int n32 = rows >> 5, rem = rows & 31;
  if (rem > 16) {  // a remainder beyond 16 rows is a (padded) 32-row tile of its own
    ++n32;
    rem = 0;
  }
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lq = lane & 31, hh = lane >> 5;   // 32 x 32 layout: query column, lane half
  const int lr = lane & 15, lg = lane >> 4;   // 16 x 16 layout (remainder tile)
  const bool t32 = wave < n32;
  const bool quarter = rem > 0 && wave >= NW - 4;
  const int qk = wave & 3;                    // a quarter unit's key block in each chunk
  const int S = meta.sess_S[b];
  const int total = S + n1;
  const int nchunks = (total + KC - 1) / KC;
  const int cps = (nchunks + nsplit - 1) / nsplit;
  const int c0 = split * cps;
  const int c1 = min(nchunks, c0 + cps);
  const bf16 *kb = ck + ((size_t)b * Hkv + g) * capacity * HD;
  const bf16 *vb = cv + ((size_t)b * Hkv + g) * HD * capacity;
  const __amdgpu_buffer_rsrc_t kr = make_rsrc(kb, (uint32_t)((size_t)capacity * HD * 2));
  const __amdgpu_buffer_rsrc_t vr = make_rsrc(vb, (uint32_t)((size_t)capacity * HD * 2));
  const size_t row0 = (size_t)b * n1;
  const int q_stride = H * HD;
  const float sscale = LOG2E / sqrtf((float)HD);
  const float lazy = LAZY_LOG2 / sscale;

  // This wave's 32-row tile: query rlo + 32 wave + lq.  Padding rows (and the tile of a
  // wave without one) multiply zeros; their outputs are dropped.
  f16x8 qf[KS16];
  uint64_t anc;
  float m_run = -INFINITY, l_run = 0.f;
  f32x16 o[NDB];
  {
    const int qv = rlo + wave * 32 + lq;
    const bool pad = !t32 || qv >= rlo + rows;
    const int qi = min(qv, QR - 1);
    const int r = qi / G, h = g * G + (qi - r * G);
    const f16 *qp = qin + (row0 + r) * q_stride + h * HD;
#pragma unroll
    for (int s = 0; s < KS16; ++s) {
      const f16x8 v = *(const f16x8 *)(qp + s * 16 + hh * 8);
      qf[s] = pad ? f16x8{} : v;
    }
    anc = meta.anc[row0 + r];
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int i = 0; i < 16; ++i) o[db][i] = 0.f;
  }
  // The remainder tile (quarter waves): query rlo + 32 n32 + lr.
  f16x8 qq[KS32];
  uint64_t ancq;
  float mq = -INFINITY, lsq = 0.f;
  f32x4 oq[NB16];
  {
    const int qv = rlo + n32 * 32 + lr;
    const bool pad = !quarter || lr >= rem;
    const int qi = min(qv, QR - 1);
    const int r = qi / G, h = g * G + (qi - r * G);
    const f16 *qp = qin + (row0 + r) * q_stride + h * HD;
#pragma unroll
    for (int s = 0; s < KS32; ++s) {
      const f16x8 v = *(const f16x8 *)(qp + s * 32 + lg * 8);
      qq[s] = pad ? f16x8{} : v;
    }
    ancq = meta.anc[row0 + r];
#pragma unroll
    for (int nb = 0; nb < NB16; ++nb) oq[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  wait_vmcnt<0>();   // the loop's vmcnt accounting covers the DMA only

  auto stage_of = [&](int c) { return smem + ((c - c0) % NST) * STAGE; };
  const int wt = tid, wstride = NW * 64;   // every wave widens its share

  // Prologue: chunks c0 .. c0+NST-2 in flight, chunk c0 widened.
#pragma unroll
  for (int i = 0; i < NST - 1; ++i)
    if (c0 + i < c1)
      issue_chunk<HD, NW, true>(stage_of(c0 + i), kr, vr, (c0 + i) * KC, capacity, wave, lane);
  if (c0 < c1) {
    if (c0 + NST - 2 < c1) wait_vmcnt<(NST - 2) * L_DMA>(); else wait_vmcnt<0>();
    lds_barrier();
    widen_chunk<HD>(stage_of(c0), wt, wstride, c0 * KC, total);
  }

  // Fragment offsets (lane registers; blocks add compile-time constants): K row p32(lq)
  // (+32 for the second key block) at piece 2 s + hh; V^T row lq (+32 db) at piece
  // 2 ks + hh; the quarter unit's K row key_of_row(qk, lr) at piece 4 s + lg and its V^T
  // half-piece.
  const int krow = p32(lq), ksl = ksw32<HD>(krow);
  int koff[KS16];
#pragma unroll
  for (int s = 0; s < KS16; ++s) koff[s] = krow * HD + (((s * 2 + hh) ^ ksl) << 3);
  int voff[4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) voff[ks] = lq * KC + (((ks * 2 + hh) ^ vsw(lq)) << 3);
  const int qkey = key_of_row(qk, lr), qksl = ksw32<HD>(qkey);
  int qkoff[KS32];
#pragma unroll
  for (int s = 0; s < KS32; ++s) qkoff[s] = qkey * HD + (((s * 4 + lg) ^ qksl) << 3);
  const int qvoff = lr * KC + (((((qk >> 1) * 4) + lg) ^ vsw(lr)) << 3) + (qk & 1) * 4;

  for (int c = c0; c < c1; ++c) {
    if (c + 1 < c1) {
      if (c + NST - 2 < c1) wait_vmcnt<(NST - 3) * L_DMA>(); else wait_vmcnt<0>();
    }
    chunk_barrier();
    if (c + NST - 1 < c1)
      issue_chunk<HD, NW, true>(stage_of(c + NST - 1), kr, vr, (c + NST - 1) * KC, capacity,
                                wave, lane);
    if (c + 1 < c1) widen_chunk<HD>(stage_of(c + 1), wt, wstride, (c + 1) * KC, total);

    const uint16_t *st = stage_of(c);
    const f16 *sk = (const f16 *)st;
    const f16 *sv = (const f16 *)(st + KC * HD);
    const int key0 = c * KC;
    const bool tree_chunk = key0 + KC > S;
    if (t32) {
      // S^T for the chunk's two 32-key blocks: sc[kb][i] is the score of slot
      // key0 + 32 kb + key32_of_score(i, hh) against this lane's query.  Both blocks are
      // issued first; then each block gets its own online-softmax step and its P.V
      // products, so block 0's softmax runs on the VALU while block 1's scores are still
      // in the matrix pipe, and block 1's softmax while block 0's P.V runs.
      f32x16 sc[2];
#pragma unroll
      for (int kb2 = 0; kb2 < 2; ++kb2) {
#pragma unroll
        for (int i = 0; i < 16; ++i) sc[kb2][i] = 0.f;
#pragma unroll
        for (int s = 0; s < KS16; ++s) {
          const f16x8 kf = *(const f16x8 *)(sk + koff[s] + kb2 * 32 * HD);
          sc[kb2] = __builtin_amdgcn_mfma_f32_32x32x16_f16(kf, qf[s], sc[kb2], 0, 0, 0);
        }
      }
#pragma unroll
      for (int kb2 = 0; kb2 < 2; ++kb2) {
        SCHED_FENCE();
        f32x16 &z = sc[kb2];
        if (tree_chunk) {
          MASK_BRANCH();
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int j = key0 + kb2 * 32 + key32_of_score(i, hh) - S;  // tree row, or < 0
            const int sh = min(max(j - 1, 0), 63);
            const bool vis = (j < 0) | ((j < n1) & ((j == 0) | (bool)((anc >> sh) & 1ull)));
            z[i] = vis ? z[i] : -INFINITY;
          }
        }
        float mx = -INFINITY;
#pragma unroll
        for (int i = 0; i < 16; ++i) mx = fmaxf(mx, z[i]);
        mx = halves_max(mx);
        const float m_new = lazy_ref(m_run, mx, lazy);
        const float m_use = m_new == -INFINITY ? 0.f : m_new;
        const float alpha = __builtin_amdgcn_exp2f((m_run - m_use) * sscale);
        m_run = m_new;
        const float mb = m_use * sscale;
        // the block's probabilities as the B operands of its two 16-key steps: step
        // (j / 2) takes scores 4 j + e at positions (j % 2) * 4 + e
        f16x8 pk[2];
        float rs = 0.f;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float pz = __builtin_amdgcn_exp2f(fmaf(z[i], sscale, -mb));
          rs += pz;
          const int j = i >> 2, e = i & 3;
          pk[j >> 1][(j & 1) * 4 + e] = (f16)pz;
        }
        l_run = l_run * alpha + rs;
        if (__ballot(alpha < 1.f)) {
#pragma unroll
          for (int db = 0; db < NDB; ++db)
#pragma unroll
            for (int i = 0; i < 16; ++i) o[db][i] *= alpha;
        }
#pragma unroll
        for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
          for (int db = 0; db < NDB; ++db) {
            const f16x8 va = *(const f16x8 *)(sv + voff[kb2 * 2 + k2] + db * 32 * KC);
            o[db] = __builtin_amdgcn_mfma_f32_32x32x16_f16(va, pk[k2], o[db], 0, 0, 0);
          }
      }
      SCHED_FENCE();
    }
    if (quarter) {
      // key block qk of the chunk for the remainder tile: 4 scores a lane
      f32x4 sq = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < KS32; ++s) {
        const f16x8 kf = *(const f16x8 *)(sk + qkoff[s]);
        sq = __builtin_amdgcn_mfma_f32_16x16x32_f16(kf, qq[s], sq, 0, 0, 0);
      }
      if (tree_chunk) {
        MASK_BRANCH();
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int j = key0 + key_of_score(qk, lg, e) - S;
          const int sh = min(max(j - 1, 0), 63);
          const bool vis = (j < 0) | ((j < n1) & ((j == 0) | (bool)((ancq >> sh) & 1ull)));
          sq[e] = vis ? sq[e] : -INFINITY;
        }
      }
      float mx = fmaxf(fmaxf(sq[0], sq[1]), fmaxf(sq[2], sq[3]));
      mx = rows4_max(mx);
      const float m_new = lazy_ref(mq, mx, lazy);
      const float m_use = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = __builtin_amdgcn_exp2f((mq - m_use) * sscale);
      mq = m_new;
      const float mb = m_use * sscale;
      f16x4 pq;
      float rs = 0.f;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float p = __builtin_amdgcn_exp2f(fmaf(sq[e], sscale, -mb));
        rs += p;
        pq[e] = (f16)p;
      }
      lsq = lsq * alpha + rs;
      if (__ballot(alpha < 1.f)) {
#pragma unroll
        for (int nb = 0; nb < NB16; ++nb)
#pragma unroll
          for (int e = 0; e < 4; ++e) oq[nb][e] *= alpha;
      }
#pragma unroll
      for (int nb = 0; nb < NB16; ++nb) {
        const f16x4 va = *(const f16x4 *)(sv + qvoff + nb * 16 * KC);
        oq[nb] = __builtin_amdgcn_mfma_f32_16x16x16f16(va, pq, oq[nb], 0, 0, 0);
      }
    }
  }
  wait_vmcnt<0>();

  if (rem > 0) {
    // Merge the remainder tile's four quarter units (the ring is free once every wave is
    // past its last chunk); quarter wave qk finalises head-dim blocks qk * NB16/4 ...
    __syncthreads();
    f32x4 *mo = (f32x4 *)smem;                                 // [quarter][NB16][64 lanes]
    float *mml = (float *)smem + (size_t)4 * NB16 * 64 * 4;    // [quarter][16 queries][2]
    if (quarter) {
      const float l = rows4_sum(lsq);
#pragma unroll
      for (int nb = 0; nb < NB16; ++nb) mo[(qk * NB16 + nb) * 64 + lane] = oq[nb];
      if (lg == 0) {
        mml[(qk * 16 + lr) * 2 + 0] = mq == -INFINITY ? -INFINITY : mq * sscale;
        mml[(qk * 16 + lr) * 2 + 1] = l;
      }
    }
    __syncthreads();
    if (quarter) {
      float mj[4], wj[4];
      float M = -INFINITY;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        mj[j] = mml[(j * 16 + lr) * 2];
        M = fmaxf(M, mj[j]);
      }
      float L = 0.f;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        wj[j] = mj[j] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mj[j] - M);
        L += wj[j] * mml[(j * 16 + lr) * 2 + 1];
      }
      const int qi = rlo + n32 * 32 + lr;
      if (lr < rem) {
        const int r = qi / G, h = g * G + (qi - r * G);
        const size_t item = ((size_t)b * Hkv + g) * nsplit + split;
#pragma unroll
        for (int i = 0; i < NB16 / 4; ++i) {
          const int nb = qk * (NB16 / 4) + i;
          f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const f32x4 v = mo[(j * NB16 + nb) * 64 + lane];
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[e] += wj[j] * v[e];
          }
          if (nsplit == 1) {
            const float inv = L > 0.f ? 1.0f / L : 0.f;
            f16x4 v;
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = (f16)(acc[e] * inv);
            *(f16x4 *)(out + (row0 + r) * (size_t)q_stride + h * HD + nb * 16 + lg * 4) = v;
          } else {
            *(f32x4 *)(part_o + (item * QR + qi) * HD + nb * 16 + lg * 4) = acc;
          }
        }
        if (nsplit > 1 && qk == 0 && lg == 0) {
          part_ml[(item * QR + qi) * 2 + 0] = M;
          part_ml[(item * QR + qi) * 2 + 1] = L;
        }
      }
    }
  }

  // o[db][4 j + e] is head dim 32 db + 8 j + 4 hh + e of query rlo + 32 wave + lq.
  if (t32) {
    const float l = halves_sum(l_run);
    const int qi = rlo + wave * 32 + lq;
    if (qi < rlo + rows) {
      const int r = qi / G, h = g * G + (qi - r * G);
      if (nsplit == 1) {
        const float inv = l > 0.f ? 1.0f / l : 0.f;
        f16 *op = out + (row0 + r) * (size_t)q_stride + h * HD + hh * 4;
#pragma unroll
        for (int db = 0; db < NDB; ++db)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            f16x4 v;
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = (f16)(o[db][j * 4 + e] * inv);
            *(f16x4 *)(op + db * 32 + j * 8) = v;
          }
      } else {
        const size_t item = ((size_t)b * Hkv + g) * nsplit + split;
        float *po = part_o + (item * QR + qi) * HD + hh * 4;
#pragma unroll
        for (int db = 0; db < NDB; ++db)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            *(f32x4 *)(po + db * 32 + j * 8) =
                f32x4{o[db][j * 4], o[db][j * 4 + 1], o[db][j * 4 + 2], o[db][j * 4 + 3]};
        if (hh == 0) {
          part_ml[(item * QR + qi) * 2 + 0] = m_run == -INFINITY ? -INFINITY : m_run * sscale;
          part_ml[(item * QR + qi) * 2 + 1] = l;
        }
      }
    }
  }
}

// Merge of the split partials.  grid: (ceil(QR * HD / 4 / 256), kv heads, sessions); one
// thread per 4 head dims of one query row.  part_ml holds (max in base-2 exponent units,
// sum) per (item, query row).
template <typename T>
__global__ __launch_bounds__(256) void attn_combine_kernel(const float *__restrict__ part_o,
                                                           const float *__restrict__ part_ml,
                                                           T *__restrict__ out, int n1, int H,
                                                           int Hkv, int HD, int nsplit) {
  const int g = blockIdx.y, b = blockIdx.z;
  const int G = H / Hkv, QR = G * n1, hd4 = HD >> 2;
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= QR * hd4) return;
  const int qi = idx / hd4, d = (idx - qi * hd4) * 4;
  const size_t item0 = ((size_t)b * Hkv + g) * nsplit;
  float M = -INFINITY;
  for (int s = 0; s < nsplit; ++s) M = fmaxf(M, part_ml[((item0 + s) * QR + qi) * 2]);
  float4 num = make_float4(0.f, 0.f, 0.f, 0.f);
  float den = 0.f;
  for (int s = 0; s < nsplit; ++s) {
    const float m = part_ml[((item0 + s) * QR + qi) * 2];
    if (m == -INFINITY) continue;
    const float w = exp2f(m - M);
    den += w * part_ml[((item0 + s) * QR + qi) * 2 + 1];
    const float4 v = *(const float4 *)(part_o + ((item0 + s) * QR + qi) * HD + d);
    num.x += w * v.x;
    num.y += w * v.y;
    num.z += w * v.z;
    num.w += w * v.w;
  }
  const float inv = den > 0.f ? 1.f / den : 0.f;
  const int r = qi / G, h = g * G + (qi - r * G);
  T *o = out + ((size_t)b * n1 + r) * (H * HD) + h * HD + d;
  o[0] = from_f32<T>(num.x * inv);
  o[1] = from_f32<T>(num.y * inv);
  o[2] = from_f32<T>(num.z * inv);
  o[3] = from_f32<T>(num.w * inv);
}

// fp32 path: one wave per (tree row, query head); lane i owns dims i and i + 64.
__global__ __launch_bounds__(64) void tree_attn_f32_kernel(
    const float *__restrict__ qin, const float *__restrict__ ck, const float *__restrict__ cv,
    TreeMeta meta, float *__restrict__ out, int n1, int H, int Hkv, int HD, int capacity) {
  const int h = blockIdx.x, row = blockIdx.y;
  const int b = row / n1;
  const int G = H / Hkv, g = h / G, lane = threadIdx.x;
  const int S = meta.sess_S[b];
  const uint64_t anc = meta.anc[row];
  const float *q = qin + (size_t)row * H * HD + h * HD;
  const float q0 = lane < HD ? q[lane] : 0.f, q1 = lane + 64 < HD ? q[lane + 64] : 0.f;
  const float *kb = ck + ((size_t)b * Hkv + g) * capacity * HD;
  const float *vb = cv + ((size_t)b * Hkv + g) * HD * capacity;   // [HD][capacity]
  const float scale = 1.0f / sqrtf((float)HD);
  float m = -INFINITY, l = 0.f, o0 = 0.f, o1 = 0.f;
  for (int slot = 0; slot < S + n1; ++slot) {
    if (!tree_visible(slot, S, n1, anc)) continue;
    const float *k = kb + (size_t)slot * HD;
    float part = (lane < HD ? q0 * k[lane] : 0.f) + (lane + 64 < HD ? q1 * k[lane + 64] : 0.f);
    const float s = wave_sum(part) * scale;
    const float mn = fmaxf(m, s);
    const float a = expf(m - mn), p = expf(s - mn);
    l = l * a + p;
    o0 = o0 * a + p * (lane < HD ? vb[(size_t)lane * capacity + slot] : 0.f);
    o1 = o1 * a + p * (lane + 64 < HD ? vb[(size_t)(lane + 64) * capacity + slot] : 0.f);
    m = mn;
  }
  float *op = out + (size_t)row * (H * HD) + h * HD;
  if (lane < HD) op[lane] = o0 / l;
  if (lane + 64 < HD) op[lane + 64] = o1 / l;
}

// Ring depth: 4 stages of 32 KB (head_dim 128) or 16 KB (head_dim 64).
template <int HD> struct AttnCfg { static constexpr int NST = 4; };

template <int HD, int NW, int UPW>
void launch_mfma(dim3 grid, hipStream_t s, const f16 *q, const bf16 *ck, const bf16 *cv,
                 const TreeMeta &meta, f16 *out, float *po, float *pml, int n1, int H, int Hkv,
                 int capacity, int nsplit, int tpg) {
  hipLaunchKernelGGL((tree_attn_mfma_kernel<HD, NW, UPW, AttnCfg<HD>::NST>), grid,
                     dim3(NW * 64), 0, s, q, ck, cv, meta, out, po, pml, n1, H, Hkv,
                     capacity, nsplit, tpg);
}

}  // namespace

namespace acespec {

template <>
hipError_t launch_attention<bf16>(const f16 *q, const bf16 *ck, const bf16 *cv,
                                  const TreeMeta &meta, f16 *out, float *part_o,
                                  float *part_ml, long long part_capacity, int B, int n1, int H,
                                  int Hkv, int hd, int capacity, int cus, hipStream_t s,
                                  int *nsplit_used) {
  const int G = H / Hkv, QR = G * n1;
  const int all_tiles = (QR + 15) / 16;
  if (capacity % KC != 0) return hipErrorInvalidValue;
  // Up to 16 tiles of 16 rows: 16 waves, one tile per wave, the others widen (measured
  // fastest on the 8B shape: 5 tiles).  More rows: 8 waves of 32-row tiles plus a
  // remainder of at most 16 rows, i.e. up to 272 rows a workgroup; beyond that the rows
  // are dealt to query groups of equal size (8 query heads per kv head under a 64-node
  // tree: 520 rows, two groups of 260), each streaming the key range once.
  const bool t32 = all_tiles > 16;
  const int nqg = t32 ? (QR + 271) / 272 : 1;
  const int rpg = (QR + nqg - 1) / nqg;
  // Key splits so that every CU gets a workgroup, keeping at least 4 chunks per split.
  const int slots = cus;
  const int items = B * Hkv * nqg;
  const int nchunks = capacity / KC;
  int nsplit = (slots + items - 1) / items;
  nsplit = nsplit < nchunks / 4 ? nsplit : nchunks / 4;
  if (nsplit < 1) nsplit = 1;
  while (nsplit > 1 && (long long)B * Hkv * nsplit * QR * hd > part_capacity) --nsplit;
  *nsplit_used = nsplit;
  const dim3 grid(nsplit * nqg, Hkv, B);
  if (t32) {
    if (hd == 128)
      hipLaunchKernelGGL((tree_attn_t32_kernel<128, AttnCfg<128>::NST>), grid, dim3(512), 0, s,
                         q, ck, cv, meta, out, part_o, part_ml, n1, H, Hkv, capacity, nsplit,
                         rpg);
    else
      hipLaunchKernelGGL((tree_attn_t32_kernel<64, AttnCfg<64>::NST>), grid, dim3(512), 0, s,
                         q, ck, cv, meta, out, part_o, part_ml, n1, H, Hkv, capacity, nsplit,
                         rpg);
  } else if (hd == 128) {
    launch_mfma<128, 16, 1>(grid, s, q, ck, cv, meta, out, part_o, part_ml, n1, H, Hkv,
                            capacity, nsplit, all_tiles);
  } else {
    launch_mfma<64, 16, 1>(grid, s, q, ck, cv, meta, out, part_o, part_ml, n1, H, Hkv,
                           capacity, nsplit, all_tiles);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || nsplit == 1) return e;
  const int cblocks = (QR * (hd / 4) + 255) / 256;
  hipLaunchKernelGGL(attn_combine_kernel<f16>, dim3(cblocks, Hkv, B), dim3(256), 0, s, part_o,
                     part_ml, out, n1, H, Hkv, hd, nsplit);
  return hipGetLastError();
}

template <>
hipError_t launch_attention<float>(const float *q, const float *ck, const float *cv,
                                   const TreeMeta &meta, float *out, float *, float *,
                                   long long, int B, int n1, int H, int Hkv, int hd,
                                   int capacity, int, hipStream_t s, int *nsplit_used) {
  *nsplit_used = 1;
  hipLaunchKernelGGL(tree_attn_f32_kernel, dim3(H, B * n1), dim3(64), 0, s, q, ck, cv, meta,
                     out, n1, H, Hkv, hd, capacity);
  return hipGetLastError();
}

}  // namespace acespec
