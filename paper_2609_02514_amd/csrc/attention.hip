// Tree-masked grouped-query attention of the verify pass.
//
// Every drafted node of a session is verified in one forward pass (Section III-C): a
// node attends to the whole verified context (the KV prefix) and, among the tree's own
// slots, only to its ancestors and itself; the root is every node's ancestor.  Keys and
// values of tree row j sit in cache slot prefix_len + j, so one contiguous key range
// [0, prefix_len + N + 1) covers everything and the mask applies to its tail only.
//
// bf16 model: one workgroup per (split, kv head, session).  The G query heads of the
// kv head times the N+1 tree rows form the query rows (row = tree_row * G + head), in
// 16-row MFMA tiles spread over the workgroup's waves.  The key range of the split is
// streamed in 64-key chunks with coalesced 16-byte loads into LDS (keys XOR-swizzled,
// values with a padded row stride), converted from the bf16 cache to fp16 on the way
// (exact in the fp16 normal range); the next chunk's loads are in flight while the
// current chunk is processed.  Queries arrive in fp16.  S = Q K^T and O += P V use
// v_mfma_f32_16x16x32_f16 with fp32 accumulation and an online softmax in base 2; P
// (in [0, 1]) is rounded to fp16 and goes through a per-wave LDS tile to become an MFMA
// operand.  With several splits, unnormalised partial outputs
// and (max, sum) pairs are merged by a small combine kernel.
//
// fp32 kernel (tiny models): one wave per (tree row, query head), keys in sequence.
#include "common.h"

namespace {

constexpr int KC = 64;            // keys per chunk
constexpr float LOG2E = 1.4426950408889634f;

template <int HD>
struct AttnSmem {
  static constexpr int VSTRIDE = HD + 2;                   // fp16 elements per V row
  f16 k[KC * HD];
  f16 v[KC * VSTRIDE];
};

template <int HD>
AS_DEVICE int kswz(int key, int chunk) {  // 16-byte chunk index swizzled within the row
  return key * HD + ((chunk ^ (key & 7)) << 3);
}

AS_DEVICE bool tree_visible(int slot, int S, int n1, uint64_t anc) {
  if (slot < S) return true;
  const int j = slot - S;
  if (j >= n1) return false;
  return j == 0 || ((anc >> (j - 1)) & 1ull);
}

constexpr int NWAVES = 8;  // waves per workgroup (tiles are dealt to them in order)

template <int HD, int TPW>
__global__ __launch_bounds__(NWAVES * 64) void tree_attn_mfma_kernel(
    const f16 *__restrict__ qin, const bf16 *__restrict__ ck, const bf16 *__restrict__ cv,
    TreeMeta meta, f16 *__restrict__ out, float *__restrict__ part_o,
    float *__restrict__ part_ml, int n1, int H, int Hkv, int capacity, int nsplit) {
  constexpr int KSTEPS = HD / 32, NB = HD / 16, PSTRIDE = KC + 8;
  constexpr int VST = AttnSmem<HD>::VSTRIDE;
  __shared__ __attribute__((aligned(16))) AttnSmem<HD> sm;
  __shared__ __attribute__((aligned(16))) f16 sP[NWAVES][16 * PSTRIDE];

  const int split = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int G = H / Hkv, QR = G * n1;
  const int ntiles = (QR + 15) / 16;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lk = lane >> 4;
  const bool active = wave * TPW < ntiles;
  const int S = meta.sess_S[b];
  const int total = S + n1;
  const int nchunks = (total + KC - 1) / KC;
  const int cps = (nchunks + nsplit - 1) / nsplit;
  const int c_begin = split * cps;
  const int c_end = min(nchunks, c_begin + cps);
  const size_t kvbase = ((size_t)b * Hkv + g) * capacity * HD;
  const size_t row0 = (size_t)b * n1;
  const int q_stride = H * HD;
  const float sscale = LOG2E / sqrtf((float)HD);

  // Query fragments (A operand of S = Q K^T) and running softmax state.
  f16x8 qf[TPW][KSTEPS];
  f32x4 o[TPW][NB];
  float m_run[TPW][4], l_run[TPW][4];
#pragma unroll
  for (int t = 0; t < TPW; ++t) {
    const int tile = wave * TPW + t;
    int qi = tile * 16 + lr;
    qi = qi < QR ? qi : QR - 1;
    const int r = qi / G, h = g * G + (qi - r * G);
    const f16 *qp = qin + (row0 + r) * q_stride + h * HD;
#pragma unroll
    for (int s = 0; s < KSTEPS; ++s) qf[t][s] = *(const f16x8 *)(qp + s * 32 + lk * 8);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      m_run[t][e] = -INFINITY;
      l_run[t][e] = 0.f;
    }
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) o[t][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // Chunk staging: KC*HD/8 pieces of 16 bytes per operand.
  constexpr int PIECES = KC * HD / 8;
  constexpr int PPT = PIECES / (NWAVES * 64);
  bf16x8 rk[PPT], rv[PPT];
  auto load_chunk = [&](int c) {
    const int key0 = c * KC;
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
      const int p = tid + i * NWAVES * 64;
      const int key = p / (HD / 8), ch = p - key * (HD / 8);
      int slot = key0 + key;
      slot = slot < capacity ? slot : capacity - 1;
      rk[i] = *(const bf16x8 *)(ck + kvbase + (size_t)slot * HD + ch * 8);
      rv[i] = *(const bf16x8 *)(cv + kvbase + (size_t)slot * HD + ch * 8);
    }
  };
  auto store_chunk = [&]() {
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
      const int p = tid + i * NWAVES * 64;
      const int key = p / (HD / 8), ch = p - key * (HD / 8);
      *(f16x8 *)(&sm.k[kswz<HD>(key, ch)]) = bf16x8_to_f16x8(rk[i]);
      const f16x8 v16 = bf16x8_to_f16x8(rv[i]);
      uint32_t *vd = (uint32_t *)(&sm.v[key * VST + ch * 8]);
      const uint32_t *vs = (const uint32_t *)(&v16);
      vd[0] = vs[0];
      vd[1] = vs[1];
      vd[2] = vs[2];
      vd[3] = vs[3];
    }
  };

  if (c_begin < c_end) load_chunk(c_begin);
  f16 *myP = sP[wave];
  for (int c = c_begin; c < c_end; ++c) {
    __syncthreads();  // previous chunk fully consumed
    store_chunk();
    __syncthreads();
    if (c + 1 < c_end) load_chunk(c + 1);
    if (!active) continue;
    const int key0 = c * KC;
    const bool tree_chunk = key0 + KC > S;  // chunk reaches the tree slots: apply the mask

#pragma unroll
    for (int t = 0; t < TPW; ++t) {
      const int tile = wave * TPW + t;
      if (tile >= ntiles) break;
      // S = Q K^T for 4 blocks of 16 keys.
      f32x4 sc[4];
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        sc[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < KSTEPS; ++s) {
          const f16x8 kf = *(const f16x8 *)(&sm.k[kswz<HD>(kb * 16 + lr, s * 4 + lk)]);
          sc[kb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(qf[t][s], kf, sc[kb], 0, 0, 0);
        }
      }
      // Scale, mask (tree slots only), running max.  sc[kb][e] is the score of query row
      // tile*16 + lk*4 + e against key key0 + kb*16 + lr.
      uint64_t anc[4] = {~0ull, ~0ull, ~0ull, ~0ull};
      if (tree_chunk) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          int qo = tile * 16 + lk * 4 + e;
          qo = qo < QR ? qo : QR - 1;
          anc[e] = meta.anc[row0 + qo / G];
        }
      }
      float mx[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        const int slot = key0 + kb * 16 + lr;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          float v = sc[kb][e] * sscale;
          if (tree_chunk && !tree_visible(slot, S, n1, anc[e])) v = -INFINITY;
          sc[kb][e] = v;
          mx[e] = fmaxf(mx[e], v);
        }
      }
      float alpha[4], mref[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float v = mx[e];
        v = fmaxf(v, __shfl_xor(v, 1));
        v = fmaxf(v, __shfl_xor(v, 2));
        v = fmaxf(v, __shfl_xor(v, 4));
        v = fmaxf(v, __shfl_xor(v, 8));
        const float mnew = fmaxf(m_run[t][e], v);
        mref[e] = mnew == -INFINITY ? 0.f : mnew;
        alpha[e] = exp2f(m_run[t][e] - mref[e]);
        m_run[t][e] = mnew;
      }
      float rs[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const f16 pb = (f16)exp2f(sc[kb][e] - mref[e]);
          rs[e] += (float)pb;
          myP[(lk * 4 + e) * PSTRIDE + kb * 16 + lr] = pb;
        }
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float v = rs[e];
        v += __shfl_xor(v, 1);
        v += __shfl_xor(v, 2);
        v += __shfl_xor(v, 4);
        v += __shfl_xor(v, 8);
        l_run[t][e] = l_run[t][e] * alpha[e] + v;
      }
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int e = 0; e < 4; ++e) o[t][nb][e] *= alpha[e];

      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      // O += P V over two k-steps of 32 keys.  Both operands use key = s2*32 + lk*8 + j.
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        const f16x8 pa = *(const f16x8 *)(&myP[lr * PSTRIDE + s2 * 32 + lk * 8]);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          f16x8 vb;
          const f16 *vcol = &sm.v[(s2 * 32 + lk * 8) * VST + nb * 16 + lr];
#pragma unroll
          for (int j = 0; j < 8; ++j) vb[j] = vcol[j * VST];
          o[t][nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(pa, vb, o[t][nb], 0, 0, 0);
        }
      }
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    }
  }
  if (!active) return;

  // Output: o[t][nb][e] is row tile*16 + lk*4 + e, dim nb*16 + lr.
#pragma unroll
  for (int t = 0; t < TPW; ++t) {
    const int tile = wave * TPW + t;
    if (tile >= ntiles) break;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int qi = tile * 16 + lk * 4 + e;
      if (qi >= QR) continue;
      const int r = qi / G, h = g * G + (qi - r * G);
      if (nsplit == 1) {
        const float inv = l_run[t][e] > 0.f ? 1.0f / l_run[t][e] : 0.f;
        f16 *op = out + (row0 + r) * (size_t)(H * HD) + h * HD;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) op[nb * 16 + lr] = (f16)(o[t][nb][e] * inv);
      } else {
        const size_t item = ((size_t)b * Hkv + g) * nsplit + split;
        float *po = part_o + (item * QR + qi) * HD;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) po[nb * 16 + lr] = o[t][nb][e];
        if (lr == 0) {
          part_ml[(item * QR + qi) * 2 + 0] = m_run[t][e];
          part_ml[(item * QR + qi) * 2 + 1] = l_run[t][e];
        }
      }
    }
  }
}

// Merge of the split partials: one block per (kv head, session), one thread per value.
template <typename T>
__global__ void attn_combine_kernel(const float *__restrict__ part_o,
                                    const float *__restrict__ part_ml, T *__restrict__ out,
                                    int n1, int H, int Hkv, int HD, int nsplit) {
  const int g = blockIdx.x, b = blockIdx.y;
  const int G = H / Hkv, QR = G * n1;
  const size_t item0 = ((size_t)b * Hkv + g) * nsplit;
  for (int idx = threadIdx.x; idx < QR * HD; idx += blockDim.x) {
    const int qi = idx / HD, d = idx - qi * HD;
    float M = -INFINITY;
    for (int s = 0; s < nsplit; ++s) M = fmaxf(M, part_ml[((item0 + s) * QR + qi) * 2]);
    float num = 0.f, den = 0.f;
    for (int s = 0; s < nsplit; ++s) {
      const float m = part_ml[((item0 + s) * QR + qi) * 2];
      if (m == -INFINITY) continue;
      const float w = exp2f(m - M);
      den += w * part_ml[((item0 + s) * QR + qi) * 2 + 1];
      num += w * part_o[((item0 + s) * QR + qi) * HD + d];
    }
    const int r = qi / G, h = g * G + (qi - r * G);
    out[((size_t)b * n1 + r) * (H * HD) + h * HD + d] = from_f32<T>(den > 0.f ? num / den : 0.f);
  }
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
  const size_t kvbase = ((size_t)b * Hkv + g) * capacity * HD;
  const float scale = 1.0f / sqrtf((float)HD);
  float m = -INFINITY, l = 0.f, o0 = 0.f, o1 = 0.f;
  for (int slot = 0; slot < S + n1; ++slot) {
    if (!tree_visible(slot, S, n1, anc)) continue;
    const float *k = ck + kvbase + (size_t)slot * HD;
    const float *v = cv + kvbase + (size_t)slot * HD;
    float part = (lane < HD ? q0 * k[lane] : 0.f) + (lane + 64 < HD ? q1 * k[lane + 64] : 0.f);
    const float s = wave_sum(part) * scale;
    const float mn = fmaxf(m, s);
    const float a = expf(m - mn), p = expf(s - mn);
    l = l * a + p;
    o0 = o0 * a + p * (lane < HD ? v[lane] : 0.f);
    o1 = o1 * a + p * (lane + 64 < HD ? v[lane + 64] : 0.f);
    m = mn;
  }
  float *op = out + (size_t)row * (H * HD) + h * HD;
  if (lane < HD) op[lane] = o0 / l;
  if (lane + 64 < HD) op[lane + 64] = o1 / l;
}

template <int HD, int TPW>
void launch_mfma(dim3 grid, hipStream_t s, const f16 *q, const bf16 *ck, const bf16 *cv,
                 const TreeMeta &meta, f16 *out, float *po, float *pml, int n1, int H, int Hkv,
                 int capacity, int nsplit) {
  hipLaunchKernelGGL((tree_attn_mfma_kernel<HD, TPW>), grid, dim3(NWAVES * 64), 0, s, q, ck, cv,
                     meta, out, po, pml, n1, H, Hkv, capacity, nsplit);
}

}  // namespace

namespace acespec {

template <>
hipError_t launch_attention<bf16>(const f16 *q, const bf16 *ck, const bf16 *cv,
                                  const TreeMeta &meta, f16 *out, float *part_o,
                                  float *part_ml, long long part_capacity, int B, int n1, int H,
                                  int Hkv, int hd, int capacity, hipStream_t s,
                                  int *nsplit_used) {
  const int G = H / Hkv, QR = G * n1;
  const int tiles = (QR + 15) / 16;
  const int tpw = (tiles + NWAVES - 1) / NWAVES;
  if (tpw > 4) return hipErrorInvalidValue;
  // Splits over the key range so that the launch has enough workgroups to fill the
  // chip, keeping at least 8 chunks (512 keys) per split.
  const int items = B * Hkv;
  const int nchunks = (capacity + KC - 1) / KC;
  int nsplit = (512 + items - 1) / items;
  nsplit = nsplit < nchunks / 8 ? nsplit : nchunks / 8;
  if (nsplit < 1) nsplit = 1;
  while (nsplit > 1 && (long long)items * nsplit * QR * hd > part_capacity) --nsplit;
  *nsplit_used = nsplit;
  const dim3 grid(nsplit, Hkv, B);
#define GO(HD_, TPW_)                                                                     \
  launch_mfma<HD_, TPW_>(grid, s, q, ck, cv, meta, out, part_o, part_ml, n1, H, Hkv,      \
                         capacity, nsplit)
  if (hd == 128) {
    if (tpw == 1) GO(128, 1); else if (tpw == 2) GO(128, 2); else if (tpw == 3) GO(128, 3); else GO(128, 4);
  } else {
    if (tpw == 1) GO(64, 1); else if (tpw == 2) GO(64, 2); else if (tpw == 3) GO(64, 3); else GO(64, 4);
  }
#undef GO
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || nsplit == 1) return e;
  hipLaunchKernelGGL(attn_combine_kernel<f16>, dim3(Hkv, B), dim3(256), 0, s, part_o, part_ml,
                     out, n1, H, Hkv, hd, nsplit);
  return hipGetLastError();
}

template <>
hipError_t launch_attention<float>(const float *q, const float *ck, const float *cv,
                                   const TreeMeta &meta, float *out, float *, float *,
                                   long long, int B, int n1, int H, int Hkv, int hd,
                                   int capacity, hipStream_t s, int *nsplit_used) {
  *nsplit_used = 1;
  hipLaunchKernelGGL(tree_attn_f32_kernel, dim3(H, B * n1), dim3(64), 0, s, q, ck, cv, meta,
                     out, n1, H, Hkv, hd, capacity);
  return hipGetLastError();
}

}  // namespace acespec
