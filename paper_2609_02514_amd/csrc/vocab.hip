// Fused vocabulary-wide verification: one workgroup per tree row, nothing of size
// [rows, vocab] is written back.
//
// For row r with logits z (fp32) the target distribution is p~ = softmax(z / T) cut to
// the top-p nucleus (the smallest most-probable set whose mass reaches top_p, ties in
// probability broken by lower token id, crossing token kept) and renormalised: p_r.
// The row produces
//   - the top-k payload: the k most probable ids and p_r on them renormalised (the sparse
//     partial distribution the cloud returns downlink, Section III-B),
//   - a bonus sample from p_r (inverse CDF in token-id order),
// and decides each drafted child n of r (token x, draft distribution Q = q[r]) by the
// speculative acceptance test of Chen et al. (cited in Section II):
//   accept[n] = u0 * Q(x) < p_r(x)         (u0 < min(1, p/q)),
//   resample[n] = inverse CDF of max(0, p_r - Q) at u1 (of p_r if that has no mass).
//
// Arithmetic: e = exp2((z - max) * log2(e) / T) in fp32 (the factor log2(e) / T and the
// nucleus normaliser each carried as a pair of floats); probability mass is summed in
// 2^-40 fixed point (64-bit integers), so every reduction is exact, order independent
// and run-to-run deterministic.  The nucleus and top-k thresholds are found by a radix
// select on the order-preserving 32-bit key of z (12 + 11 + 9 bits, histograms in LDS
// weighted by mass for top-p and by count for top-k), which finds the exact threshold
// logit and the number of tied ids to keep (ids ascending).  The inverse CDFs run over
// 256-id segments: segment masses are prefix-summed in LDS, and the chosen segment is
// re-read and scanned across a wavefront.
// Occupancy: 512 threads, 51 KB of LDS (the histograms of each pass and the segment
// tables share storage; the refinement levels are sized to fit under pass 1's) and at most
// 80 VGPRs per row, so three rows are in flight per CU and their scans and selections
// overlap each other's passes over memory (two rows a CU give about 1.45x the throughput
// of one, three about 10 % more than two); the row passes keep the next step's loads in
// flight while processing the current one.
#include "common.h"

namespace {

constexpr int VT = 512;             // threads per row (three rows in flight per CU)
constexpr int NWV = VT / 64;        // waves
constexpr int SEG = 256;            // ids per segment (one float4 per lane)
constexpr int SEGMAX = 1024;        // vocab <= 262144
constexpr int KMAX = 256;

typedef unsigned long long u64;

struct VSmem {
  // The threshold histograms (passes 1-3) and the per-segment tables (tie pass, pass 4)
  // are never live together; sharing their storage keeps two rows in flight per CU.
  union {
    struct {  // pass 1: bits 31..20 of the key
      uint32_t cnt[4096];
      u64 mass[4096];
    } h;
    struct {  // passes 2 and 3: bits 19..9, then 8..0, inside the selected bins
      uint32_t cnt[2048];
      u64 mass[2048];
      uint32_t cntk[2048];
    } r;
    struct {
      u64 seg_p[SEGMAX];       // per-segment mass of p_r, then its exclusive prefix
      u64 seg_r[SEGMAX];       // same for the residual max(0, p_r - Q)
      uint32_t tie_p[SEGMAX];  // per-segment count of ids tied at the top-p threshold (prefix)
      uint32_t tie_k[SEGMAX];
    } g;
  };
  u64 wsum[NWV];
  uint32_t wsum32[NWV];
  float wmax[NWV];
  uint32_t cand_key[KMAX];
  int32_t cand_id[KMAX];
  uint32_t cand_in[KMAX];
  uint32_t ncand;
  uint32_t nbin;           // elements of the selected top-p / top-k bins (pass 2)
  // selection results
  u64 above_p;
  uint32_t above_k;
  int sel_p, sel_k;
  int flag;                // data-error code of the row (0 = none)
};

AS_DEVICE u64 fixw(float v) { return __float2ull_rn(v * AS_FX_SCALE); }
// fixw(v) as a float, exactly: for v <= 1 the product is at most 2^40, and either it is
// already an integer (>= 2^23) or its rounding is below 2^24, so the value is representable.
AS_DEVICE float fixw_f(float v) { return rintf(v * AS_FX_SCALE); }

AS_DEVICE float key_to_f32(uint32_t key) {  // inverse of f32_key
  return __uint_as_float((key & 0x80000000u) ? (key & 0x7FFFFFFFu) : ~key);
}

// Block-wide exclusive scan (u64).  All threads must call it.
AS_DEVICE u64 block_scan_excl(u64 v, VSmem &sm, u64 &total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  u64 x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const u64 y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) sm.wsum[wave] = x;
  __syncthreads();
  u64 off = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < NWV; ++w) {
    const u64 s = sm.wsum[w];
    off += w < wave ? s : 0;
    tot += s;
  }
  __syncthreads();
  total = tot;
  return off + x - v;
}

AS_DEVICE u64 block_sum(u64 v, VSmem &sm) {
  u64 t;
  block_scan_excl(v, sm, t);
  return t;
}

AS_DEVICE float block_max(float v, VSmem &sm) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  v = wave_max(v);
  if (lane == 0) sm.wmax[wave] = v;
  __syncthreads();
  float m = sm.wmax[0];
#pragma unroll
  for (int w = 1; w < NWV; ++w) m = fmaxf(m, sm.wmax[w]);
  __syncthreads();
  return m;
}

// Descending radix step: bins b = nb-1 .. 0 hold (count, mass).  Finds the bin where the
// running mass from the top first reaches `target` (mass mode) or where the running
// count first reaches `target` (count mode); returns the bin and the amount strictly
// above it.  nb is 4096, 2048 or 512.
template <bool MASS>
AS_DEVICE void select_bin(VSmem &sm, const uint32_t *cnt, const u64 *mass, int nb, u64 target,
                          u64 base, int &sel, u64 &above) {
  const int t = threadIdx.x;
  if (t == 0) {  // defined result even if no bin qualifies (cannot happen for valid sums)
    if (MASS) { sm.sel_p = 0; sm.above_p = base; }
    else { sm.sel_k = 0; sm.above_k = (uint32_t)base; }
  }
  const int per = nb / VT > 0 ? nb / VT : 1;   // bins per thread
  const bool owner = t * per < nb;
  u64 local = 0;
  if (owner) {
    for (int j = 0; j < per; ++j) {
      const int bin = nb - 1 - (t * per + j);
      local += MASS ? mass[bin] : (u64)cnt[bin];
    }
  }
  u64 tot;
  u64 run = base + block_scan_excl(local, sm, tot);
  if (owner) {
    for (int j = 0; j < per; ++j) {
      const int bin = nb - 1 - (t * per + j);
      const u64 v = MASS ? mass[bin] : (u64)cnt[bin];
      if (run < target && run + v >= target) {
        if (MASS) { sm.sel_p = bin; sm.above_p = run; }
        else { sm.sel_k = bin; sm.above_k = (uint32_t)run; }
      }
      run += v;
    }
  }
  __syncthreads();
  sel = MASS ? sm.sel_p : sm.sel_k;
  above = MASS ? sm.above_p : (u64)sm.above_k;
  __syncthreads();
}

struct Sel {
  uint32_t tau_p, tau_k;   // exact threshold keys
  u64 above_p;             // mass strictly above tau_p
  uint32_t above_k;        // count strictly above tau_k
  uint32_t j_p, j_k;       // tied ids (ascending) kept at the thresholds
  uint32_t c_p, c_k;       // tie counts at the thresholds
  float M;                 // row max
  float c_hi, c_lo;        // log2(e) / T as a float pair
  float inv_hi, inv_lo;    // 1 / nucleus mass (fixed point units) as a float pair
};

// The raw v_exp_f32: for exponents >= -126 it is exactly exp2f (whose extra steps only
// rescale subnormal results), and anything below 2^-41 rounds to 0 in fixed point anyway.
// The exponent (z - M) log2(e) / T takes the factor as a float pair, so its error is the
// rounding of z - M and of the final sum only (random from element to element, not a
// tilt of the whole distribution).
AS_DEVICE float elem_e(float z, const Sel &s) {
  const float d = z - s.M;
  return __builtin_amdgcn_exp2f(fmaf(d, s.c_hi, d * s.c_lo));
}

// p_r of one element given its nucleus membership: the weight's fixed-point value times
// 1 / (nucleus mass), the latter again as a float pair.
AS_DEVICE float elem_p(float z, bool in, const Sel &s) {
  const float f = fixw_f(elem_e(z, s));
  return in ? fmaf(f, s.inv_hi, f * s.inv_lo) : 0.f;
}

// Nucleus / top-k membership given the element's rank among ids tied at the threshold.
AS_DEVICE bool in_nucleus(uint32_t key, uint32_t tie_rank, const Sel &s) {
  return key > s.tau_p || (key == s.tau_p && tie_rank < s.j_p);
}
AS_DEVICE bool in_topk(uint32_t key, uint32_t tie_rank, const Sel &s) {
  return key > s.tau_k || (key == s.tau_k && tie_rank < s.j_k);
}

// Wave-level exclusive prefix of per-lane counts.
AS_DEVICE uint32_t wave_excl_u32(uint32_t v) {
  const int lane = threadIdx.x & 63;
  uint32_t x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  return x - v;
}
AS_DEVICE u64 wave_incl_u64(u64 v) {
  const int lane = threadIdx.x & 63;
  u64 x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const u64 y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  return x;
}

// Per-lane tie ranks of the 4 elements a lane holds in segment s (ids s*256+lane*4+i).
AS_DEVICE void tie_ranks(const uint32_t key[4], bool valid, uint32_t tau, uint32_t base,
                         uint32_t rank[4]) {
  uint32_t n = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) n += (valid && key[i] == tau) ? 1u : 0u;
  uint32_t r = base + wave_excl_u32(n);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    rank[i] = r;
    r += (valid && key[i] == tau) ? 1u : 0u;
  }
}

// Inverse CDF inside segment s: the smallest id whose running mass exceeds `target`,
// where `excl` is the mass before the segment.  mode 0: p_r, mode 1: max(0, p_r - Q).
// Executed by one whole wave; returns the id (in every lane).
AS_DEVICE int seg_inverse_cdf(const float *z, const float *q, int V, int s, u64 excl, u64 target,
                              int mode, const Sel &sel, const VSmem &sm) {
  const int lane = threadIdx.x & 63;
  const int id0 = s * SEG + lane * 4;
  const bool valid = id0 < V;
  float4 z4 = make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
  float4 q4 = make_float4(0.f, 0.f, 0.f, 0.f);
  if (valid) {
    z4 = *(const float4 *)(z + id0);
    if (mode == 1) q4 = *(const float4 *)(q + id0);
  }
  const float zz[4] = {z4.x, z4.y, z4.z, z4.w};
  const float qq[4] = {q4.x, q4.y, q4.z, q4.w};
  uint32_t key[4], rank[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) key[i] = f32_key(zz[i]);
  if (sel.c_p > 1) tie_ranks(key, valid, sel.tau_p, sm.g.tie_p[s], rank);
  else {
#pragma unroll
    for (int i = 0; i < 4; ++i) rank[i] = 0;
  }
  u64 w[4];
  u64 lt = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float p = valid ? elem_p(zz[i], in_nucleus(key[i], rank[i], sel), sel) : 0.f;
    const float v = mode == 1 ? fmaxf(p - qq[i], 0.f) : p;
    w[i] = valid ? fixw(v) : 0;
    lt += w[i];
  }
  const u64 incl = excl + wave_incl_u64(lt);
  u64 run = incl - lt;
  int found = 0x7fffffff;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    run += w[i];
    if (found == 0x7fffffff && run > target && w[i] > 0) found = id0 + i;
  }
  // smallest id over the wave
  int f = found;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) f = min(f, __shfl_xor(f, o));
  return f < V ? f : V - 1;
}

// Finds the segment whose [excl, excl + mass) contains target (mass > 0); arrays hold
// exclusive prefixes.  Any lane may call it.
AS_DEVICE int find_segment(const u64 *excl, int nseg, u64 target) {
  int lo = 0, hi = nseg - 1;  // last segment with excl <= target
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (excl[mid] <= target) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

// Loads the VR float4 this thread handles in one step of a pass over the row, all issued
// before any is used: one load in flight per thread leaves the passes bound by memory
// latency rather than bandwidth.  Past the end of the row the row's last float4 is
// loaded again (V is a multiple of 4): every load is unconditional, so the compiler can
// wait for the older loads only, and the callers skip those entries (or, for the row
// maximum, take them: they repeat real elements).
constexpr int VR = 2;  // float4 a thread per step of the row passes (the segment pass: VU)
constexpr int VU = 2;
AS_DEVICE void load_step(const float *z, int V, int i0, float4 (&v)[VR]) {
#pragma unroll
  for (int u = 0; u < VR; ++u) {
    const int i = i0 + u * VT * 4;
    v[u] = *(const float4 *)(z + (i < V ? i : V - 4));
  }
}

// A pass over the row, VR float4 per thread a step: the next step's loads are issued
// before the current step is processed, so a thread always has loads in flight.
struct RowStream {
  const float *z;
  int V, i0;
  float4 cur[VR], nxt[VR];
  AS_DEVICE RowStream(const float *z_, int V_, int start) : z(z_), V(V_), i0(start) {
    load_step(z, V, i0, cur);
  }
  AS_DEVICE bool more() const { return i0 < V; }
  AS_DEVICE void prefetch() { load_step(z, V, i0 + VT * 4 * VR, nxt); }
  AS_DEVICE void advance() {
#pragma unroll
    for (int u = 0; u < VR; ++u) cur[u] = nxt[u];
    i0 += VT * 4 * VR;
  }
};

// (six waves a SIMD: three 8-wave rows per CU, which caps the kernel at 80 VGPRs)
__global__ __launch_bounds__(VT, 6) void vocab_verify_kernel(acespec::VocabArgs a) {
  __shared__ VSmem sm;
  const int row = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int V = a.V;
  const float *z = a.logits + (size_t)row * V;
  const int nseg = (V + SEG - 1) / SEG;

  // ---- pass 0: row max (+inf when a logit is not finite) -------------------------------
  float mx = -INFINITY;
  if (tid == 0) sm.flag = 0;
  if (a.tile_max) {  // the LM head's epilogue left the row's maximum per column tile
    const float *tm = a.tile_max + (size_t)row * a.ntile;
    for (int t = tid; t < a.ntile; t += VT) mx = max_or_inf(mx, tm[t]);
  } else {
    for (RowStream rs(z, V, tid * 4); rs.more(); rs.advance()) {
      rs.prefetch();
      const float4 (&vv)[VR] = rs.cur;
#pragma unroll
      for (int u = 0; u < VR; ++u)
        mx = max_or_inf(max_or_inf(max_or_inf(max_or_inf(mx, vv[u].x), vv[u].y), vv[u].z),
                        vv[u].w);
    }
  }
  Sel sel;
  sel.M = block_max(mx, sm);
  sel.c_hi = a.c_hi;
  sel.c_lo = a.c_lo;
  const bool tail = a.tail != 0;
  const int b = row / a.n1, r = row - b * a.n1;
  const size_t srow0 = (size_t)b * a.n1;
  if (!(sel.M <= 3.402823466e38f)) {
    // A logit of this row is NaN or infinite (an activation overflowed upstream): the row
    // gets no decisions, the session's status reports it.  Outputs stay defined.
    const int k = a.k;
    if (tid < k) {
      a.topk_ids[(size_t)row * k + tid] = -1;
      a.topk_probs[(size_t)row * k + tid] = 0.f;
    }
    if (tid == 0) {
      a.bonus[row] = -1;
      a.rowflag[row] = ACESPEC_ENONFINITE;
      if (!tail && r == 0) {
        a.accept[row] = 1;
        a.resample[row] = -1;
      }
    }
    const int c_lo = tail ? 0 : r + 1, c_hi = tail ? 1 : a.n1;
    for (int ci = c_lo + tid; ci < c_hi; ci += VT) {
      const int child = tail ? row : (int)(srow0 + ci);
      if (!tail && a.par[srow0 + ci] != r) continue;
      a.accept[child] = 0;
      a.resample[child] = -1;
    }
    return;
  }

  // ---- pass 1: total mass, 12-bit histograms ---------------------------------------
  for (int i = tid; i < 4096; i += VT) {
    sm.h.cnt[i] = 0;
    sm.h.mass[i] = 0;
  }
  if (tid == 0) sm.ncand = 0;
  __syncthreads();
  u64 tot = 0;
  for (RowStream rs(z, V, tid * 4); rs.more(); rs.advance()) {
    rs.prefetch();
    const int i0 = rs.i0;
    const float4 (&vv)[VR] = rs.cur;
#pragma unroll
    for (int u = 0; u < VR; ++u) {
      if (i0 + u * VT * 4 >= V) break;
      const float zz[4] = {vv[u].x, vv[u].y, vv[u].z, vv[u].w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t key = f32_key(zz[j]);
        const u64 w = fixw(elem_e(zz[j], sel));
        tot += w;
        atomicAdd(&sm.h.cnt[key >> 20], 1u);
        atomicAdd(&sm.h.mass[key >> 20], w);
      }
    }
  }
  const u64 S_fx = block_sum(tot, sm);  // includes a barrier after the histogram writes
  double tp = ceil((double)a.top_p * (double)S_fx);
  u64 T_p = (u64)tp;
  if (T_p < 1) T_p = 1;
  if (T_p > S_fx) T_p = S_fx;
  const u64 K = (u64)a.k;

  int bp, bk;
  u64 ap, ak;
  select_bin<true>(sm, sm.h.cnt, sm.h.mass, 4096, T_p, 0, bp, ap);
  select_bin<false>(sm, sm.h.cnt, sm.h.mass, 4096, K, 0, bk, ak);

  // ---- pass 2: refine bits 19..9 inside the selected bins ------------------------------
  // The keys of those bins' elements also go to a per-row scratch list (kept in L2), so
  // that pass 3 can read them instead of the row when they fit.
  __syncthreads();  // pass 1's bins are read; their storage is reused
  for (int i = tid; i < 2048; i += VT) {
    sm.r.cnt[i] = 0;
    sm.r.mass[i] = 0;
    sm.r.cntk[i] = 0;
  }
  if (tid == 0) sm.nbin = 0;
  uint32_t *cl = a.cand ? a.cand + (size_t)row * a.cand_cap : nullptr;
  __syncthreads();
  for (RowStream rs(z, V, tid * 4); rs.more(); rs.advance()) {
    rs.prefetch();
    const int i0 = rs.i0;
    const float4 (&vv)[VR] = rs.cur;
#pragma unroll
    for (int u = 0; u < VR; ++u) {
      if (i0 + u * VT * 4 >= V) break;
      const float zz[4] = {vv[u].x, vv[u].y, vv[u].z, vv[u].w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t key = f32_key(zz[j]);
        const int hi = key >> 20, mid = (key >> 9) & 0x7FF;
        if (hi == bp) {
          atomicAdd(&sm.r.cnt[mid], 1u);
          atomicAdd(&sm.r.mass[mid], fixw(elem_e(zz[j], sel)));
        }
        if (hi == bk) atomicAdd(&sm.r.cntk[mid], 1u);
        if (cl && (hi == bp || hi == bk)) {
          const uint32_t slot = atomicAdd(&sm.nbin, 1u);
          if (slot < (uint32_t)a.cand_cap) cl[slot] = key;
        }
      }
    }
  }
  __syncthreads();
  int sp, sk;
  u64 ap2, ak2;
  select_bin<true>(sm, sm.r.cnt, sm.r.mass, 2048, T_p, ap, sp, ap2);
  select_bin<false>(sm, sm.r.cntk, sm.r.mass, 2048, K, ak, sk, ak2);
  const uint32_t pre_p = ((uint32_t)bp << 11) | (uint32_t)sp;  // key bits 31..9
  const uint32_t pre_k = ((uint32_t)bk << 11) | (uint32_t)sk;

  // ---- pass 3: refine bits 8..0 ------------------------------------------------------
  for (int i = tid; i < 512; i += VT) {
    sm.r.cnt[i] = 0;
    sm.r.mass[i] = 0;
    sm.r.cntk[i] = 0;
  }
  const uint32_t nbin = sm.nbin;  // final: pass 2 ended with a barrier
  __syncthreads();
  if (cl && nbin <= (uint32_t)a.cand_cap) {
    // the candidates' keys (a key maps back to its logit exactly)
    for (uint32_t i = tid; i < nbin; i += VT) {
      const uint32_t key = cl[i];
      if ((key >> 9) == pre_p) {
        atomicAdd(&sm.r.cnt[key & 0x1FF], 1u);
        atomicAdd(&sm.r.mass[key & 0x1FF], fixw(elem_e(key_to_f32(key), sel)));
      }
      if ((key >> 9) == pre_k) atomicAdd(&sm.r.cntk[key & 0x1FF], 1u);
    }
  } else
  for (RowStream rs(z, V, tid * 4); rs.more(); rs.advance()) {
    rs.prefetch();
    const int i0 = rs.i0;
    const float4 (&vv)[VR] = rs.cur;
#pragma unroll
    for (int u = 0; u < VR; ++u) {
      if (i0 + u * VT * 4 >= V) break;
      const float zz[4] = {vv[u].x, vv[u].y, vv[u].z, vv[u].w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t key = f32_key(zz[j]);
        if ((key >> 9) == pre_p) {
          atomicAdd(&sm.r.cnt[key & 0x1FF], 1u);
          atomicAdd(&sm.r.mass[key & 0x1FF], fixw(elem_e(zz[j], sel)));
        }
        if ((key >> 9) == pre_k) atomicAdd(&sm.r.cntk[key & 0x1FF], 1u);
      }
    }
  }
  __syncthreads();
  int lp, lk;
  u64 ap3, ak3;
  select_bin<true>(sm, sm.r.cnt, sm.r.mass, 512, T_p, ap2, lp, ap3);
  select_bin<false>(sm, sm.r.cntk, sm.r.mass, 512, K, ak2, lk, ak3);
  sel.tau_p = (pre_p << 9) | (uint32_t)lp;
  sel.tau_k = (pre_k << 9) | (uint32_t)lk;
  sel.c_p = sm.r.cnt[lp];
  sel.c_k = sm.r.cntk[lk];
  sel.above_p = ap3;
  sel.above_k = (uint32_t)ak3;
  {
    const u64 w_tau = sm.r.mass[lp] / (sel.c_p ? sel.c_p : 1);
    const u64 need = T_p - ap3;  // > 0
    u64 j = w_tau ? (need + w_tau - 1) / w_tau : 1;
    if (j < 1) j = 1;
    if (j > sel.c_p) j = sel.c_p;
    sel.j_p = (uint32_t)j;
    sel.j_k = (uint32_t)(K - ak3);
    const u64 SN = ap3 + j * w_tau;
    const double inv = 1.0 / (double)SN;
    sel.inv_hi = (float)inv;
    sel.inv_lo = (float)(inv - (double)sel.inv_hi);
  }
  __syncthreads();

  // ---- optional pass: tie ranks at the thresholds (ids ascending) ------------------------
  const bool ties = sel.c_p > 1 || sel.c_k > 1;
  if (ties) {
    for (int s = wave; s < nseg; s += NWV) {
      const int id0 = s * SEG + lane * 4;
      uint32_t np = 0, nk = 0;
      if (id0 < V) {
        const float4 v = *(const float4 *)(z + id0);
        const float zz[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const uint32_t key = f32_key(zz[j]);
          np += key == sel.tau_p;
          nk += key == sel.tau_k;
        }
      }
      np = (uint32_t)wave_sum_i32((int)np);
      nk = (uint32_t)wave_sum_i32((int)nk);
      if (lane == 0) {
        sm.g.tie_p[s] = np;
        sm.g.tie_k[s] = nk;
      }
    }
    __syncthreads();
    if (tid == 0) {  // exclusive prefixes over segments (sequential: rare path)
      uint32_t rp = 0, rk = 0;
      for (int s = 0; s < nseg; ++s) {
        const uint32_t a0 = sm.g.tie_p[s], b0 = sm.g.tie_k[s];
        sm.g.tie_p[s] = rp;
        sm.g.tie_k[s] = rk;
        rp += a0;
        rk += b0;
      }
    }
    __syncthreads();
  }

  // ---- pass 4: id-ordered segments: masses of p_r and of the residual, top-k ids ----------
  bool has_child = tail;
  if (!tail) {
    for (int c = r + 1; c < a.n1; ++c) has_child |= a.par[srow0 + c] == r;
  }
  // Scalar mode: the uplink carries only q-hat of each drafted token (one float per
  // child row); the cloud then tests acceptance and does no sampling, so the residual
  // mass (the only reader of a dense q row) is not needed.
  const bool dense_q = a.q_scalar == nullptr;
  const bool resid = has_child && dense_q;
  const float *q = dense_q ? a.q + (size_t)row * V : nullptr;
  // The VU segments of a step are loaded before any is used.  Past the end of the row the
  // last float4 is loaded again (unconditional loads); those lanes are not valid below.
  // Every draft probability read is checked: NaN, infinite or negative flags the row.
  bool badq = false;
  for (int s0 = wave; s0 < nseg; s0 += NWV * VU) {
  float4 z4u[VU], q4u[VU];
#pragma unroll
  for (int u = 0; u < VU; ++u) {
    const int id0 = (s0 + u * NWV) * SEG + lane * 4;
    const int ld = id0 < V ? id0 : V - 4;
    // last pass over the row and its draft q: streamed past L2 and the MALL (the
    // earlier passes keep the default policy, so their re-reads may hit the MALL)
    z4u[u] = ld_stream(z + ld);
    q4u[u] = resid ? ld_stream(q + ld) : make_float4(0.f, 0.f, 0.f, 0.f);
  }
#pragma unroll
  for (int u = 0; u < VU; ++u) {
    const int s = s0 + u * NWV;
    if (s >= nseg) break;
    const int id0 = s * SEG + lane * 4;
    const bool valid = id0 < V;
    const float4 z4 = z4u[u], q4 = q4u[u];
    const float zz[4] = {z4.x, z4.y, z4.z, z4.w};
    const float qq[4] = {q4.x, q4.y, q4.z, q4.w};
    uint32_t key[4], rp[4], rk[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) key[j] = f32_key(zz[j]);
    if (sel.c_p > 1) tie_ranks(key, valid, sel.tau_p, sm.g.tie_p[s], rp);
    else {
#pragma unroll
      for (int j = 0; j < 4; ++j) rp[j] = 0;
    }
    if (sel.c_k > 1) tie_ranks(key, valid, sel.tau_k, sm.g.tie_k[s], rk);
    else {
#pragma unroll
      for (int j = 0; j < 4; ++j) rk[j] = 0;
    }
    u64 sp_ = 0, sr_ = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (!valid) continue;
      const bool inn = in_nucleus(key[j], rp[j], sel);
      const float p = elem_p(zz[j], inn, sel);
      sp_ += fixw(p);
      if (resid) {
        badq |= !(qq[j] >= 0.f && qq[j] <= 3.402823466e38f);
        sr_ += fixw(fmaxf(p - qq[j], 0.f));
      }
      if (in_topk(key[j], rk[j], sel)) {
        const uint32_t slot = atomicAdd(&sm.ncand, 1u);
        if (slot < KMAX) {
          sm.cand_key[slot] = key[j];
          sm.cand_id[slot] = id0 + j;
          sm.cand_in[slot] = inn ? 1u : 0u;
        }
      }
    }
    sp_ = wave_sum_u64(sp_);
    sr_ = wave_sum_u64(sr_);
    if (lane == 0) {
      sm.g.seg_p[s] = sp_;
      sm.g.seg_r[s] = sr_;
    }
  }
  }
  if (__syncthreads_or(badq) && tid == 0) sm.flag = ACESPEC_EBADDRAFT;
  // exclusive prefixes over segments
  u64 Ptot, Rtot;
  {
    constexpr int SPT = SEGMAX / VT;  // consecutive segments per thread
    u64 lp[SPT], lr[SPT], vp = 0, vr = 0;
#pragma unroll
    for (int j = 0; j < SPT; ++j) {
      const int sg = tid * SPT + j;
      lp[j] = sg < nseg ? sm.g.seg_p[sg] : 0;
      lr[j] = sg < nseg ? sm.g.seg_r[sg] : 0;
      vp += lp[j];
      vr += lr[j];
    }
    u64 ep = block_scan_excl(vp, sm, Ptot);
    u64 er = block_scan_excl(vr, sm, Rtot);
#pragma unroll
    for (int j = 0; j < SPT; ++j) {
      const int sg = tid * SPT + j;
      if (sg < nseg) {
        sm.g.seg_p[sg] = ep;
        sm.g.seg_r[sg] = er;
      }
      ep += lp[j];
      er += lr[j];
    }
  }
  __syncthreads();

  // ---- top-k payload: exactly k candidates, sorted by (key desc, id asc) -----------------
  const int k = a.k;
  {
    u64 wc = 0;
    int rank = 0, cid = 0;
    if (tid < k) {
      const uint32_t mk = sm.cand_key[tid];
      cid = sm.cand_id[tid];
      for (int j = 0; j < k; ++j) {
        const uint32_t ok = sm.cand_key[j];
        rank += (ok > mk) || (ok == mk && sm.cand_id[j] < cid);
      }
      wc = fixw(elem_p(key_to_f32(mk), sm.cand_in[tid] != 0, sel));
    }
    const u64 ksum = block_sum(wc, sm);
    if (tid < k) {
      a.topk_ids[(size_t)row * k + rank] = cid;
      a.topk_probs[(size_t)row * k + rank] = ksum ? (float)((double)wc / (double)ksum) : 0.f;
    }
  }

  // ---- bonus sample from p_r --------------------------------------------------------------
  const float *u = a.u;
  if (wave == 0) {
    int id = -1;
    if (dense_q) {
      const u64 target = (u64)floor((double)u[(size_t)row * 3 + 2] * (double)Ptot);
      const int sg = find_segment(sm.g.seg_p, nseg, target);
      id = seg_inverse_cdf(z, q, V, sg, sm.g.seg_p[sg], target, 0, sel, sm);
    }
    if (lane == 0) a.bonus[row] = id;
  }

  // ---- children: accept test and residual resample ------------------------------------------
  if (!tail && r == 0 && tid == 0) {
    a.accept[row] = 1;
    a.resample[row] = -1;
  }
  // Waves 1.. take the children in turn (wave 0 drew the bonus).
  if (has_child && wave >= 1) {
    int seen = 0;
    const int c_lo = tail ? 0 : r + 1, c_hi = tail ? 1 : a.n1;
    for (int ci = c_lo; ci < c_hi; ++ci) {
      int child;
      if (tail) {
        child = row;
      } else {
        if (a.par[srow0 + ci] != r) continue;
        child = (int)(srow0 + ci);
      }
      const bool mine = (seen % (NWV - 1)) + 1 == wave;
      ++seen;
      if (!mine) continue;
      int x = a.tok[child];
      x = x < 0 ? 0 : (x >= V ? V - 1 : x);
      // p_r(x): nucleus membership needs x's rank among ids tied at the threshold
      const float zx = z[x];
      const uint32_t kx = f32_key(zx);
      uint32_t rx = 0;
      if (kx == sel.tau_p && sel.c_p > 1) {
        const int sx = x / SEG;
        const int id0 = sx * SEG + lane * 4;
        const bool valid = id0 < V;
        const float4 z4 = valid ? *(const float4 *)(z + id0) : make_float4(0.f, 0.f, 0.f, 0.f);
        const uint32_t keys[4] = {f32_key(z4.x), f32_key(z4.y), f32_key(z4.z), f32_key(z4.w)};
        uint32_t rk4[4];
        tie_ranks(keys, valid, sel.tau_p, sm.g.tie_p[sx], rk4);
        const int src = (x - sx * SEG) >> 2;
        const uint32_t mine_rank = rk4[0] * ((x & 3) == 0) + rk4[1] * ((x & 3) == 1) +
                                   rk4[2] * ((x & 3) == 2) + rk4[3] * ((x & 3) == 3);
        rx = __shfl(mine_rank, src);
      }
      const float px = elem_p(zx, in_nucleus(kx, rx, sel), sel);
      const float qx = dense_q ? q[x] : a.q_scalar[child];
      if (!dense_q && !(qx >= 0.f && qx <= 1.f) && lane == 0) sm.flag = ACESPEC_EBADDRAFT;
      const float u0 = u[(size_t)child * 3 + 0], u1 = u[(size_t)child * 3 + 1];
      const bool acc = u0 * qx < px;
      int res = -1;
      if (!dense_q) {
        // no cloud-side resampling in the scalar protocol
      } else if (Rtot > 0) {
        const u64 target = (u64)floor((double)u1 * (double)Rtot);
        const int sg = find_segment(sm.g.seg_r, nseg, target);
        res = seg_inverse_cdf(z, q, V, sg, sm.g.seg_r[sg], target, 1, sel, sm);
      } else {
        const u64 target = (u64)floor((double)u1 * (double)Ptot);
        const int sg = find_segment(sm.g.seg_p, nseg, target);
        res = seg_inverse_cdf(z, q, V, sg, sm.g.seg_p[sg], target, 0, sel, sm);
      }
      if (lane == 0) {
        a.accept[child] = acc ? 1 : 0;
        a.resample[child] = res;
      }
    }
  }
  __syncthreads();
  if (tid == 0) a.rowflag[row] = sm.flag;
}

}  // namespace

namespace acespec {

hipError_t launch_vocab(const VocabArgs &a, hipStream_t s) {
  if (a.V > SEGMAX * SEG || a.k > KMAX || a.k < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(vocab_verify_kernel, dim3(a.rows), dim3(VT), 0, s, a);
  return hipGetLastError();
}

}  // namespace acespec
