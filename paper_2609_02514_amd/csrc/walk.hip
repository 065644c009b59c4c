// Per-session path walk over the verification results (Algorithm 1: the walk after verification).
//
// From the root, follow the main (lowest-index) child while it is accepted.  When the
// main child is rejected, its residual resample is looked up among the other children
// of the same node (the outcome w = (pi, x_resampled) queried in the drafted tree): a hit
// continues down that sibling, a miss ends the path with the resampled token.  A node
// without children ends the path with its bonus token.  Also derives, per row, the
// number of leading accepted nodes on its root-to-row path, and reports a data error the
// vocabulary kernel found in any of the session's rows in its status.
#include "common.h"

namespace {

constexpr int WALK_THREADS = 128;  // one thread per tree row (at most 65 rows)

// One workgroup per session.  Leading accepted nodes of row r's root-to-r path:
// min(depth[r], f[r] - 1), f[r] the depth of the shallowest rejected node on the path
// (the root is never tested), folded in by pointer jumping over the parents (7 rounds
// cover 65 rows).  The walk itself then runs on one thread over the session's data in
// LDS, with each node's main child found beforehand by an LDS minimum.
__global__ __launch_bounds__(WALK_THREADS) void walk_kernel(
    const int32_t *__restrict__ tok, const int32_t *__restrict__ par,
    const int32_t *__restrict__ depth, const uint8_t *__restrict__ accept,
    const int32_t *__restrict__ resample, const int32_t *__restrict__ bonus,
    const int32_t *__restrict__ rowflag, int B, int n1, int32_t *__restrict__ acc_prefix_len,
    int32_t *__restrict__ path, int32_t *__restrict__ path_len,
    int32_t *__restrict__ next_token, uint8_t *__restrict__ sibling_hit,
    int32_t *__restrict__ status) {
  constexpr int NONE = 1 << 30;
  __shared__ int s_flag;
  __shared__ int s_par[WALK_THREADS], s_tok[WALK_THREADS], s_rs[WALK_THREADS];
  __shared__ int s_bonus[WALK_THREADS], s_main[WALK_THREADS], s_jump[WALK_THREADS];
  __shared__ int s_f[WALK_THREADS];
  __shared__ uint8_t s_acc[WALK_THREADS];
  const int b = blockIdx.x, r = threadIdx.x;
  const size_t base = (size_t)b * n1;
  const bool in = r < n1;
  const int p = in ? par[base + r] : -1;
  const int d = in ? depth[base + r] : 0;
  const bool ok = r == 0 || !in || accept[base + r] != 0;
  s_par[r] = p;
  s_tok[r] = in ? tok[base + r] : -1;
  s_rs[r] = in ? resample[base + r] : -1;
  s_bonus[r] = in ? bonus[base + r] : -1;
  s_acc[r] = ok ? 1 : 0;
  s_main[r] = NONE;
  s_jump[r] = p < 0 ? 0 : p;
  s_f[r] = ok ? NONE : d;
  if (r == 0) s_flag = 0;
  __syncthreads();
  if (p >= 0) atomicMin(&s_main[p], r);
  // data-error codes of the session's rows (negative; the smallest, ENONFINITE, wins)
  if (in && rowflag[base + r] != 0) atomicMin(&s_flag, rowflag[base + r]);
  for (int round = 0; round < 7; ++round) {
    __syncthreads();
    const int jr = s_jump[r];
    const int f = min(s_f[r], s_f[jr]);
    const int jj = s_jump[jr];
    __syncthreads();
    s_f[r] = f;
    s_jump[r] = jj;
  }
  if (in) acc_prefix_len[base + r] = min(d, s_f[r] - 1);
  __syncthreads();  // main children and row flags complete
  if (r != 0) return;
  // a valid tree (tree prep wrote OK) with a data error in one of its rows
  if (s_flag != 0 && status[b] == ACESPEC_OK) status[b] = s_flag;
  int cur = 0, len = 0, hit = 0, nxt = -1;
  while (true) {  // every step moves to a higher row, so at most n1 steps
    const int main_c = s_main[cur];
    if (main_c == NONE) { nxt = s_bonus[cur]; break; }
    if (s_acc[main_c]) {
      path[base + len++] = main_c;
      cur = main_c;
      continue;
    }
    const int rs = s_rs[main_c];
    int sib = -1;
    for (int c = main_c + 1; c < n1; ++c)
      if (s_par[c] == cur && s_tok[c] == rs) { sib = c; break; }
    if (sib < 0) { nxt = rs; break; }
    path[base + len++] = sib;
    cur = sib;
    hit = 1;
  }
  for (int i = len; i < n1; ++i) path[base + i] = -1;
  path_len[b] = len;
  next_token[b] = nxt;
  sibling_hit[b] = (uint8_t)hit;
}

// LM-head tail: chains of chain_len rows, row i the parent of drafted token i.
__global__ void walk_tail_kernel(const uint8_t *__restrict__ accept,
                                 const int32_t *__restrict__ resample,
                                 const int32_t *__restrict__ draft,
                                 const int32_t *__restrict__ rowflag, int nchains, int chain_len,
                                 int V, int32_t *__restrict__ acc_prefix_len,
                                 int32_t *__restrict__ path, int32_t *__restrict__ path_len,
                                 int32_t *__restrict__ next_token,
                                 uint8_t *__restrict__ sibling_hit, int32_t *__restrict__ status) {
  const int c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= nchains) return;
  const size_t base = (size_t)c * chain_len;
  int i = 0;
  while (i < chain_len && accept[base + i]) ++i;
  bool ok = true;
  int flag = 0;
  for (int j = 0; j < chain_len; ++j) {
    const int t = draft[base + j];
    ok = ok && t >= 0 && t < V;
    flag = min(flag, rowflag[base + j]);
    acc_prefix_len[base + j] = i < j + 1 ? i : j + 1;
    path[base + j] = j < i ? j : -1;
  }
  path_len[c] = i;
  next_token[c] = i < chain_len ? resample[base + i] : -1;
  sibling_hit[c] = 0;
  status[c] = ok ? flag : ACESPEC_EBADTREE;
}

}  // namespace

namespace acespec {

hipError_t launch_walk(const int32_t *tok, const int32_t *par, const int32_t *depth,
                       const uint8_t *accept,
                       const int32_t *resample, const int32_t *bonus,
                       const int32_t *rowflag, int B, int n1, int32_t *acc_prefix_len,
                       int32_t *path, int32_t *path_len, int32_t *next_token,
                       uint8_t *sibling_hit, int32_t *status, hipStream_t s) {
  if (n1 > WALK_THREADS) return hipErrorInvalidValue;
  hipLaunchKernelGGL(walk_kernel, dim3(B), dim3(WALK_THREADS), 0, s, tok, par, depth, accept,
                     resample, bonus, rowflag, B, n1, acc_prefix_len, path, path_len,
                     next_token, sibling_hit, status);
  return hipGetLastError();
}

hipError_t launch_walk_tail(const uint8_t *accept, const int32_t *resample,
                            const int32_t *draft, const int32_t *rowflag, int R,
                            int chain_len, int V,
                            int32_t *acc_prefix_len, int32_t *path, int32_t *path_len,
                            int32_t *next_token, uint8_t *sibling_hit, int32_t *status,
                            hipStream_t s) {
  const int nchains = R / chain_len;
  hipLaunchKernelGGL(walk_tail_kernel, dim3((nchains + 63) / 64), dim3(64), 0, s, accept,
                     resample, draft, rowflag, nchains, chain_len, V, acc_prefix_len, path, path_len,
                     next_token, sibling_hit, status);
  return hipGetLastError();
}

}  // namespace acespec
