// Per-session path walk over the verification results (Algorithm 1: the walk after verification).
//
// From the root, follow the main (lowest-index) child while it is accepted.  When the
// main child is rejected, its residual resample is looked up among the other children
// of the same node (the outcome w = (pi, x_resampled) queried in the drafted tree): a hit
// continues down that sibling, a miss ends the path with the resampled token.  A node
// without children ends the path with its bonus token.  Also derives, per row, the
// number of leading accepted nodes on its root-to-row path.
#include "common.h"

namespace {

constexpr int MAXN1 = 65;

__global__ void walk_kernel(const int32_t *__restrict__ tok, const int32_t *__restrict__ par,
                            const uint8_t *__restrict__ accept,
                            const int32_t *__restrict__ resample,
                            const int32_t *__restrict__ bonus, int B, int n1,
                            int32_t *__restrict__ acc_prefix_len, int32_t *__restrict__ path,
                            int32_t *__restrict__ path_len, int32_t *__restrict__ next_token,
                            uint8_t *__restrict__ sibling_hit) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  const size_t base = (size_t)b * n1;
  int depth[MAXN1], acc[MAXN1];
  depth[0] = 0;
  acc[0] = 0;
  acc_prefix_len[base] = 0;
  for (int r = 1; r < n1; ++r) {
    const int p = par[base + r];
    depth[r] = depth[p] + 1;
    const bool full = acc[p] == depth[p];
    acc[r] = (full && accept[base + r]) ? acc[p] + 1 : acc[p];
    acc_prefix_len[base + r] = acc[r];
  }
  int cur = 0, len = 0, hit = 0, nxt = -1;
  while (true) {
    int main_c = -1;
    for (int c = cur + 1; c < n1; ++c)
      if (par[base + c] == cur) { main_c = c; break; }
    if (main_c < 0) { nxt = bonus[base + cur]; break; }
    if (accept[base + main_c]) {
      path[base + len++] = main_c;
      cur = main_c;
      continue;
    }
    const int rs = resample[base + main_c];
    int sib = -1;
    for (int c = main_c + 1; c < n1; ++c)
      if (par[base + c] == cur && tok[base + c] == rs) { sib = c; break; }
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
                                 const int32_t *__restrict__ draft, int nchains, int chain_len,
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
  for (int j = 0; j < chain_len; ++j) {
    const int t = draft[base + j];
    ok = ok && t >= 0 && t < V;
    acc_prefix_len[base + j] = i < j + 1 ? i : j + 1;
    path[base + j] = j < i ? j : -1;
  }
  path_len[c] = i;
  next_token[c] = i < chain_len ? resample[base + i] : -1;
  sibling_hit[c] = 0;
  status[c] = ok ? ACESPEC_OK : ACESPEC_EBADTREE;
}

}  // namespace

namespace acespec {

hipError_t launch_walk(const int32_t *tok, const int32_t *par, const uint8_t *accept,
                       const int32_t *resample, const int32_t *bonus, int B, int n1,
                       int32_t *acc_prefix_len, int32_t *path, int32_t *path_len,
                       int32_t *next_token, uint8_t *sibling_hit, hipStream_t s) {
  if (n1 > MAXN1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(walk_kernel, dim3((B + 63) / 64), dim3(64), 0, s, tok, par, accept,
                     resample, bonus, B, n1, acc_prefix_len, path, path_len, next_token,
                     sibling_hit);
  return hipGetLastError();
}

hipError_t launch_walk_tail(const uint8_t *accept, const int32_t *resample,
                            const int32_t *draft, int R, int chain_len, int V,
                            int32_t *acc_prefix_len, int32_t *path, int32_t *path_len,
                            int32_t *next_token, uint8_t *sibling_hit, int32_t *status,
                            hipStream_t s) {
  const int nchains = R / chain_len;
  hipLaunchKernelGGL(walk_tail_kernel, dim3((nchains + 63) / 64), dim3(64), 0, s, accept,
                     resample, draft, nchains, chain_len, V, acc_prefix_len, path, path_len,
                     next_token, sibling_hit, status);
  return hipGetLastError();
}

}  // namespace acespec
