// Tree preparation: validates each session's drafted tree and derives the per-row data
// the forward pass needs.  All drafted nodes of a session go through the target in one
// pass (Section III-C); a node may attend to the verified context and to its own
// ancestral sequence only, so each row gets the set of its ancestors as a bit mask over
// the drafted rows (the root, row 0, is every row's ancestor and is always visible).
// Positions: siblings share a position, prefix_len + depth; keys/values of row r live
// in cache slot prefix_len + r.
#include "common.h"

namespace {

__global__ void tree_prep_kernel(const int32_t *__restrict__ tokens,
                                 const int32_t *__restrict__ parents,
                                 const int32_t *__restrict__ prefix_len, int B, int n1,
                                 int V, int capacity, TreeMeta meta,
                                 int32_t *__restrict__ status) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  const int32_t *tk = tokens + (size_t)b * n1;
  const int32_t *pr = parents + (size_t)b * n1;
  int S = prefix_len[b];
  bool ok = (S >= 0) && ((long long)S + n1 <= capacity) && (pr[0] == -1);
  for (int r = 1; r < n1 && ok; ++r) ok = (pr[r] >= 0) && (pr[r] < r);
  for (int r = 0; r < n1 && ok; ++r) ok = (tk[r] >= 0) && (tk[r] < V);
  if (S < 0) S = 0;
  if (S > capacity - n1) S = capacity - n1;
  meta.sess_S[b] = S;
  status[b] = ok ? ACESPEC_OK : ACESPEC_EBADTREE;
  const size_t base = (size_t)b * n1;
  // Rows are processed in order; parent < row, so the parent's entries are ready.
  for (int r = 0; r < n1; ++r) {
    int p = ok ? pr[r] : r - 1;  // malformed trees are replaced by a chain
    int t = tk[r];
    t = t < 0 ? 0 : (t >= V ? V - 1 : t);
    int depth = 0;
    uint64_t anc = 0;
    if (p >= 0) {
      depth = meta.depth[base + p] + 1;
      anc = meta.anc[base + p] | (1ull << (r - 1));
    }
    meta.tok[base + r] = t;
    meta.par[base + r] = p;
    meta.depth[base + r] = depth;
    meta.anc[base + r] = anc;
    meta.pos[base + r] = S + depth;
  }
}

}  // namespace

namespace acespec {

hipError_t launch_tree_prep(const int32_t *tokens, const int32_t *parents,
                            const int32_t *prefix_len, int B, int n1, int V, int capacity,
                            TreeMeta meta, int32_t *status, hipStream_t s) {
  const int threads = 64;
  hipLaunchKernelGGL(tree_prep_kernel, dim3((B + threads - 1) / threads), dim3(threads), 0, s,
                     tokens, parents, prefix_len, B, n1, V, capacity, meta, status);
  return hipGetLastError();
}

}  // namespace acespec
