// Tree preparation: validates each session's drafted tree and derives the per-row data
// the forward pass needs.  All drafted nodes of a session go through the target in one
// pass (Section III-C); a node may attend to the verified context and to its own
// ancestral sequence only, so each row gets the set of its ancestors as a bit mask over
// the drafted rows (the root, row 0, is every row's ancestor and is always visible).
// Positions: siblings share a position, prefix_len + depth; keys/values of row r live
// in cache slot prefix_len + r.
#include "common.h"

namespace {

constexpr int TP_THREADS = 128;  // one thread per tree row (at most 65 rows)

// One workgroup per session.  A row's ancestor mask is its own bit and its ancestors'
// (the root carries none); it is built by pointer jumping, every row doubling the span of
// ancestors it has folded in per round (7 rounds cover 65 rows), and the row's depth is
// the mask's population count.
__global__ __launch_bounds__(TP_THREADS) void tree_prep_kernel(
    const int32_t *__restrict__ tokens, const int32_t *__restrict__ parents,
    const int32_t *__restrict__ prefix_len, int B, int n1, int V, int capacity, TreeMeta meta,
    int32_t *__restrict__ status) {
  __shared__ int s_jump[TP_THREADS];
  __shared__ uint64_t s_anc[TP_THREADS];
  const int b = blockIdx.x, r = threadIdx.x;
  const size_t base = (size_t)b * n1;
  const bool in = r < n1;
  const int pr = in ? parents[base + r] : 0;
  const int tk = in ? tokens[base + r] : 0;
  int S = prefix_len[b];
  const bool row_ok = !in || (((r == 0) ? (pr == -1) : (pr >= 0 && pr < r)) && tk >= 0 && tk < V);
  const bool ok = __syncthreads_and(row_ok) && S >= 0 && (long long)S + n1 <= capacity;
  if (S < 0) S = 0;
  if (S > capacity - n1) S = capacity - n1;
  const int p = !in || r == 0 ? -1 : (ok ? pr : r - 1);  // malformed trees become a chain
  s_jump[r] = p < 0 ? 0 : p;
  s_anc[r] = (in && r > 0) ? (1ull << (r - 1)) : 0ull;
  for (int round = 0; round < 7; ++round) {
    __syncthreads();
    const int jr = s_jump[r];
    const uint64_t a = s_anc[r] | s_anc[jr];
    const int jj = s_jump[jr];
    __syncthreads();
    s_anc[r] = a;
    s_jump[r] = jj;
  }
  if (r == 0) {
    meta.sess_S[b] = S;
    status[b] = ok ? ACESPEC_OK : ACESPEC_EBADTREE;
  }
  if (!in) return;
  const uint64_t anc = s_anc[r];
  const int depth = __popcll(anc);
  meta.tok[base + r] = tk < 0 ? 0 : (tk >= V ? V - 1 : tk);
  meta.par[base + r] = p;
  meta.depth[base + r] = depth;
  meta.anc[base + r] = anc;
  meta.pos[base + r] = S + depth;
}

}  // namespace

namespace acespec {

hipError_t launch_tree_prep(const int32_t *tokens, const int32_t *parents,
                            const int32_t *prefix_len, int B, int n1, int V, int capacity,
                            TreeMeta meta, int32_t *status, hipStream_t s) {
  if (n1 > TP_THREADS) return hipErrorInvalidValue;
  hipLaunchKernelGGL(tree_prep_kernel, dim3(B), dim3(TP_THREADS), 0, s, tokens, parents,
                     prefix_len, B, n1, V, capacity, meta, status);
  return hipGetLastError();
}

}  // namespace acespec
