// Commit of the verified path into the KV cache (Algorithm 1, COMPACT_KV; Section III-B:
// the cloud keeps the state of the accepted prefix and discards the rest of the tree).
//
// After a verify step the tree's keys and values sit in slots prefix_len + row.  The root
// (row 0) and the kept drafted rows path[0 .. path_len) move to the contiguous slots
// prefix_len + 0 .. prefix_len + path_len, i.e. to the positions a plain causal decode of
// the accepted tokens would have filled (a kept node at depth i has RoPE position
// prefix_len + i, so its rotated key is already the right one).  One workgroup per
// (layer, kv head, session); every source entry is read into LDS before any destination
// is written, because a destination slot may be another entry's source.
#include "common.h"

namespace {

constexpr int MAXE = 64 * 128;   // max moved entries (path rows x head dim) per workgroup

template <typename T>
__global__ __launch_bounds__(256) void commit_kv_kernel(T *__restrict__ ck, T *__restrict__ cv,
                                                        const int32_t *__restrict__ prefix_len,
                                                        const int32_t *__restrict__ path,
                                                        const int32_t *__restrict__ path_len,
                                                        const int32_t *__restrict__ status,
                                                        int B, int n1, int Hkv, int hd,
                                                        int capacity, int32_t *new_len) {
  __shared__ T kbuf[MAXE], vbuf[MAXE];
  const int lg = blockIdx.x, b = blockIdx.y;
  const int l = lg / Hkv, g = lg - l * Hkv;
  const int tid = threadIdx.x;
  const int S = prefix_len[b];
  const int np = path_len[b];
  bool ok = (status == nullptr || status[b] == ACESPEC_OK) && S >= 0 && S + n1 <= capacity &&
            np >= 0 && np < n1;
  // every kept row must be a drafted row of this tree
  const int32_t *pb = path + (size_t)b * n1;
  bool bad = !ok;
  if (ok && tid < np) bad = pb[tid] < 1 || pb[tid] >= n1;
  bad = __syncthreads_or(bad);
  if (lg == 0 && tid == 0) new_len[b] = bad ? -1 : S + 1 + np;
  if (bad || np == 0) return;

  const size_t head = ((size_t)l * B + b) * Hkv + g;   // (layer, session, kv head)
  T *kb = ck + head * capacity * hd;                   // [capacity][hd]
  T *vb = cv + head * hd * capacity;                   // [hd][capacity]
  const int ne = np * hd;
  // entry e: kept row i = e / hd + 1 (1-based; row 0 stays in place), dim d = e % hd
  for (int e = tid; e < ne; e += 256) {
    const int i = e / hd, d = e - i * hd;
    kbuf[e] = kb[(size_t)(S + pb[i]) * hd + d];
  }
  // values: slot-fastest order, so the writes below are contiguous runs of a row
  for (int e = tid; e < ne; e += 256) {
    const int d = e / np, i = e - d * np;
    vbuf[e] = vb[(size_t)d * capacity + S + pb[i]];
  }
  __syncthreads();
  for (int e = tid; e < ne; e += 256) {
    const int i = e / hd, d = e - i * hd;
    kb[(size_t)(S + 1 + i) * hd + d] = kbuf[e];
  }
  for (int e = tid; e < ne; e += 256) {
    const int d = e / np, i = e - d * np;
    vb[(size_t)d * capacity + S + 1 + i] = vbuf[e];
  }
}


// Value-cache layout conversion (not part of the verify step): every plane (layer,
// session, kv head) is a [rows][cols] matrix, written transposed as [cols][rows] --
// slot-major [capacity][head_dim] <-> the head-dim-major [head_dim][capacity] the verify
// step reads.  32 x 32 tiles pass through LDS so that reads and writes both run along
// rows; elements move as raw bits (E: 2 or 4 bytes).  One workgroup per tile.
template <typename E>
__global__ __launch_bounds__(256) void transpose_planes_kernel(const E *__restrict__ src,
                                                               E *__restrict__ dst, int rows,
                                                               int cols, int tiles_r,
                                                               int tiles_c) {
  __shared__ E tile[32][33];
  const int per_plane = tiles_r * tiles_c;
  const long long plane = blockIdx.x / per_plane;
  const int t = (int)(blockIdx.x - plane * per_plane);
  const int tr = t / tiles_c, tc = t - tr * tiles_c;
  const size_t base = (size_t)plane * rows * cols;
  const int x = threadIdx.x & 31, y = threadIdx.x >> 5;  // 32 x 8 threads
  for (int i = y; i < 32; i += 8) {
    const int r = tr * 32 + i, c = tc * 32 + x;
    if (r < rows && c < cols) tile[i][x] = src[base + (size_t)r * cols + c];
  }
  __syncthreads();
  for (int i = y; i < 32; i += 8) {
    const int c = tc * 32 + i, r = tr * 32 + x;  // destination row c, column r
    if (c < cols && r < rows) dst[base + (size_t)c * rows + r] = tile[x][i];
  }
}

}  // namespace

namespace acespec {

template <typename T>
hipError_t launch_commit_kv(T *ck, T *cv, const int32_t *prefix_len, const int32_t *path,
                            const int32_t *path_len, const int32_t *status, int L, int B,
                            int n1, int Hkv, int hd, int capacity, int32_t *new_len,
                            hipStream_t s) {
  if ((n1 - 1) * hd > MAXE) return hipErrorInvalidValue;
  hipLaunchKernelGGL(commit_kv_kernel<T>, dim3(L * Hkv, B), dim3(256), 0, s, ck, cv,
                     prefix_len, path, path_len, status, B, n1, Hkv, hd, capacity, new_len);
  return hipGetLastError();
}

template hipError_t launch_commit_kv<float>(float *, float *, const int32_t *, const int32_t *,
                                            const int32_t *, const int32_t *, int, int, int,
                                            int, int, int, int32_t *, hipStream_t);
template hipError_t launch_commit_kv<bf16>(bf16 *, bf16 *, const int32_t *, const int32_t *,
                                           const int32_t *, const int32_t *, int, int, int, int,
                                           int, int, int32_t *, hipStream_t);

hipError_t launch_transpose_planes(const void *src, void *dst, int elem_bytes, int planes,
                                   int rows, int cols, hipStream_t s) {
  if (planes < 1 || rows < 1 || cols < 1 || (elem_bytes != 2 && elem_bytes != 4))
    return hipErrorInvalidValue;
  const int tiles_r = (rows + 31) / 32, tiles_c = (cols + 31) / 32;
  const long long blocks = (long long)planes * tiles_r * tiles_c;
  if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
  if (elem_bytes == 2)
    hipLaunchKernelGGL(transpose_planes_kernel<uint16_t>, dim3((unsigned)blocks), dim3(256), 0, s,
                       (const uint16_t *)src, (uint16_t *)dst, rows, cols, tiles_r, tiles_c);
  else
    hipLaunchKernelGGL(transpose_planes_kernel<uint32_t>, dim3((unsigned)blocks), dim3(256), 0, s,
                       (const uint32_t *)src, (uint32_t *)dst, rows, cols, tiles_r, tiles_c);
  return hipGetLastError();
}

}  // namespace acespec
