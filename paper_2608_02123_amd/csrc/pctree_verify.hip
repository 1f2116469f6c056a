// Verification bookkeeping after a round (paper Sec. 4.2 and App. A, "Tensor
// implementation"): the padded root-to-leaf retrieve rows of the emitted
// tree, the greedy tree acceptance over those rows once the target has
// predicted a next token at every node, and the compaction of the accepted
// row's per-node cache entries right after the verified prefix.
//
// All three are small integer or gather steps, one workgroup per request
// (retrieve, accept) or a grid over cache columns (compact).  Every index
// that comes from memory is range-checked before it is used, so malformed
// inputs never read or write out of bounds.
#include "pctree.h"

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pctree_verify.h"

namespace pctree {
namespace {

constexpr int kVerifyThreads = 256;
constexpr int kMaxNodes = PCTREE_MAX_MASK_BUDGET;  // nodes one workgroup holds in LDS

// The parent of node i if it is an edge of the tree (an index in [0, i)),
// else -1: a malformed entry simply ends an upward walk.
__device__ __forceinline__ int edge_of(const int* par, int i) {
  const int p = par[i];
  return (p >= 0 && p < i) ? p : -1;
}

// Exclusive prefix sum of one value per thread over the workgroup, plus the
// total.  `sh` holds blockDim.x / 64 ints.
__device__ int block_exclusive_scan(int v, int* sh, int& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nwave = blockDim.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) sh[wave] = x;
  __syncthreads();
  int base = 0;
  total = 0;
  for (int w = 0; w < nwave; ++w) {
    const int s = sh[w];
    if (w < wave) base += s;
    total += s;
  }
  __syncthreads();
  return base + x - v;
}

// Retrieve rows: leaves are the selected nodes that are no selected node's
// parent; leaf q (in ascending node order) gets row q, the nodes from the
// head of its upward walk (the root, for a well-formed tree) down to the
// leaf, padded with -1 to W = max_depth + 1 entries.
__global__ __launch_bounds__(kVerifyThreads) void retrieve_kernel(const int* __restrict__ parent,
                                                                  const int* __restrict__ count,
                                                                  int N, int W,
                                                                  int* __restrict__ rows,
                                                                  int* __restrict__ nrows) {
  __shared__ int sh_par[kMaxNodes];
  __shared__ unsigned char sh_child[kMaxNodes];
  __shared__ int sh_scan[kVerifyThreads / 64];
  const int req = blockIdx.x;
  const int tid = threadIdx.x;
  const int c = min(max(count[req], 0), N);
  for (int i = tid; i < N; i += blockDim.x) {
    sh_par[i] = parent[(size_t)req * N + i];
    sh_child[i] = 0;
  }
  __syncthreads();
  for (int j = tid; j < c; j += blockDim.x) {
    const int p = edge_of(sh_par, j);
    if (p >= 0) sh_child[p] = 1;  // every writer stores the same value
  }
  __syncthreads();
  // each thread owns a contiguous run of nodes, so the leaf ranks follow node order
  const int per = (N + blockDim.x - 1) / blockDim.x;
  const int i0 = min(tid * per, N), i1 = min(i0 + per, N);
  int mine = 0;
  for (int i = i0; i < i1; ++i) mine += (i < c && !sh_child[i]) ? 1 : 0;
  int total = 0;
  int q = block_exclusive_scan(mine, sh_scan, total);
  int* out = rows + (size_t)req * N * W;
  for (int i = i0; i < i1; ++i) {
    if (i >= c || sh_child[i]) continue;
    int len = 1;
    for (int j = edge_of(sh_par, i); j >= 0; j = edge_of(sh_par, j)) ++len;
    // the walk visits nodes leaf first; node t steps above the leaf sits at
    // position len - 1 - t, and only positions below W are kept
    int* row = out + (size_t)q * W;
    int pos = len - 1;
    for (int j = i; j >= 0; j = edge_of(sh_par, j), --pos)
      if (pos < W) row[pos] = j;
    for (int m = len; m < W; ++m) row[m] = -1;
    ++q;
  }
  for (int e = total * W + tid; e < N * W; e += blockDim.x) out[e] = -1;
  if (tid == 0) nrows[req] = total;
}

// Greedy tree acceptance: along row j, position l >= 1 is accepted while its
// token equals the target's prediction at position l - 1; the row accepting
// the most positions wins, the lowest row on ties.
__global__ __launch_bounds__(kVerifyThreads) void accept_kernel(
    const int* __restrict__ token, const int* __restrict__ rows, const int* __restrict__ nrows,
    const int* __restrict__ target, int N, int W, int* __restrict__ accept_len,
    int* __restrict__ accept_row, int* __restrict__ accept_node, int* __restrict__ bonus) {
  __shared__ int sh_best[kVerifyThreads / 64];
  const int req = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = min(max(nrows[req], 0), N);
  const int* tok = token + (size_t)req * N;
  const int* tgt = target + (size_t)req * N;
  const int* rr = rows + (size_t)req * N * W;
  // key = accepted length above the inverted row index: the maximum is the
  // longest row, the lowest index among equals; -1 = no usable row
  int best = -1;
  for (int j = tid; j < n; j += blockDim.x) {
    const int* row = rr + (size_t)j * W;
    int prev = row[0];
    if (prev < 0 || prev >= N) continue;
    int a = 0;
    for (int l = 1; l < W; ++l) {
      const int v = row[l];
      if (v < 0 || v >= N || tok[v] != tgt[prev]) break;
      a = l;
      prev = v;
    }
    best = max(best, (a << 11) | (2047 - j));
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) best = max(best, __shfl_xor(best, o, 64));
  if (lane == 0) sh_best[wave] = best;
  __syncthreads();
  best = sh_best[0];
  for (int w = 1; w < (int)(blockDim.x >> 6); ++w) best = max(best, sh_best[w]);
  const int a = best < 0 ? 0 : best >> 11;
  const int j = best < 0 ? -1 : 2047 - (best & 2047);
  int* nodes = accept_node + (size_t)req * W;
  for (int m = tid; m < W; m += blockDim.x) nodes[m] = (j >= 0 && m <= a) ? rr[(size_t)j * W + m] : -1;
  if (tid == 0) {
    accept_len[req] = a;
    accept_row[req] = j;
    bonus[req] = j >= 0 ? tgt[rr[(size_t)j * W + a]] : -1;
  }
}

// Compaction: for request r with accepted nodes n_0 < n_1 < ... < n_a, the
// 16-byte column c of slot prefix + n_m moves to slot prefix + m in every
// group.  Because n_m >= m and the nodes increase, a slot is always read
// before any earlier step could overwrite it, so one thread per (group,
// column) copies in path order, in batches whose loads all issue before
// their stores.  A request whose accepted path is out of range or not
// increasing is left untouched.
constexpr int kCompactBatch = 8;

__global__ __launch_bounds__(kVerifyThreads) void compact_kernel(
    char* __restrict__ cache, long long request_stride, long long group_stride, int groups,
    int capacity, int chunks, const int* __restrict__ prefix_len,
    const int* __restrict__ accept_node, const int* __restrict__ accept_len, int N, int W) {
  const int req = blockIdx.y;
  const int a = accept_len[req];
  const int pre = prefix_len[req];
  if (a < 0 || a >= W || pre < 0) return;
  const int* nodes = accept_node + (size_t)req * W;
  // validate the path (uniform across the workgroup)
  int last = -1;
  for (int m = 0; m <= a; ++m) {
    const int v = nodes[m];
    if (v <= last || v >= N || pre + v >= capacity) return;
    last = v;
  }
  const long long col = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (col >= (long long)groups * chunks) return;
  const int g = (int)(col / chunks), c = (int)(col - (long long)g * chunks);
  char* base = cache + req * request_stride + g * group_stride + (long long)c * 16;
  const long long slot_bytes = (long long)chunks * 16;
  for (int m0 = 0; m0 <= a; m0 += kCompactBatch) {
    uint4 v[kCompactBatch];
#pragma unroll
    for (int b = 0; b < kCompactBatch; ++b) {
      const int m = m0 + b;
      if (m <= a && nodes[m] != m)
        v[b] = *(const uint4*)(base + (long long)(pre + nodes[m]) * slot_bytes);
    }
#pragma unroll
    for (int b = 0; b < kCompactBatch; ++b) {
      const int m = m0 + b;
      if (m <= a && nodes[m] != m) *(uint4*)(base + (long long)(pre + m) * slot_bytes) = v[b];
    }
  }
}

}  // namespace

hipError_t launch_retrieve(const int* parent, const int* count, int R, int N, int W, int* rows,
                           int* nrows, hipStream_t st) {
  hipLaunchKernelGGL(retrieve_kernel, dim3(R), dim3(kVerifyThreads), 0, st, parent, count, N, W,
                     rows, nrows);
  return hipGetLastError();
}

hipError_t launch_accept(const int* token, const int* rows, const int* nrows, const int* target,
                         int R, int N, int W, int* accept_len, int* accept_row, int* accept_node,
                         int* bonus, hipStream_t st) {
  hipLaunchKernelGGL(accept_kernel, dim3(R), dim3(kVerifyThreads), 0, st, token, rows, nrows,
                     target, N, W, accept_len, accept_row, accept_node, bonus);
  return hipGetLastError();
}

hipError_t launch_compact(void* cache, long long request_stride, long long group_stride,
                          int groups, int capacity, int slot_bytes, const int* prefix_len,
                          const int* accept_node, const int* accept_len, int R, int N, int W,
                          hipStream_t st) {
  const int chunks = slot_bytes / 16;
  const long long cols = (long long)groups * chunks;
  const unsigned gx = (unsigned)((cols + kVerifyThreads - 1) / kVerifyThreads);
  hipLaunchKernelGGL(compact_kernel, dim3(gx, R), dim3(kVerifyThreads), 0, st, (char*)cache,
                     request_stride, group_stride, groups, capacity, chunks, prefix_len,
                     accept_node, accept_len, N, W);
  return hipGetLastError();
}

}  // namespace pctree
