// Internal launcher of the tree-masked verification attention
// (pctree_attention.hip), called by the C ABI after its argument checks.
// Not part of the public interface.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace pctree {

// Work split of one call, a pure function of the shape and the CU count.
struct AttnPlan {
  int qblocks;      // 64-row query blocks per (request, key/value head)
  int nsplit;       // key-slot runs per query block (1: no merge pass)
  int split_keys;   // slots per run, a multiple of 64
  int blocks;       // workgroups of the attention kernel (XCD-grouped, padded)
  size_t ws_bytes;  // workspace of the merge pass (0 when nsplit == 1)
};

struct AttnArgs {
  const uint16_t* q;      // [R][N][Hq][D] bf16
  const uint16_t* k;      // [R][Hkv][C][D] bf16
  const uint16_t* v;      // [R][Hkv][C][D] bf16
  const uint32_t* mask;   // [R][N][NW]
  const int* count;       // [R]
  const int* prefix_len;  // [R]
  uint16_t* out;          // [R][N][Hq][D] bf16
  float* part_o;          // [nsplit][R][N][Hq][D] (split runs only)
  float* part_ml;         // [nsplit][R][N][Hq][2] (max of q.k, sum of weights)
  int R, N, Hq, Hkv, C, NW, g;
  int qblocks, nsplit, split_keys;
  float scale_log2;       // softmax scale times log2(e), > 0
};

AttnPlan plan_attention(int R, int N, int Hq, int Hkv, int D, int C, int cus);

hipError_t launch_attention(AttnArgs a, int blocks, int D, hipStream_t stream);

}  // namespace pctree
