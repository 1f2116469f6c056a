// Internal launchers of the verification kernels (pctree_verify.hip), called
// by the C ABI after its argument checks.  Not part of the public interface.
#pragma once

#include <hip/hip_runtime.h>

namespace pctree {

hipError_t launch_retrieve(const int* parent, const int* count, int R, int N, int W, int* rows,
                           int* nrows, hipStream_t stream);

hipError_t launch_accept(const int* token, const int* rows, const int* nrows, const int* target,
                         int R, int N, int W, int* accept_len, int* accept_row, int* accept_node,
                         int* bonus, hipStream_t stream);

hipError_t launch_compact(void* cache, long long request_stride, long long group_stride,
                          int groups, int capacity, int slot_bytes, const int* prefix_len,
                          const int* accept_node, const int* accept_len, int R, int N, int W,
                          hipStream_t stream);

}  // namespace pctree
