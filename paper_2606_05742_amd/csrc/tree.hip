// Reuse construction (Sec. 3.5) organised as a draft tree (Sec. 3.6): one
// wave per sequence reads its ranked list and builds the tree (the shared
// wave routine in tree_device.h).
#include "adapld_internal.h"
#include "device_utils.h"
#include "tree_device.h"

namespace adapld {
namespace {

__global__ __launch_bounds__(kWave) void build_draft_tree_kernel(
    const int32_t* __restrict__ tokens, const int32_t* __restrict__ lens,
    const int32_t* __restrict__ topk_pos, const int32_t* __restrict__ topk_count,
    const int32_t* __restrict__ kind, int L_stride, int k, int W, int S, int T_max,
    int32_t* __restrict__ node_token, int32_t* __restrict__ node_parent,
    int32_t* __restrict__ node_depth, int32_t* __restrict__ node_src,
    int32_t* __restrict__ node_count, uint64_t* __restrict__ tree_mask) {
  __shared__ __attribute__((aligned(8))) int s_start[2 * ADAPLD_MAX_TREE_NODES];
  const int b = blockIdx.x;
  const int lane = lane_id();
  const int L = min(max(lens[b], 0), L_stride);
  // The counts and the ranked positions are independent loads (entries past the
  // count are read but not used).
  int cnt = min(max(topk_count[b], 0), k);
  const int kd = kind[b];
  int r = lane < k ? topk_pos[(size_t)b * k + lane] : -1;
  if (kd == ADAPLD_KIND_NONE) cnt = 0;

  const TreeOut t{tokens, W, S, T_max, node_token, node_parent, node_depth, node_src, node_count, tree_mask};
  build_tree_wave(t, b, L_stride, L, r, cnt, s_start);
}

}  // namespace

hipError_t launch_build_draft_tree(const int32_t* tokens, const int32_t* lens,
                                   const int32_t* topk_pos, const int32_t* topk_count,
                                   const int32_t* kind, int B, int L_stride, int k, int W, int S,
                                   int T_max, int32_t* node_token, int32_t* node_parent,
                                   int32_t* node_depth, int32_t* node_src, int32_t* node_count,
                                   uint64_t* tree_mask, hipStream_t stream) {
  hipLaunchKernelGGL(build_draft_tree_kernel, dim3(B), dim3(kWave), 0, stream, tokens, lens,
                     topk_pos, topk_count, kind, L_stride, k, W, S, T_max, node_token, node_parent,
                     node_depth, node_src, node_count, tree_mask);
  return hipGetLastError();
}

}  // namespace adapld
