// Reuse construction (Sec. 3.5) organised as a draft tree (Sec. 3.6).
//
// One wave per sequence.  Lane i takes ranked entry i (k <= 64): its successor
// token M[r+1] opens a branch unless a lower lane already holds that token;
// ballots number the branches and keep the first W.  A wave prefix sum of the
// branch lengths gives each branch its node offset, so every node, its parent
// link and its ancestor bits are written without serial dependence.  Because
// every branch is a chain, the ancestor-or-self set of node u is the
// contiguous node range [start of u's branch, u], which is how the mask rows
// are filled.
#include "adapld_internal.h"
#include "device_utils.h"

namespace adapld {
namespace {

__global__ __launch_bounds__(kWave) void build_draft_tree_kernel(
    const int32_t* __restrict__ tokens, const int32_t* __restrict__ lens,
    const int32_t* __restrict__ topk_pos, const int32_t* __restrict__ topk_count,
    const int32_t* __restrict__ kind, int L_stride, int k, int W, int S, int T_max,
    int32_t* __restrict__ node_token, int32_t* __restrict__ node_parent,
    int32_t* __restrict__ node_depth, int32_t* __restrict__ node_src,
    int32_t* __restrict__ node_count, uint64_t* __restrict__ tree_mask) {
  __shared__ int s_start[ADAPLD_MAX_TREE_NODES];
  const int b = blockIdx.x;
  const int lane = lane_id();
  const int L = min(max(lens[b], 0), L_stride);
  const int32_t* __restrict__ M = tokens + (size_t)b * L_stride;
  // The counts and the ranked positions are independent loads (entries past the
  // count are read but not used).
  int cnt = min(max(topk_count[b], 0), k);
  const int kd = kind[b];
  int r = lane < k ? topk_pos[(size_t)b * k + lane] : -1;
  if (kd == ADAPLD_KIND_NONE) cnt = 0;

  int tok = -1;
  const bool valid = lane < cnt && r >= 0 && r <= L - 2;
  if (valid) tok = M[r + 1];
  // A lane is a new branch if no lower valid lane holds the same successor token.
  bool dup = false;
  for (int j = 0; j < cnt; ++j) {   // lane j's token and validity as scalars
    const int tj = __builtin_amdgcn_readlane(tok, j);
    const int vj = __builtin_amdgcn_readlane((int)valid, j);
    dup |= (j < lane) && vj && tj == tok;
  }
  const bool opens = valid && !dup;
  const int branch = __popcll(__ballot(opens) & lanes_below());
  const bool keep = opens && branch < W;
  const int len = keep ? min(S + 1, L - 1 - r) : 0;

  // Exclusive prefix sum of branch lengths over lanes (branch order = lane order).
  const int incl = wave_incl_scan_i32(len);
  const int start = incl - len;
  const int T = __builtin_amdgcn_readlane(incl, kWave - 1);

  const size_t nb = (size_t)b * T_max;
  for (int dd = 0; dd < len; ++dd) {
    const int u = start + dd;
    node_token[nb + u] = M[r + 1 + dd];
    node_parent[nb + u] = dd == 0 ? -1 : u - 1;
    node_depth[nb + u] = dd;
    node_src[nb + u] = r + 1 + dd;
    s_start[u] = start;
  }
  if (lane == 0) node_count[b] = T;
  __syncthreads();

  const int nw = (T_max + 63) / 64;
  uint64_t* __restrict__ mrow = tree_mask + nb * nw;
  for (int idx = lane; idx < T_max * nw; idx += kWave) {
    const int u = idx / nw;
    const int w = idx - u * nw;
    uint64_t bits = 0;
    if (u < T) {
      const int lo = max(s_start[u], 64 * w);
      const int hi = min(u, 64 * w + 63);  // inclusive
      if (lo <= hi) {
        const int n = hi - lo + 1;
        bits = (n == 64 ? ~0ull : ((1ull << n) - 1)) << (lo - 64 * w);
      }
    }
    mrow[idx] = bits;
  }
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
