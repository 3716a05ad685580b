// Greedy acceptance of the draft tree (Sec. 3.6: verification follows the
// standard speculative-decoding rule, which with greedy decoding keeps a draft
// token when it equals the target's own choice, Appendix C) and compaction of
// the accepted nodes' K/V into the cache.
//
// One workgroup of 256 threads per sequence, thread u for node u (T_max is at
// most 256).  Node u matches when its token equals the target's next token
// after its parent (after the context for a depth-0 node); four ballots give
// the match bitset, and u is accepted when its ancestor-or-self row of the
// tree mask lies inside that bitset, so no thread walks a path.  The deepest
// accepted node (the lowest index among equally deep ones) is a workgroup max
// of the key depth:~u, and its mask row is the accepted path: node v of the
// row goes to path slot node_depth[v].  Then all threads copy the path's K
// and V rows, 16 bytes at a time, to cache positions L, L+1, ... of every kv
// head.
#include "adapld_internal.h"
#include "device_utils.h"

namespace adapld {
namespace {

constexpr int kAcceptThreads = 256;
static_assert(kAcceptThreads >= ADAPLD_MAX_TREE_NODES, "one thread per node");
constexpr int kMaskWordsMax = (ADAPLD_MAX_TREE_NODES + 63) / 64;
constexpr int kRowChunks = ADAPLD_HEAD_DIM * 2 / 16;   // 16-byte pieces of one K or V row

struct AcceptArgs {
  const int32_t* node_token;
  const int32_t* node_parent;
  const int32_t* node_depth;
  const int32_t* node_count;
  const uint64_t* tree_mask;
  const int32_t* target_next;
  const int32_t* lens;
  const uint16_t* k_tree;
  const uint16_t* v_tree;
  int L_stride, T_max, Hkv;
  int32_t* accept_len;
  int32_t* accept_nodes;
  int32_t* out_tokens;
  uint16_t* k_ctx;
  uint16_t* v_ctx;
};

__global__ __launch_bounds__(kAcceptThreads) void accept_greedy_kernel(const AcceptArgs a) {
  __shared__ uint64_t s_match[kMaskWordsMax];
  __shared__ uint64_t s_row[kMaskWordsMax];   // the accepted path's mask row
  __shared__ int s_best[kAcceptThreads / kWave];
  __shared__ int s_path[ADAPLD_MAX_TREE_NODES];

  const int b = blockIdx.x;
  const int u = threadIdx.x;
  const int lane = lane_id();
  const int wave = u / kWave;
  const int T_max = a.T_max;
  const int nw = (T_max + 63) / 64;
  const int T = min(max(a.node_count[b], 0), T_max);
  const size_t nb = (size_t)b * T_max;
  const int32_t* __restrict__ next = a.target_next + (size_t)b * (T_max + 1);

  // Match bit of node u: its token against the target's token after its parent.
  // Every field of the node, its mask row included, is loaded at once and
  // before node_count is known (rows below T_max are in bounds), so the loads
  // share one memory round trip.
  bool match = false;
  int depth = 0;
  uint64_t myrow[kMaskWordsMax];
#pragma unroll
  for (int w = 0; w < kMaskWordsMax; ++w)
    myrow[w] = (u < T_max && w < nw) ? a.tree_mask[(nb + u) * nw + w] : 0ull;
  if (u < T_max) {
    const int p = a.node_parent[nb + u];
    const int tok = a.node_token[nb + u];
    const int dep = a.node_depth[nb + u];
    const int want = p < 0 ? next[0] : (p < T_max ? next[1 + p] : INT32_MIN);
    match = u < T && tok == want;
    depth = min(max(dep, 0), T_max - 1);
  }
  if (u >= T) {
#pragma unroll
    for (int w = 0; w < kMaskWordsMax; ++w) myrow[w] = 0ull;
  }
  if (u < ADAPLD_MAX_TREE_NODES) s_path[u] = -1;
  const uint64_t bits = __ballot(match);
  if (lane == 0 && wave < kMaskWordsMax) s_match[wave] = bits;
  __syncthreads();

  // Accepted: every ancestor-or-self bit is a match bit.  Key: deeper first,
  // then the lower node index.
  int key = -1;
  if (u < T) {
    bool ok = true;
#pragma unroll
    for (int w = 0; w < kMaskWordsMax; ++w) ok &= w >= nw || (myrow[w] & ~s_match[w]) == 0;
    if (ok) key = (depth << 9) | (ADAPLD_MAX_TREE_NODES - 1 - u);
  }
  key = wave_max_i32(key);
  if (lane == 0) s_best[wave] = key;
  __syncthreads();
  int best_key = -1;
#pragma unroll
  for (int w = 0; w < kAcceptThreads / kWave; ++w) best_key = max(best_key, s_best[w]);
  const int best = best_key < 0 ? -1 : ADAPLD_MAX_TREE_NODES - 1 - (best_key & 511);

  // The path: the best node's ancestor-or-self row (handed over by its
  // thread), placed by depth.
  int n_acc = 0;
  if (best >= 0) {
    if (u == best) {
#pragma unroll
      for (int w = 0; w < kMaskWordsMax; ++w) s_row[w] = myrow[w];
    }
    __syncthreads();
    for (int w = 0; w < nw; ++w) n_acc += __popcll(s_row[w]);
    if (u < T && ((s_row[u >> 6] >> (u & 63)) & 1ull) && depth < n_acc) s_path[depth] = u;
  }
  __syncthreads();

  const int L = min(max(a.lens[b], 0), a.L_stride);
  int32_t* __restrict__ ot = a.out_tokens + (size_t)b * (T_max + 1);
  if (u < n_acc) {
    const int v = s_path[u];
    a.accept_nodes[nb + u] = v;
    ot[u] = v >= 0 ? a.node_token[nb + v] : -1;
  }
  if (u == 0) {
    ot[n_acc] = best >= 0 ? next[1 + best] : next[0];   // the bonus token
    a.accept_len[b] = n_acc;
  }

  // KV compaction: path slot i goes to cache position L + i, inside the capacity.
  if (!a.k_ctx) return;
  const int n_copy = min(n_acc, a.L_stride - L);
  const int per_row = a.Hkv * kRowChunks;
  for (int idx = u; idx < n_copy * per_row; idx += kAcceptThreads) {
    const int i = idx / per_row;
    const int rem = idx - i * per_row;
    const int g = rem / kRowChunks;
    const int c = rem - g * kRowChunks;
    const int v = s_path[i];
    if (v < 0) continue;
    const size_t src = ((nb + v) * a.Hkv + g) * ADAPLD_HEAD_DIM + 8 * c;
    const size_t dst = (((size_t)b * a.Hkv + g) * a.L_stride + L + i) * ADAPLD_HEAD_DIM + 8 * c;
    *reinterpret_cast<uint4*>(a.k_ctx + dst) = *reinterpret_cast<const uint4*>(a.k_tree + src);
    *reinterpret_cast<uint4*>(a.v_ctx + dst) = *reinterpret_cast<const uint4*>(a.v_tree + src);
  }
}

}  // namespace

hipError_t launch_accept_greedy(const int32_t* node_token, const int32_t* node_parent,
                                const int32_t* node_depth, const int32_t* node_count,
                                const uint64_t* tree_mask, const int32_t* target_next,
                                const int32_t* lens, const uint16_t* k_tree, const uint16_t* v_tree,
                                int B, int L_stride, int T_max, int Hkv, int32_t* accept_len,
                                int32_t* accept_nodes, int32_t* out_tokens, uint16_t* k_ctx,
                                uint16_t* v_ctx, hipStream_t stream) {
  AcceptArgs a{};
  a.node_token = node_token; a.node_parent = node_parent; a.node_depth = node_depth;
  a.node_count = node_count; a.tree_mask = tree_mask; a.target_next = target_next; a.lens = lens;
  a.k_tree = k_tree; a.v_tree = v_tree;
  a.L_stride = L_stride; a.T_max = T_max; a.Hkv = Hkv;
  a.accept_len = accept_len; a.accept_nodes = accept_nodes; a.out_tokens = out_tokens;
  a.k_ctx = k_ctx; a.v_ctx = v_ctx;
  hipLaunchKernelGGL(accept_greedy_kernel, dim3(B), dim3(kAcceptThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace adapld
