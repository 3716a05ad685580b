// The draft tree of one sequence from its ranked list (Sec. 3.5 reuse
// construction organised as a draft tree, Sec. 3.6), built by one wave.
// Used by the tree kernel and by the rerank's merge kernel when the step asks
// it to build the tree right after ranking.
//
// Lane i holds ranked entry r (i < cnt): its successor token M[r+1] opens a
// branch unless a lower lane already holds that token; ballots number the
// branches and keep the first W.  A wave prefix sum of the branch lengths
// gives each branch its node offset, so every node, its parent link and its
// ancestor bits are written without serial dependence.  Because every branch
// is a chain, the ancestor-or-self set of node u is the contiguous node range
// [start of u's branch, u], which is how the mask rows are filled.
#pragma once

#include "adapld_internal.h"
#include "device_utils.h"

namespace adapld {


// Called by every lane of one wave; s_start holds 2 * ADAPLD_MAX_TREE_NODES
// ints of LDS, 8-byte aligned, that only this wave uses (node u's branch
// start and source row as a pair).
__device__ __forceinline__ void build_tree_wave(const TreeOut& t, int b, int L_stride, int L, int r, int cnt,
                                                int* s_start) {
  const int lane = lane_id();
  const int32_t* __restrict__ M = t.tokens + (size_t)b * L_stride;
  int tok = -1;
  const bool valid = lane < cnt && r >= 0 && r <= L - 2;
  if (valid) tok = M[r + 1];
  // A lane is a new branch if no lower valid lane holds the same successor
  // token.  The tokens and validity of 8 lanes at a time are read as scalars
  // together (independent reads, not one dependent read per lane); lanes at
  // or past cnt are never valid.
  bool dup = false;
  for (int j0 = 0; j0 < cnt; j0 += 8) {
    int tj[8], vj[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      tj[i] = __builtin_amdgcn_readlane(tok, min(j0 + i, kWave - 1));
      vj[i] = __builtin_amdgcn_readlane((int)valid, min(j0 + i, kWave - 1));
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) dup |= (j0 + i < lane) && vj[i] && tj[i] == tok;
  }
  const bool opens = valid && !dup;
  const int branch = __popcll(__ballot(opens) & lanes_below());
  const bool keep = opens && branch < t.W;
  const int len = keep ? min(t.S + 1, L - 1 - r) : 0;

  // Exclusive prefix sum of branch lengths over lanes (branch order = lane order).
  const int incl = wave_incl_scan_i32(len);
  const int start = incl - len;
  const int T = __builtin_amdgcn_readlane(incl, kWave - 1);

  const size_t nb = (size_t)b * t.T_max;
  // Every node's branch start and source row go to LDS as one pair; the
  // nodes are then written 64 at a time across the lanes, with the token
  // loads of all of them in flight together (a lane walking its own branch
  // would wait for each token, and for its earlier stores, in turn).
  int2* s_pair = reinterpret_cast<int2*>(s_start);
  for (int dd = 0; dd < len; ++dd) s_pair[start + dd] = make_int2(start, r);
  if (lane == 0) t.node_count[b] = T;
  // The pairs are written and read by this wave only; its LDS
  // operations complete in order, so a wave-level fence is enough.
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  if (T > 0) {
    constexpr int kChunks = (ADAPLD_MAX_TREE_NODES + kWave - 1) / kWave;
    int tok_u[kChunks], src_u[kChunks], dd_u[kChunks];
#pragma unroll
    for (int c = 0; c < kChunks; ++c) {
      if (c * kWave >= T) break;                      // wave-uniform
      const int u = min(c * kWave + lane, T - 1);   // past T: a repeat of node T-1, not stored
      const int2 pr = s_pair[u];
      dd_u[c] = u - pr.x;
      src_u[c] = pr.y + 1 + dd_u[c];                 // <= L-1 by the branch length
      tok_u[c] = M[src_u[c]];
    }
#pragma unroll
    for (int c = 0; c < kChunks; ++c) {
      const int u = c * kWave + lane;
      if (u < T) {
        t.node_token[nb + u] = tok_u[c];
        t.node_parent[nb + u] = dd_u[c] == 0 ? -1 : u - 1;
        t.node_depth[nb + u] = dd_u[c];
        t.node_src[nb + u] = src_u[c];
      }
    }
  }

  const int nw = (t.T_max + 63) / 64;
  uint64_t* __restrict__ mrow = t.tree_mask + nb * nw;
  for (int idx = lane; idx < t.T_max * nw; idx += kWave) {
    const int u = idx / nw;
    const int w = idx - u * nw;
    uint64_t bits = 0;
    if (u < T) {
      const int lo = max(s_pair[u].x, 64 * w);
      const int hi = min(u, 64 * w + 63);  // inclusive
      if (lo <= hi) {
        const int n = hi - lo + 1;
        bits = (n == 64 ? ~0ull : ((1ull << n) - 1)) << (lo - 64 * w);
      }
    }
    mrow[idx] = bits;
  }
}

}  // namespace adapld
