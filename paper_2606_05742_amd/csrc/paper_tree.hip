// The paper's draft construction (Sec. 3.5, Algorithm 1): the main copy path
// of a lexical anchor, branch tokens from the target's top tokens after the
// anchor, and one successor per branch (the token after the occurrence of
// the branch token whose preceding hidden state is closest to the anchor's).
//
// setup kernel: one workgroup per sequence.  One wave takes the anchor j*
// (the top of the ranked list), reads the W top tokens after it from the
// caller's per-position table and keeps the distinct valid ones (without the
// main path's first token on a lexical hit).  Then every thread scans part
// of the context once for all branch tokens together: each occurrence t in
// [1, L-2] of branch token i appends row t-1 to candidate list (b, i).  The
// W lists of a sequence share one query, the anchor's hidden state H[j*],
// copied once per sequence.
//
// successor backoff (with an embedding table): a branch token that never
// occurs in [1, L-2] takes instead the positions whose token embedding has
// cosine >= tau with its own (Sec. 3.5 applies the lexical-first backoff of
// Sec. 3.3 to the successor query), from the embedding fallback's kernels
// run over the B*W lists.
//
// Successors are drafted for every branch (the text of Sec. 3.5) or only
// after a semantic anchor (Algorithm 1's strict branch drafts none),
// selected by succ_mode.
//
// rerank: the hidden-state scan and merge with k = 1 over the B*W lists (a
// list reads the bank rows and the query of its sequence), so the argmax of
// cos(H[t-1], H[j*]) costs one pass over the candidate rows of all branches
// of all sequences, spread over the whole GPU.
//
// assembly kernel: one wave per sequence writes the main path as a chain,
// then each branch token followed by its successor, and the ancestor-or-self
// mask rows.
#include "adapld_internal.h"
#include "device_utils.h"

namespace adapld {
namespace {

constexpr int kSetupThreads = 256;

struct PaperTreeArgs {
  const int32_t* tokens;
  const int32_t* lens;
  const uint16_t* bank;
  const int32_t* topk_pos;
  const int32_t* topk_count;
  const int32_t* kind;
  const int32_t* top_tokens;   // [B][L_stride][W]
  int k, W, S, B, L_stride, d, T_max;
  int succ_mode;               // ADAPLD_SUCC_*
  // workspace
  int32_t* btok;     // [B][W] branch tokens
  int32_t* nbr;      // [B]    number of branches
  int32_t* vcand;    // [B*W][L_stride] candidate rows t-1
  int32_t* vcount;   // [B*W]
  int32_t* vlens;    // [B*W]  the sequence's L
  uint16_t* vquery;  // [B][d]   H[j*], the query of the sequence's W lists
  int32_t* vpos;     // [B*W]  the winning row (k = 1)
  float* vscore;
  int32_t* vcnt;     // [B*W]  1 if the branch has a successor
  int32_t* vkind;
  int32_t* vskip;    // [B*W]  nonzero: no embedding backoff for the list
  // outputs
  int32_t* node_token;
  int32_t* node_parent;
  int32_t* node_depth;
  int32_t* node_src;
  int32_t* node_count;
  uint64_t* tree_mask;
};

// The anchor of sequence b, or -1 when there is no tree (no retrieval, or an
// anchor without a following token).
__device__ __forceinline__ int anchor_of(const PaperTreeArgs& a, int b, int L, int& kd) {
  kd = a.kind[b];
  const int cnt = a.topk_count[b];
  const int j0 = a.topk_pos[(size_t)b * a.k];   // in bounds for every b: read without waiting for cnt
  const int j = cnt > 0 && kd != ADAPLD_KIND_NONE ? j0 : -1;
  return j >= 0 && j <= L - 2 ? j : -1;
}

// Tokens a setup thread holds per pass: kSetupVec 16-byte loads, coalesced
// across the workgroup (thread x loads int4 number i*kSetupThreads + x).
constexpr int kSetupVec = 8;
constexpr int kSetupPass = kSetupThreads * kSetupVec * 4;
constexpr int kQueryVec = (ADAPLD_MAX_HIDDEN / 8 + kSetupThreads - 1) / kSetupThreads;

__global__ __launch_bounds__(kSetupThreads) void paper_tree_setup_kernel(const PaperTreeArgs a) {
  __shared__ int s_tok[kWave];
  __shared__ int s_cnt[kWave];
  __shared__ int s_nb;
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int L = min(max(a.lens[b], 0), a.L_stride);
  const int32_t* __restrict__ M = a.tokens + (size_t)b * a.L_stride;
  // The first pass's tokens are requested before the anchor and L are known:
  // every load stays inside the row (L_stride tokens) and positions at or
  // beyond L are masked afterwards.  A whole pass over a 16-byte-aligned row
  // loads int4s; any other pass loads single tokens at clamped positions.
  // Both forms are branch-free so that all loads of a pass are in flight
  // together.
  const bool vec = (reinterpret_cast<uintptr_t>(M) & 15) == 0;
  int4 cur[kSetupVec];
  auto load_pass = [&](int base) {
    if (vec && base + kSetupPass <= a.L_stride) {
#pragma unroll
      for (int i = 0; i < kSetupVec; ++i)
        cur[i] = *reinterpret_cast<const int4*>(M + base + 4 * (i * kSetupThreads + tid));
    } else {
      const int last = a.L_stride - 1;
#pragma unroll
      for (int i = 0; i < kSetupVec; ++i) {
        const int t0 = base + 4 * (i * kSetupThreads + tid);
        cur[i].x = M[min(t0, last)];
        cur[i].y = M[min(t0 + 1, last)];
        cur[i].z = M[min(t0 + 2, last)];
        cur[i].w = M[min(t0 + 3, last)];
      }
    }
  };
  load_pass(0);
  int kd;
  const int j = anchor_of(a, b, L, kd);
  // The anchor's hidden state, the query of all its branch lists, copied
  // while the branch tokens are chosen (d/8 <= kSetupThreads * kQueryVec
  // 16-byte chunks; row max(j, 0) and clamped chunks keep the loads in
  // bounds and branch-free).
  {
    const int chunks = a.d / 8;
    const uint4* __restrict__ src =
        reinterpret_cast<const uint4*>(a.bank + ((size_t)b * a.L_stride + max(j, 0)) * a.d);
    uint4* __restrict__ dst = reinterpret_cast<uint4*>(a.vquery + (size_t)b * a.d);
    // (four named registers: an array here would be placed in LDS)
    static_assert(kQueryVec == 4, "query chunks per thread");
    const uint4 q0 = src[min(tid, chunks - 1)];
    const uint4 q1 = src[min(tid + kSetupThreads, chunks - 1)];
    const uint4 q2 = src[min(tid + 2 * kSetupThreads, chunks - 1)];
    const uint4 q3 = src[min(tid + 3 * kSetupThreads, chunks - 1)];
    if (j >= 0) {
      if (tid < chunks) dst[tid] = q0;
      if (tid + kSetupThreads < chunks) dst[tid + kSetupThreads] = q1;
      if (tid + 2 * kSetupThreads < chunks) dst[tid + 2 * kSetupThreads] = q2;
      if (tid + 3 * kSetupThreads < chunks) dst[tid + 3 * kSetupThreads] = q3;
    }
  }
  if (tid < kWave) {
    // Branch tokens: the valid, distinct top tokens after the anchor, in order.
    int tok = -1;
    if (j >= 0 && lane < a.W) tok = a.top_tokens[((size_t)b * a.L_stride + j) * a.W + lane];
    const int first = j >= 0 && kd == ADAPLD_KIND_LEX ? M[j + 1] : -1;
    bool ok = tok >= 0 && tok != first;
    for (int i = 0; i < a.W; ++i) {   // a lower lane holding the same token wins
      const int ti = __builtin_amdgcn_readlane(tok, i);
      ok = ok && !(i < lane && ti == tok);
    }
    const uint64_t keep = __ballot(ok);
    const int idx = __popcll(keep & lanes_below());
    if (ok) s_tok[idx] = tok;
    if (lane < a.W) s_cnt[lane] = 0;
    if (lane == 0) {
      s_nb = __popcll(keep);
      a.nbr[b] = __popcll(keep);
    }
  }
  __syncthreads();
  const int nb = s_nb;
  // Algorithm 1 drafts no successor after a lexical anchor.
  const bool drafts = j >= 0 && (a.succ_mode == ADAPLD_SUCC_EVERY_BRANCH || kd == ADAPLD_KIND_SEM);
  const int nscan = drafts ? nb : 0;
  // One pass over the context for all branch tokens: occurrence t (with a
  // preceding hidden state and a following token, t in [1, L-2]) of branch i
  // adds row t-1 to list i.  Per branch a thread compares its tokens in
  // registers into a 32-bit mask, takes that many slots and writes the rows.
  // List order is arbitrary: the rerank breaks ties by position.
  for (int base = 0; nscan > 0 && base < L; base += kSetupPass) {
    if (base > 0) load_pass(base);
    uint32_t valid = 0;   // bit 4i+e: token e of load i is an occurrence position
#pragma unroll
    for (int i = 0; i < kSetupVec; ++i) {
      const int t0 = base + 4 * (i * kSetupThreads + tid);
#pragma unroll
      for (int e = 0; e < 4; ++e) valid |= (t0 + e >= 1 && t0 + e <= L - 2 ? 1u : 0u) << (4 * i + e);
    }
    for (int br = 0; br < nscan; ++br) {
      const int c = s_tok[br];
      uint32_t hit = 0;
#pragma unroll
      for (int i = 0; i < kSetupVec; ++i) {
        hit |= (cur[i].x == c ? 1u : 0u) << (4 * i);
        hit |= (cur[i].y == c ? 1u : 0u) << (4 * i + 1);
        hit |= (cur[i].z == c ? 1u : 0u) << (4 * i + 2);
        hit |= (cur[i].w == c ? 1u : 0u) << (4 * i + 3);
      }
      hit &= valid;
      // Slots: a prefix sum of the hit counts over the wave and one LDS
      // atomic per wave (a per-lane atomic with per-lane operands costs a
      // loop over the active lanes).
      const int n = __popc(hit);
      const int incl = wave_incl_scan_i32(n);
      const int total = __builtin_amdgcn_readlane(incl, kWave - 1);
      if (total > 0) {
        int first = 0;
        if (lane == kWave - 1) first = atomicAdd(&s_cnt[br], total);
        int slot = __builtin_amdgcn_readlane(first, kWave - 1) + incl - n;
        int32_t* __restrict__ dst = a.vcand + ((size_t)b * a.W + br) * a.L_stride;
        while (hit) {
          const int bit = __builtin_ctz(hit);
          hit &= hit - 1;
          const int t = base + 4 * ((bit >> 2) * kSetupThreads + tid) + (bit & 3);
          dst[slot++] = t - 1;
        }
      }
    }
  }
  __syncthreads();
  if (tid < a.W) {
    const size_t v = (size_t)b * a.W + tid;
    const int cnt = tid < nscan ? s_cnt[tid] : 0;
    a.vcount[v] = cnt;
    a.vlens[v] = L;
    a.vskip[v] = tid < nscan && cnt == 0 ? 0 : 1;   // a drafted branch token with no occurrence
    a.btok[v] = tid < nb ? s_tok[tid] : -1;
  }
}

__global__ __launch_bounds__(kWave) void paper_tree_assemble_kernel(const PaperTreeArgs a) {
  __shared__ int s_par[ADAPLD_MAX_TREE_NODES];
  const int b = blockIdx.x;
  const int lane = lane_id();
  const int L = min(max(a.lens[b], 0), a.L_stride);
  const int32_t* __restrict__ M = a.tokens + (size_t)b * a.L_stride;
  int kd;
  const int j = anchor_of(a, b, L, kd);
  const int ell = j >= 0 && kd == ADAPLD_KIND_LEX ? min(a.S + 1, L - 1 - j) : 0;   // main path length
  const int nb = j >= 0 ? a.nbr[b] : 0;
  const size_t nbase = (size_t)b * a.T_max;

  // Branch i (lane i) takes 1 + has_successor nodes after the main path.
  const size_t v = (size_t)b * a.W + lane;
  const bool is_br = lane < nb;
  const bool has = is_br && a.vcnt[v] > 0;
  const int size = is_br ? 1 + (has ? 1 : 0) : 0;
  const int incl = wave_incl_scan_i32(size);
  const int start = ell + incl - size;
  const int T = ell + __builtin_amdgcn_readlane(incl, kWave - 1);

  for (int dd = lane; dd < ell; dd += kWave) {
    a.node_token[nbase + dd] = M[j + 1 + dd];
    s_par[dd] = dd == 0 ? -1 : dd - 1;
    a.node_parent[nbase + dd] = dd == 0 ? -1 : dd - 1;
    a.node_depth[nbase + dd] = dd;
    a.node_src[nbase + dd] = j + 1 + dd;
  }
  if (is_br) {
    a.node_token[nbase + start] = a.btok[v];
    s_par[start] = -1;
    a.node_parent[nbase + start] = -1;
    a.node_depth[nbase + start] = 0;
    a.node_src[nbase + start] = -1;
    if (has) {
      const int t = a.vpos[v] + 1;   // the winning occurrence; its row was t-1
      a.node_token[nbase + start + 1] = M[t + 1];
      s_par[start + 1] = start;
      a.node_parent[nbase + start + 1] = start;
      a.node_depth[nbase + start + 1] = 1;
      a.node_src[nbase + start + 1] = t + 1;
    }
  }
  if (lane == 0) a.node_count[b] = T;
  __syncthreads();   // s_par complete

  // Mask rows: a main node sees the chain up to itself, a branch node itself,
  // a successor itself and its branch node.
  const int nw = (a.T_max + 63) / 64;
  uint64_t* __restrict__ mrow = a.tree_mask + nbase * nw;
  for (int idx = lane; idx < a.T_max * nw; idx += kWave) {
    const int u = idx / nw;
    const int w = idx - u * nw;
    int lo = u, hi = u;   // inclusive node range of the ancestors-or-self
    if (u >= T) {
      lo = 1, hi = 0;     // empty
    } else if (u < ell) {
      lo = 0;
    } else {
      const int pu = s_par[u];   // a successor's parent is the node before it
      if (pu >= 0) lo = pu;
    }
    uint64_t bits = 0;
    const int l2 = max(lo, 64 * w), h2 = min(hi, 64 * w + 63);
    if (l2 <= h2) {
      const int n = h2 - l2 + 1;
      bits = (n == 64 ? ~0ull : ((1ull << n) - 1)) << (l2 - 64 * w);
    }
    mrow[idx] = bits;
  }
}

}  // namespace

size_t paper_tree_ws_bytes(int B, int L_stride, int W, int d) {
  const size_t V = (size_t)B * W;
  size_t n = 0;
  n += V * 4 + (size_t)B * 4;            // btok, nbr
  n += V * L_stride * 4;                 // vcand
  n += V * 4 * 3;                        // vcount, vlens, vskip
  n = (n + 15) / 16 * 16;
  n += (size_t)B * d * 2;                // vquery
  n += V * 4 * 4;                        // vpos, vscore, vcnt, vkind
  n = (n + 15) / 16 * 16;
  n += V * scan_lists(L_stride) * 8;     // the rerank's lists (k = 1)
  n = (n + 15) / 16 * 16;
  n += embed_flag_bytes((int)V, L_stride);   // the successor backoff's flags
  return n;
}

hipError_t launch_build_draft_tree_paper(const int32_t* tokens, const int32_t* lens, const uint16_t* bank, int d,
                                         const int32_t* topk_pos, const int32_t* topk_count, const int32_t* kind,
                                         int k, const int32_t* top_tokens, int W, int S, int succ_mode,
                                         const uint16_t* emb, int V_emb, float tau, int B, int L_stride,
                                         int T_max, int32_t* node_token, int32_t* node_parent, int32_t* node_depth,
                                         int32_t* node_src, int32_t* node_count, uint64_t* tree_mask, void* ws,
                                         hipStream_t stream) {
  PaperTreeArgs a{};
  a.tokens = tokens; a.lens = lens; a.bank = bank; a.topk_pos = topk_pos; a.topk_count = topk_count;
  a.kind = kind; a.top_tokens = top_tokens;
  a.k = k; a.W = W; a.S = S; a.B = B; a.L_stride = L_stride; a.d = d; a.T_max = T_max;
  a.succ_mode = succ_mode;
  const size_t V = (size_t)B * W;
  char* p = static_cast<char*>(ws);
  size_t off = 0;
  a.btok = reinterpret_cast<int32_t*>(p + off); off += V * 4;
  a.nbr = reinterpret_cast<int32_t*>(p + off); off += (size_t)B * 4;
  a.vcand = reinterpret_cast<int32_t*>(p + off); off += V * L_stride * 4;
  a.vcount = reinterpret_cast<int32_t*>(p + off); off += V * 4;
  a.vlens = reinterpret_cast<int32_t*>(p + off); off += V * 4;
  a.vskip = reinterpret_cast<int32_t*>(p + off); off += V * 4;
  off = (off + 15) / 16 * 16;
  a.vquery = reinterpret_cast<uint16_t*>(p + off); off += (size_t)B * d * 2;
  a.vpos = reinterpret_cast<int32_t*>(p + off); off += V * 4;
  a.vscore = reinterpret_cast<float*>(p + off); off += V * 4;
  a.vcnt = reinterpret_cast<int32_t*>(p + off); off += V * 4;
  a.vkind = reinterpret_cast<int32_t*>(p + off); off += V * 4;
  off = (off + 15) / 16 * 16;
  uint64_t* keys = reinterpret_cast<uint64_t*>(p + off); off += V * scan_lists(L_stride) * 8;
  off = (off + 15) / 16 * 16;
  uint8_t* flags = reinterpret_cast<uint8_t*>(p + off);
  a.node_token = node_token; a.node_parent = node_parent; a.node_depth = node_depth; a.node_src = node_src;
  a.node_count = node_count; a.tree_mask = tree_mask;

  hipLaunchKernelGGL(paper_tree_setup_kernel, dim3(B), dim3(kSetupThreads), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (emb) {
    e = launch_successor_embed(tokens, lens, emb, V_emb, B, W, L_stride, d, tau, a.vskip, a.btok, flags, a.vcand,
                               a.vcount, stream);
    if (e != hipSuccess) return e;
  }
  e = launch_semantic_topk(bank, a.vquery, a.vlens, a.vcand, a.vcount, (int)V, L_stride, d, 1, NAN, a.vpos,
                           a.vscore, a.vcnt, a.vkind, keys, nullptr, 1, stream, W);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(paper_tree_assemble_kernel, dim3(B), dim3(kWave), 0, stream, a);
  return hipGetLastError();
}

}  // namespace adapld
