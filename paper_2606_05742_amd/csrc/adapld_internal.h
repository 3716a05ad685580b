// Internal declarations shared by the kernels and the C-ABI glue of libadapld.
// Device code targets gfx950 (CDNA4): wave64, MFMA bf16, 160 KiB LDS per CU.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include "adapld.h"

namespace adapld {

// ---------------------------------------------------------------- launch plans
// Host-side shape decisions shared by the workspace query and the launchers,
// so that both always agree.

// Semantic scan: the scored rows of all sequences, laid end to end, are cut
// into kScanWaveSlots equal ranges, one per wave (kScanWaves per workgroup).
// A wave writes one top-k list per sequence its range meets, so a sequence
// has at most min(kScanWaveSlots, its row count) lists.  The workgroup keeps
// the row offset, length and candidate count of up to kMaxScanSeqs sequences
// in LDS.
constexpr int kScanWaves = 4;
constexpr int kScanWaveSlots = 1024;
constexpr int kMaxScanSeqs = 2048;

inline int scan_lists(int L_stride) { return L_stride < kScanWaveSlots ? L_stride : kScanWaveSlots; }

// Verify attention: keys are processed in tiles of kKeyTile; query rows
// (node u, head-in-group) are stacked per kv head, 32 rows per MFMA block.
constexpr int kKeyTile = 64;

struct VerifyPlan {
  int G;           // query heads per kv head
  int rows_max;    // T_max * G stacked query rows per (sequence, kv head)
  int nb;          // 32-row blocks per wave
  int waves;       // waves per workgroup
  int kh;          // waves sharing one row block (1, or 2: each takes half of every tile)
  int rows_per_wg;
  int rowgroups;
  int nsplit;      // context splits
  int chunk;       // context keys per split (multiple of kKeyTile)
};

VerifyPlan plan_verify(int B, int L_stride, int T_max, int Hq, int Hkv);
size_t verify_ws_bytes(const VerifyPlan& p, int B, int Hkv);

// Stores e as the calling thread's adapld_last_hip_error and returns
// ADAPLD_ERR_HIP.
int record_hip_error(hipError_t e);

// Incremental n-gram index: per (sequence, n-gram length) level, a table of
// 16-byte slots (a power of two, at least twice the context capacity), a
// pool of position arrays and a 16-byte header.
__host__ __device__ inline size_t ngram_slots(int L_stride) {
  size_t s = 16;
  while (s < 2 * (size_t)L_stride) s <<= 1;
  return s;
}
// Every array's capacity is a power of two >= 4 that doubles when full, so an
// array of c positions has used at most max(8, 4c) ints over its life: the
// pool never needs more than 8 per n-gram plus 4 per position, 12 per token.
__host__ __device__ inline size_t ngram_pool_ints(int L_stride) { return 12 * (size_t)L_stride + 16; }
__host__ __device__ inline size_t ngram_level_bytes(int L_stride) {
  const size_t n = ngram_slots(L_stride) * 16 + ngram_pool_ints(L_stride) * 4 + 16;
  return (n + 255) / 256 * 256;
}

// ---------------------------------------------------------------- launchers
// Each returns the hipError_t of its launches (hipSuccess on success).
hipError_t launch_lexical_match(const int32_t* tokens, const int32_t* lens, int B, int L_stride,
                                int n_max, int32_t* cand_pos, int32_t* cand_count,
                                int32_t* match_n, hipStream_t stream);

// Where a draft tree is written (the layouts of adapld_build_draft_tree).
struct TreeOut {
  const int32_t* tokens;   // [B, L_stride]
  int W, S, T_max;
  int32_t* node_token;
  int32_t* node_parent;
  int32_t* node_depth;
  int32_t* node_src;
  int32_t* node_count;
  uint64_t* tree_mask;
};

// With `tree`, the merge kernel also builds each sequence's draft tree from
// the ranked list it has just formed (the step's fused rank + tree).  With
// `preceding`, position j is scored by bank row j-1 (Eq. (6)); the rerank
// lists of the paper's construction already hold the rows t-1 and pass 0.
hipError_t launch_semantic_topk(const uint16_t* bank, const uint16_t* query, const int32_t* lens,
                                const int32_t* cand_pos, const int32_t* cand_count, int B,
                                int L_stride, int d, int k, float tau, int32_t* topk_pos,
                                float* topk_score, int32_t* topk_count, int32_t* kind,
                                uint64_t* ws_keys, const int32_t* cand_kind, int rerank_only,
                                hipStream_t stream, int seq_div = 1, const TreeOut* tree = nullptr,
                                int preceding = 0);

hipError_t launch_build_draft_tree(const int32_t* tokens, const int32_t* lens,
                                   const int32_t* topk_pos, const int32_t* topk_count,
                                   const int32_t* kind, int B, int L_stride, int k, int W, int S,
                                   int T_max, int32_t* node_token, int32_t* node_parent,
                                   int32_t* node_depth, int32_t* node_src, int32_t* node_count,
                                   uint64_t* tree_mask, hipStream_t stream);

hipError_t launch_tree_verify_attn(const uint16_t* q, const uint16_t* k_ctx, const uint16_t* v_ctx,
                                   const uint16_t* k_tree, const uint16_t* v_tree,
                                   const int32_t* lens, const int32_t* node_count,
                                   const uint64_t* tree_mask, int B, int L_stride, int T_max,
                                   int Hq, int Hkv, float scale, uint16_t* out, float* lse,
                                   void* ws, const VerifyPlan& plan, hipStream_t stream);

size_t embed_ws_bytes(int B, int L_stride);
size_t embed_flag_bytes(int lists, int L_stride);

// The paper's draft construction: branch tokens from the target's top tokens
// after the anchor, each followed by its hidden-state-reranked successor.
// Workspace: branch tokens, per-branch candidate lists and queries, and the
// rerank's lists.
size_t paper_tree_ws_bytes(int B, int L_stride, int W, int d);
hipError_t launch_build_draft_tree_paper(const int32_t* tokens, const int32_t* lens, const uint16_t* bank, int d,
                                         const int32_t* topk_pos, const int32_t* topk_count, const int32_t* kind,
                                         int k, const int32_t* top_tokens, int W, int S, int succ_mode,
                                         const uint16_t* emb, int V_emb, float tau, int B, int L_stride,
                                         int T_max, int32_t* node_token, int32_t* node_parent, int32_t* node_depth,
                                         int32_t* node_src, int32_t* node_count, uint64_t* tree_mask, void* ws,
                                         hipStream_t stream);

// Writes the lexical/embedding candidate set, its size and its kind into ws
// and returns pointers to them.
hipError_t launch_embedding_fallback(const int32_t* tokens, const int32_t* lens, const int32_t* cand_pos,
                                     const int32_t* cand_count, const uint16_t* emb, int V, int B,
                                     int L_stride, int d, float tau, void* ws, int32_t** cands,
                                     int32_t** counts, int32_t** kinds, hipStream_t stream);

// The successor backoff of the paper's construction: for every list v (branch
// v % W of sequence v / W) with skip[v] == 0, the positions t in [1, L-2] whose
// token embedding has cosine >= tau with branch_tok[v]'s, written as rows
// t - 1 in ascending order to lists[v] with their count.
hipError_t launch_successor_embed(const int32_t* tokens, const int32_t* lens, const uint16_t* emb, int V,
                                  int B, int W, int L_stride, int d, float tau, const int32_t* skip,
                                  const int32_t* branch_tok, uint8_t* flags, int32_t* lists,
                                  int32_t* counts, hipStream_t stream);

// Builds (rebuild = 1) or brings up to date (0) the n-gram index of every
// sequence; then answers the lexical match from it.
hipError_t launch_ngram_update(const int32_t* tokens, const int32_t* lens, int B, int L_stride, int n_max,
                               void* index, int rebuild, hipStream_t stream);
// Brings the index up to date after appends; with cand_pos also answers the
// lexical match in the same launch.
hipError_t launch_ngram_append(const int32_t* tokens, const int32_t* lens, int B, int L_stride, int n_max, void* index,
                               int32_t* cand_pos, int32_t* cand_count, int32_t* match_n, hipStream_t stream);
hipError_t launch_ngram_match(const int32_t* tokens, const int32_t* lens, const void* index, int B, int L_stride,
                              int n_max, int32_t* cand_pos, int32_t* cand_count, int32_t* match_n,
                              hipStream_t stream);

hipError_t launch_accept_greedy(const int32_t* node_token, const int32_t* node_parent,
                                const int32_t* node_depth, const int32_t* node_count,
                                const uint64_t* tree_mask, const int32_t* target_next,
                                const int32_t* lens, const uint16_t* k_tree, const uint16_t* v_tree,
                                int B, int L_stride, int T_max, int Hkv, int32_t* accept_len,
                                int32_t* accept_nodes, int32_t* out_tokens, uint16_t* k_ctx,
                                uint16_t* v_ctx, hipStream_t stream);

}  // namespace adapld
