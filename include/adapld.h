/*
 * adapld.h -- C ABI of libadapld, the AdaPLD draft-and-verify hot path on
 * AMD MI355X (gfx950).
 *
 * One decoding iteration of AdaPLD (Algorithm 1 of the paper, between two
 * target-model forward passes) is four calls, enqueued on one HIP stream with
 * no host synchronisation between them:
 *
 *   1. adapld_lexical_match     lexical anchoring (Sec. 3.3)
 *   2. adapld_semantic_topk     lexical/semantic backoff + hidden-state
 *                               reranking (Sec. 3.3, Sec. 3.4)
 *   3. adapld_build_draft_tree  reuse construction as a draft tree
 *                               (Sec. 3.5, Sec. 3.6)
 *   4. adapld_tree_verify_attn  tree-masked verify attention (Sec. 3.6)
 *
 * adapld_step enqueues calls 1-4 in that order with one host call (Algorithm
 * 1's draft-and-verify iteration), after validating all four.
 *
 * Call 2 has a drop-in alternative with the paper's own semantic signal,
 * token-embedding similarity (Sec. 3.3, Eq. (4)):
 *
 *   2'. adapld_semantic_topk_embed
 *
 * call 3 has one with the paper's branch tokens from the target's top
 * tokens and hidden-state-reranked successors (Sec. 3.5, Algorithm 1):
 *
 *   3'. adapld_build_draft_tree_paper
 *
 * and, once the target's greedy tokens for the verified tree are known,
 *
 *   5. adapld_accept_greedy     greedy acceptance of the tree and compaction
 *                               of the accepted nodes' K/V (Sec. 3.6,
 *                               Appendix C)
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Every pointer argument is DEVICE memory owned by the caller.  The library
 *   never allocates, frees or keeps a pointer after a call returns; it holds
 *   no state between calls and is safe to call from several host threads.
 * - bf16 tensors are passed as `const uint16_t*` holding the bf16 bit
 *   patterns.  All tensors are dense, row-major, in the layouts stated below;
 *   bf16 tensors must be 16-byte aligned.
 * - `B` sequences are processed per call.  Sequence b has context length
 *   `lens[b]` (device array), clamped on the device to [0, L_stride];
 *   `L_stride` is the allocated length per sequence.
 * - Arguments are validated on the host BEFORE anything is enqueued: on any
 *   error nothing is launched and the function returns a negative status.
 *   B == 0 is valid and enqueues nothing.
 * - Kernels are enqueued on `stream` (0 = the null stream); the call returns
 *   without waiting.  Faults inside a kernel surface at the caller's next
 *   synchronisation on that stream.
 * - Output entries past a per-sequence count are unspecified unless stated.
 * - Workspace: `ws` is caller-owned device scratch of at least
 *   adapld_workspace_bytes(op, ...) bytes; its contents need no
 *   initialisation and are clobbered.  Calls that share one `ws` must not
 *   overlap in time.
 */
#ifndef ADAPLD_H
#define ADAPLD_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes returned by every entry point. */
#define ADAPLD_OK 0
#define ADAPLD_ERR_NULL_ARG (-1)           /* a required pointer is NULL */
#define ADAPLD_ERR_INVALID_ARG (-2)        /* a size/shape/alignment is invalid */
#define ADAPLD_ERR_UNSUPPORTED (-3)        /* valid but outside what the kernels implement */
#define ADAPLD_ERR_WORKSPACE_TOO_SMALL (-4)
#define ADAPLD_ERR_HIP (-5)                /* a HIP launch failed; see adapld_last_hip_error */

/* Retrieval outcome of one sequence (the paper's hit-rate categories,
 * Appendix "Retrieval Hit Rate"). */
#define ADAPLD_KIND_NONE 0   /* lexical miss and the fallback found nothing: plain AR step */
#define ADAPLD_KIND_LEX 1    /* lexical hit: candidates reranked */
#define ADAPLD_KIND_SEM 2    /* lexical miss recovered by the semantic fallback */

/* Operation ids for adapld_workspace_bytes. */
#define ADAPLD_OP_LEXICAL_MATCH 1
#define ADAPLD_OP_SEMANTIC_TOPK 2
#define ADAPLD_OP_BUILD_DRAFT_TREE 3
#define ADAPLD_OP_TREE_VERIFY_ATTN 4
#define ADAPLD_OP_SEMANTIC_TOPK_EMBED 5
#define ADAPLD_OP_BUILD_DRAFT_TREE_PAPER 6
#define ADAPLD_OP_STEP 7

/* Limits of this implementation (larger values return ADAPLD_ERR_UNSUPPORTED). */
#define ADAPLD_MAX_NMAX 64
#define ADAPLD_MAX_K 64
#define ADAPLD_MAX_HIDDEN 8192
#define ADAPLD_MAX_TREE_NODES 256
#define ADAPLD_HEAD_DIM 128
#define ADAPLD_MAX_SEMANTIC_BATCH 2048   /* sequences per adapld_semantic_topk call */

/* Human-readable text for a status code (static storage, never NULL). */
const char* adapld_status_string(int status);

/* The hipError_t of the most recent ADAPLD_ERR_HIP on the calling thread
 * (0 if none). */
int adapld_last_hip_error(void);

/* Library version, major*10000 + minor*100 + patch. */
int adapld_version(void);

/* Bytes of device workspace that `op` needs for these sizes (0 if none).
 * Arguments that an op does not use are ignored; for
 * ADAPLD_OP_BUILD_DRAFT_TREE_PAPER the `k` argument carries W.  Returns 0 for
 * invalid sizes (the entry point itself reports the error). */
size_t adapld_workspace_bytes(int op, int B, int L_stride, int d, int k, int T_max,
                              int Hq, int Hkv, int D);

/* How adapld_tree_verify_attn decomposes a problem of these sizes (host
 * only, no device work): info[0] waves per workgroup, info[1] waves sharing
 * one 32-row block of stacked query rows (1, or 2: each takes half of every
 * key tile), info[2] stacked rows per workgroup, info[3] workgroups per
 * (sequence, kv head) along the rows, info[4] context splits (the partials
 * of more than one are merged by a second kernel), info[5] context keys per
 * split.  `info` is host memory of at least 6 ints, owned by the caller.
 * Returns ADAPLD_OK, ADAPLD_ERR_NULL_ARG, or ADAPLD_ERR_INVALID_ARG /
 * ADAPLD_ERR_UNSUPPORTED for sizes the entry point itself would reject. */
int adapld_verify_plan(int B, int L_stride, int T_max, int Hq, int Hkv, int32_t* info);

/*
 * adapld_lexical_match -- lexical anchoring (Sec. 3.3: the exact-match
 * candidate set of the query anchor, the most recent token), generalised to
 * the longest matching suffix n-gram.
 *
 * For sequence b with context M = tokens[b, 0..L-1], L = lens[b]: for
 * n = n_max down to 1, C_n = { j in [n-1, L-2] : M[j-n+1..j] == M[L-n..L-1] }.
 * The first non-empty level n* is kept (n* = 0 and no candidates if none).
 * n_max = 1 is exactly the paper's single-token match.
 *
 *   tokens     int32 [B, L_stride]          token ids
 *   lens       int32 [B]                    context lengths
 *   n_max      1..ADAPLD_MAX_NMAX
 *   cand_pos   int32 [B, L_stride]  (out)   C_{n*} in ascending order
 *   cand_count int32 [B]            (out)   |C_{n*}|
 *   match_n    int32 [B]            (out)   n*
 *
 * Errors: NULL_ARG for a NULL pointer; INVALID_ARG for B < 0 or
 * L_stride < 1; UNSUPPORTED for n_max outside 1..ADAPLD_MAX_NMAX.
 */
int adapld_lexical_match(const int32_t* tokens, const int32_t* lens, int B, int L_stride,
                         int n_max, int32_t* cand_pos, int32_t* cand_count, int32_t* match_n,
                         hipStream_t stream);

/*
 * adapld_semantic_topk -- the lexical/semantic backoff rule (Sec. 3.3) and
 * hidden-state reranking (Sec. 3.4).
 *
 * The score of a candidate position r is computed with fp32 accumulation (0
 * when either norm is 0):
 *   preceding = 1  Eq. (6) as printed: the state before the candidate against
 *                  the state before the anchor, s(r) = cos(bank[b, r-1], q_b),
 *                  q_b = query[b] or, if `query` is NULL, the bank row
 *                  lens[b]-2; position 0 has no earlier state and is skipped;
 *   preceding = 0  s(r) = cos(bank[b, r], q_b), q_b = query[b] or the bank
 *                  row lens[b]-1.
 * If cand_count[b] > 0 (lexical hit) the candidates are
 * cand_pos[b, 0..cand_count[b]-1] and kind = LEX (also when none of them can
 * be scored).  Otherwise (lexical miss) every position r in [0, L-2] is a
 * candidate (the semantic fallback), entries with s < tau are dropped unless
 * tau is NaN (disabled), and kind = SEM if any entry remains, else NONE.
 * Candidates are ranked by score descending, then position ascending, and
 * the first min(k, #scored) are returned.  Candidate positions outside
 * [preceding, L-1] are skipped.
 *
 *   bank       bf16  [B, L_stride, d]       hidden states (row = position)
 *   query      bf16  [B, d] or NULL
 *   lens, cand_pos, cand_count              as produced by adapld_lexical_match
 *   d          8..ADAPLD_MAX_HIDDEN, multiple of 8
 *   k          1..ADAPLD_MAX_K
 *   tau        fallback threshold; NaN disables it
 *   preceding  0 or 1 (the score alignment above)
 *   topk_pos   int32 [B, k]       (out)     ranked positions
 *   topk_score fp32  [B, k]       (out)     their scores
 *   topk_count int32 [B]          (out)     entries written
 *   kind       int32 [B]          (out)     ADAPLD_KIND_*
 *   ws         workspace of adapld_workspace_bytes(ADAPLD_OP_SEMANTIC_TOPK, B, L_stride, d, k, ...)
 *
 * Errors: NULL_ARG; INVALID_ARG for bad sizes, preceding outside {0, 1} or
 * misaligned bf16 pointers; UNSUPPORTED for d or k beyond the limits,
 * B > ADAPLD_MAX_SEMANTIC_BATCH or B * L_stride > INT32_MAX;
 * WORKSPACE_TOO_SMALL.
 */
int adapld_semantic_topk(const uint16_t* bank, const uint16_t* query, const int32_t* lens,
                         const int32_t* cand_pos, const int32_t* cand_count, int B, int L_stride,
                         int d, int k, float tau, int preceding, int32_t* topk_pos, float* topk_score,
                         int32_t* topk_count, int32_t* kind, void* ws, size_t ws_bytes,
                         hipStream_t stream);

/*
 * adapld_build_draft_tree -- reuse construction (Sec. 3.5) organised as a
 * draft tree (Sec. 3.6).
 *
 * Walks the ranked list; the successor token M[r+1] of entry r opens a new
 * branch unless an earlier branch starts with the same token; at most W
 * branches.  Each branch is M[r+1 .. min(r+1+S, L-1)]: the branch token and
 * up to S copied tokens (with a lexical hit, branch 0 is the paper's main
 * copy path of maximum length S+1).  kind = NONE gives an empty tree.
 * Nodes are stored branch-major, by depth within a branch:
 *
 *   node_token  int32 [B, T_max]  (out)  token id of the node
 *   node_parent int32 [B, T_max]  (out)  parent node, -1 at depth 0 (the
 *                                        root is the last context token)
 *   node_depth  int32 [B, T_max]  (out)  depth; its position is lens[b] + depth
 *   node_src    int32 [B, T_max]  (out)  memory position the node copies
 *   node_count  int32 [B]         (out)  T, the number of nodes (<= W*(S+1))
 *   tree_mask   uint64 [B, T_max, ceil(T_max/64)] (out)  bit v of row u is set
 *                                        iff v is u or an ancestor of u; every
 *                                        bit of rows >= T and columns >= T is 0
 *
 * Inputs: tokens, lens as above; topk_pos, topk_count, kind from
 * adapld_semantic_topk with the same k.  Ranked entries outside [0, L-2]
 * are skipped.
 *
 * Errors: NULL_ARG; INVALID_ARG for W < 1, S < 0, k < 1 or
 * T_max < W*(S+1); UNSUPPORTED for k > ADAPLD_MAX_K or
 * T_max > ADAPLD_MAX_TREE_NODES.
 */
int adapld_build_draft_tree(const int32_t* tokens, const int32_t* lens, const int32_t* topk_pos,
                            const int32_t* topk_count, const int32_t* kind, int B, int L_stride,
                            int k, int W, int S, int T_max, int32_t* node_token,
                            int32_t* node_parent, int32_t* node_depth, int32_t* node_src,
                            int32_t* node_count, uint64_t* tree_mask, hipStream_t stream);

/*
 * adapld_step -- one draft-and-verify iteration (Algorithm 1, between two
 * target forward passes): adapld_lexical_match, adapld_semantic_topk,
 * adapld_build_draft_tree and adapld_tree_verify_attn enqueued on `stream`
 * in that order, with no host synchronisation.  Every argument has the
 * meaning, layout and limits it has in those four calls (n_max for the
 * lexical match; d, k, tau, preceding and query for the rerank; W, S and T_max for the
 * tree; Hq, Hkv, D and scale for the verify; T_max is also the verify's).
 * All four argument sets are validated before anything is enqueued; the
 * status is that of the first failing check, or of the first failing launch.
 *
 *   ws   workspace of adapld_workspace_bytes(ADAPLD_OP_STEP, B, L_stride, d, k,
 *        T_max, Hq, Hkv, D), 16-byte aligned: the rerank's lists, then the
 *        verify's partials
 *
 * Outputs are those of the four calls.
 */
int adapld_step(const int32_t* tokens, const int32_t* lens, const uint16_t* bank, const uint16_t* query,
                const uint16_t* q, const uint16_t* k_ctx, const uint16_t* v_ctx, const uint16_t* k_tree,
                const uint16_t* v_tree, int B, int L_stride, int d, int n_max, int k, int W, int S,
                int T_max, int Hq, int Hkv, int D, float tau, int preceding, float scale, int32_t* cand_pos,
                int32_t* cand_count, int32_t* match_n, int32_t* topk_pos, float* topk_score,
                int32_t* topk_count, int32_t* kind, int32_t* node_token, int32_t* node_parent,
                int32_t* node_depth, int32_t* node_src, int32_t* node_count, uint64_t* tree_mask,
                uint16_t* out, float* lse, void* ws, size_t ws_bytes, hipStream_t stream);

/* Which branch tokens of adapld_build_draft_tree_paper get a successor. */
#define ADAPLD_SUCC_EVERY_BRANCH 0    /* every branch token (the text of Sec. 3.5) */
#define ADAPLD_SUCC_SEMANTIC_ONLY 1   /* only after a semantic anchor (Algorithm 1: the
                                         strict, lexical branch drafts no successor) */

/*
 * adapld_step_noalloc -- adapld_step for callers that cannot allocate device
 * memory (code under HIP graph capture, serving loops or harnesses that
 * forbid hipMalloc): the same arguments without `ws` and `ws_bytes`, the same
 * validation, kernels and outputs.  The workspace is a device array inside
 * the library, ADAPLD_NOALLOC_SCRATCH_BYTES per GPU, that each GPU holds
 * from its first call until the process ends; the call itself allocates
 * nothing.  The device current on the calling thread must be the one that
 * `stream` and the buffers belong to.
 *
 * Every call on one GPU shares that GPU's array: calls that overlap in time
 * on one GPU (other streams, other threads) race and give undefined
 * results.  No part of the array has to start at zero.
 *
 * Errors: those of adapld_step; WORKSPACE_TOO_SMALL when
 * adapld_workspace_bytes(ADAPLD_OP_STEP, ...) for these sizes exceeds
 * ADAPLD_NOALLOC_SCRATCH_BYTES; HIP when the array's address cannot be
 * looked up (see adapld_last_hip_error).
 */
#define ADAPLD_NOALLOC_SCRATCH_BYTES (64u << 20)
int adapld_step_noalloc(const int32_t* tokens, const int32_t* lens, const uint16_t* bank,
                        const uint16_t* query, const uint16_t* q, const uint16_t* k_ctx,
                        const uint16_t* v_ctx, const uint16_t* k_tree, const uint16_t* v_tree, int B,
                        int L_stride, int d, int n_max, int k, int W, int S, int T_max, int Hq,
                        int Hkv, int D, float tau, int preceding, float scale, int32_t* cand_pos,
                        int32_t* cand_count, int32_t* match_n, int32_t* topk_pos, float* topk_score,
                        int32_t* topk_count, int32_t* kind, int32_t* node_token,
                        int32_t* node_parent, int32_t* node_depth, int32_t* node_src,
                        int32_t* node_count, uint64_t* tree_mask, uint16_t* out, float* lse,
                        hipStream_t stream);

/*
 * adapld_build_draft_tree_paper -- the paper's own draft construction
 * (Sec. 3.5, Eqs. (8)-(15), Algorithm 1); an alternative to call 3 with the
 * same outputs.
 *
 * The anchor is j* = topk_pos[b, 0] (no tree when topk_count[b] == 0, kind
 * is NONE or j* is outside [0, L-2]).  Nodes, in this order:
 *   - on a lexical hit (kind LEX) the main path: the chain M[j*+1 ..
 *     j*+min(S+1, L-1-j*)], src = its memory positions;
 *   - the branch tokens: the entries of top_tokens[b, j*, 0..W-1] that are
 *     >= 0, not a repeat of an earlier entry and (on a lexical hit) not
 *     M[j*+1], in table order; each is a depth-0 node with src = -1;
 *   - right after each branch token c that drafts a successor (every one
 *     under ADAPLD_SUCC_EVERY_BRANCH; under ADAPLD_SUCC_SEMANTIC_ONLY only
 *     when kind is SEM), its successor.  The candidates are the occurrences
 *     t in [1, L-2] with M[t] == c; when there is none and `emb` is given,
 *     they are the positions t in [1, L-2] whose token embedding has cosine
 *     >= tau with c's (the lexical-first backoff of Sec. 3.3 applied to the
 *     successor query, as Sec. 3.5 states; a token id outside [0, V) has a
 *     zero embedding, cosine 0).  The chosen t is the candidate whose
 *     preceding hidden state bank[b, t-1] has the highest cosine with
 *     bank[b, j*] (ties: lowest t; fp32 scores as in adapld_semantic_topk);
 *     the node is M[t+1] at depth 1 with src = t+1.  A branch token without
 *     candidates has no successor.
 * Node arrays and tree_mask have the layouts of adapld_build_draft_tree;
 * T <= (S+1) + 2W.  Entries at or beyond T are unspecified except the mask
 * rows, which are 0.
 *
 *   tokens, lens      as in adapld_lexical_match
 *   bank              bf16 [B, L_stride, d] hidden states, d a multiple of 8
 *   topk_pos, topk_count, kind, k   the retrieval outcome (adapld_semantic_topk)
 *   top_tokens int32 [B, L_stride, W]  the target's top-W tokens predicted
 *                     after each position, best first; -1 marks an empty slot
 *   W                 1..64 branch tokens;  S >= 0 main-path copy length
 *   succ_mode         ADAPLD_SUCC_EVERY_BRANCH or ADAPLD_SUCC_SEMANTIC_ONLY
 *   emb               bf16 [V, d] token embeddings (same d as the bank,
 *                     16-byte aligned) for the successor backoff, or NULL
 *                     for lexical-only successor retrieval (V, tau ignored)
 *   V, tau            rows of emb; the embedding threshold (finite)
 *   ws                workspace of adapld_workspace_bytes(
 *                     ADAPLD_OP_BUILD_DRAFT_TREE_PAPER, B, L_stride, d, W, ...)
 *                     (the k slot carries W), 16-byte aligned
 *
 * Errors: NULL_ARG; INVALID_ARG for bad sizes, T_max < (S+1) + 2W, a
 * succ_mode other than the two above, V < 1 or tau not finite with emb, or
 * misaligned bank/emb/ws; UNSUPPORTED for k > ADAPLD_MAX_K, W > 64,
 * d > ADAPLD_MAX_HIDDEN, T_max > ADAPLD_MAX_TREE_NODES,
 * B*W > ADAPLD_MAX_SEMANTIC_BATCH or B*W*L_stride > INT32_MAX;
 * WORKSPACE_TOO_SMALL.
 */
int adapld_build_draft_tree_paper(const int32_t* tokens, const int32_t* lens, const uint16_t* bank,
                                  int d, const int32_t* topk_pos, const int32_t* topk_count,
                                  const int32_t* kind, int k, const int32_t* top_tokens, int W,
                                  int S, int succ_mode, const uint16_t* emb, int V, float tau,
                                  int B, int L_stride, int T_max, int32_t* node_token,
                                  int32_t* node_parent, int32_t* node_depth, int32_t* node_src,
                                  int32_t* node_count, uint64_t* tree_mask, void* ws,
                                  size_t ws_bytes, hipStream_t stream);

/*
 * adapld_tree_verify_attn -- tree attention for verification (Sec. 3.6):
 * every draft node is scored against the KV cache in one pass.
 *
 * For node u < T = node_count[b] and query head h (kv head g = h / (Hq/Hkv)):
 * the keys are k_ctx[b, g, 0..L-1] followed by k_tree[b, v, g] for every v
 * with bit v of tree_mask[b, u] set; values likewise.  With logits
 * z = scale * q . key (fp32 accumulation of bf16 products):
 *   out[b, u, h] = softmax(z) . values        (bf16)
 *   lse[b, h, u] = ln sum exp(z)              (fp32)
 * A row whose mask row is empty attends to the context keys only: that is how
 * the root (the last context token, whose K/V are already cached at L-1) is
 * verified with its tree in one call, as row 0 with the tree's rows and mask
 * bits shifted by one.
 *
 *   q          bf16 [B, T_max, Hq, D]
 *   k_ctx      bf16 [B, Hkv, L_stride, D]
 *   v_ctx      bf16 [B, Hkv, L_stride, D]
 *   k_tree     bf16 [B, T_max, Hkv, D]
 *   v_tree     bf16 [B, T_max, Hkv, D]
 *   lens, node_count, tree_mask             as above
 *   D          ADAPLD_HEAD_DIM (128)
 *   out        bf16 [B, T_max, Hq, D]  (out) rows u >= T are not written
 *   lse        fp32 [B, Hq, T_max]     (out, may be NULL) entries u >= T not written
 *   ws         workspace of adapld_workspace_bytes(ADAPLD_OP_TREE_VERIFY_ATTN, B, L_stride, 0, 0, T_max, Hq, Hkv, D)
 *              bytes (0 when the context is not split; ws may then be NULL)
 *
 * q, k and v must be finite (NaN or infinite inputs give undefined results);
 * scale must be finite and > 0 (the usual 1/sqrt(D)).
 *
 * Errors: NULL_ARG; INVALID_ARG for Hq % Hkv != 0, non-positive sizes,
 * scale not finite and > 0, or misaligned pointers; UNSUPPORTED for D != 128 or
 * T_max > ADAPLD_MAX_TREE_NODES; WORKSPACE_TOO_SMALL.
 */
int adapld_tree_verify_attn(const uint16_t* q, const uint16_t* k_ctx, const uint16_t* v_ctx,
                            const uint16_t* k_tree, const uint16_t* v_tree, const int32_t* lens,
                            const int32_t* node_count, const uint64_t* tree_mask, int B,
                            int L_stride, int T_max, int Hq, int Hkv, int D, float scale,
                            uint16_t* out, float* lse, void* ws, size_t ws_bytes,
                            hipStream_t stream);

/*
 * adapld_semantic_topk_embed -- the lexical/semantic backoff with the paper's
 * own semantic signal (Sec. 3.3, Eqs. (4)-(5)) followed by the hidden-state
 * rerank (Sec. 3.4, Eqs. (6)-(7)).  A drop-in alternative to
 * adapld_semantic_topk: same candidate inputs, same outputs.
 *
 * For a sequence with a lexical hit (cand_count[b] > 0) the candidates are
 * its lexical set.  Otherwise they are the positions j in [0, L-2] whose
 * token embedding has cosine >= tau with the embedding of the last token
 * (emb rows of tokens[b, j] and tokens[b, L-1]; a token id outside [0, V)
 * has a zero embedding, cosine 0), in ascending order.  The candidates are
 * then ranked exactly as adapld_semantic_topk ranks a lexical set (with the
 * same `preceding` alignment), and the first min(k, #scored) are kept.
 *   bank, query, lens, cand_pos, cand_count, B, L_stride, d, k, preceding,
 *   topk_*:    as for adapld_semantic_topk
 *   tokens     int32 [B, L_stride], the context
 *   emb        bf16 [V, d], the target model's token embeddings
 *              (16-byte aligned; same d as the bank)
 *   tau        the embedding threshold of Eq. (4); must be finite
 *   kind       LEX on a lexical hit, SEM when the embedding set is
 *              non-empty, NONE otherwise (topk_count 0: an autoregressive
 *              step; no hidden state is scanned for it)
 *   ws         adapld_workspace_bytes(ADAPLD_OP_SEMANTIC_TOPK_EMBED, B,
 *              L_stride, d, k, ...) bytes, 16-byte aligned
 * Errors: NULL_ARG; INVALID_ARG (B < 0, L_stride < 1, d < 8 or d % 8, k < 1,
 * V < 1, tau not finite, preceding outside {0, 1}, misaligned pointers);
 * UNSUPPORTED (d > 8192, k > 64, B > ADAPLD_MAX_SEMANTIC_BATCH);
 * WORKSPACE_TOO_SMALL.
 */
int adapld_semantic_topk_embed(const uint16_t* bank, const uint16_t* query, const int32_t* tokens,
                               const int32_t* lens, const int32_t* cand_pos, const int32_t* cand_count,
                               const uint16_t* emb, int V, int B, int L_stride, int d, int k, float tau,
                               int preceding, int32_t* topk_pos, float* topk_score, int32_t* topk_count,
                               int32_t* kind, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Incremental n-gram index -- the lexical anchoring of adapld_lexical_match
 * (Sec. 3.3, the exact-match set generalised to the longest matching suffix
 * n-gram) answered from a device-resident index that is brought up to date
 * with each iteration's new tokens, instead of a scan of the whole context
 * (the draft-search cost trade-off of Appendix E, "Boundary Conditions for
 * Effective Reuse").
 *
 * For every sequence and n = 1 .. n_max the index keeps, for each n-gram that
 * ends at a candidate position j in [n-1, L-2], the ascending array of those
 * positions.  adapld_ngram_index_match then returns exactly what
 * adapld_lexical_match returns for the current tokens and lens (same outputs,
 * bit for bit), reading C_lex as one contiguous array.
 *
 *   tokens, lens, B, L_stride, n_max   as in adapld_lexical_match; every call
 *              on one index uses the same B, L_stride and n_max
 *   index      caller-owned device buffer of adapld_ngram_index_bytes(B,
 *              L_stride, n_max) bytes, 16-byte aligned; it holds the index
 *              between calls (the one piece of state the library keeps, in
 *              the caller's memory)
 *
 * adapld_ngram_index_build   indexes the current contexts from scratch.
 * adapld_ngram_index_append  brings the index up to date after tokens were
 *              appended to the contexts (tokens[b, L_old .. L-1] written,
 *              lens[b] raised): it inserts only the positions that became
 *              candidates, j in [L_old - 1, L - 2].  A sequence whose length
 *              went down, or an index that was never built, is rebuilt.
 * adapld_ngram_index_match   cand_pos / cand_count / match_n as
 *              adapld_lexical_match; a sequence whose index does not reflect
 *              lens[b] (append not called) gets match_n = -1, cand_count = 0.
 * adapld_ngram_index_append_match  append, then match, in one launch (one
 *              iteration of the decoding loop's lexical step).
 *
 * Errors: NULL_ARG; INVALID_ARG (B < 0, L_stride < 1, misaligned index);
 * UNSUPPORTED (n_max outside 1..ADAPLD_MAX_NMAX, B > 65535, L_stride >
 * 2^24); WORKSPACE_TOO_SMALL (index_bytes below the size).
 */
size_t adapld_ngram_index_bytes(int B, int L_stride, int n_max);
int adapld_ngram_index_build(const int32_t* tokens, const int32_t* lens, int B, int L_stride, int n_max,
                             void* index, size_t index_bytes, hipStream_t stream);
int adapld_ngram_index_append(const int32_t* tokens, const int32_t* lens, int B, int L_stride, int n_max,
                              void* index, size_t index_bytes, hipStream_t stream);
int adapld_ngram_index_match(const int32_t* tokens, const int32_t* lens, const void* index, size_t index_bytes,
                             int B, int L_stride, int n_max, int32_t* cand_pos, int32_t* cand_count,
                             int32_t* match_n, hipStream_t stream);
int adapld_ngram_index_append_match(const int32_t* tokens, const int32_t* lens, int B, int L_stride, int n_max,
                                    void* index, size_t index_bytes, int32_t* cand_pos, int32_t* cand_count,
                                    int32_t* match_n, hipStream_t stream);

/*
 * adapld_accept_greedy -- greedy verification of the draft tree (Sec. 3.6:
 * verification follows the standard speculative-decoding rule; Appendix C:
 * with greedy decoding a draft token is kept when it equals the target's own
 * choice, and the first mismatch ends it) and compaction of the kept nodes'
 * K/V into the cache.
 *
 * Inputs (the tree as adapld_build_draft_tree writes it):
 *   node_token, node_parent, node_depth  int32 [B, T_max]
 *   node_count  int32 [B]   (clamped to [0, T_max] on the device)
 *   tree_mask   uint64 [B, T_max, ceil(T_max/64)]  ancestor-or-self bits
 *   target_next int32 [B, T_max + 1]: column 0 = the target's greedy token
 *               after the context, column 1 + u = after node u's path
 *   lens        int32 [B]   context length L (clamped to [0, L_stride])
 *   k_tree, v_tree  bf16 [B, T_max, Hkv, D]   the tree's K/V (verify layout)
 * Node u is kept when its token equals the target's token after its parent
 * (after the context for a depth-0 node) and so is every ancestor's; the
 * kept path ends at the deepest kept node (the lowest index among equally
 * deep ones).
 * Outputs:
 *   accept_len   int32 [B]               n = number of kept draft nodes
 *   accept_nodes int32 [B, T_max]        entries 0..n-1: the kept nodes by depth
 *   out_tokens   int32 [B, T_max + 1]    entries 0..n: the kept tokens, then
 *                the bonus token (the target's token after the last kept
 *                node, or after the context when n = 0)
 *   k_ctx, v_ctx bf16 [B, Hkv, L_stride, D]: rows L .. L+n-1 of every kv head
 *                receive the kept nodes' K/V rows in path order; rows at or
 *                beyond L_stride are not written; other rows are untouched.
 *                The bonus token's K/V come from the next forward pass.
 * k_tree, v_tree, k_ctx and v_ctx are either all given (D must be 128, each
 * 16-byte aligned) or all NULL (acceptance only; Hkv and D are then ignored).
 * Entries past n in accept_nodes and past n+1 in out_tokens are unspecified.
 * Errors: NULL_ARG (a required pointer, or some but not all of the four K/V
 * pointers); INVALID_ARG (B < 0, L_stride < 1, T_max < 1, Hkv < 1 with K/V,
 * misaligned K/V); UNSUPPORTED (T_max > ADAPLD_MAX_TREE_NODES, D != 128).
 */
int adapld_accept_greedy(const int32_t* node_token, const int32_t* node_parent,
                         const int32_t* node_depth, const int32_t* node_count,
                         const uint64_t* tree_mask, const int32_t* target_next, const int32_t* lens,
                         const uint16_t* k_tree, const uint16_t* v_tree, int B, int L_stride,
                         int T_max, int Hkv, int D, int32_t* accept_len, int32_t* accept_nodes,
                         int32_t* out_tokens, uint16_t* k_ctx, uint16_t* v_ctx,
                         hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* ADAPLD_H */
