// C ABI of libadapld: argument validation, workspace sizing, status reporting.
// Every check runs on the host before anything is enqueued.
#include <cmath>
#include <cstdint>

#include "adapld_internal.h"

namespace {

thread_local int g_last_hip_error = 0;

constexpr int kVersion = 20000;  // 2.0.0: the rerank takes the score alignment (preceding)

bool misaligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) != 0; }

int hip_status(hipError_t e) {
  if (e == hipSuccess) return ADAPLD_OK;
  g_last_hip_error = static_cast<int>(e);
  return ADAPLD_ERR_HIP;
}

size_t semantic_ws(int B, int L_stride, int k) {
  return (size_t)B * adapld::scan_lists(L_stride) * k * sizeof(uint64_t);
}

// adapld_step: the scan's lists first (rounded to 256 bytes), then the verify
// workspace.
size_t step_sem_part(int B, int L_stride, int k) { return (semantic_ws(B, L_stride, k) + 255) / 256 * 256; }

// The embedding fallback's own part (16-byte aligned), then the scan's lists.
size_t embed_head_ws(int B, int L_stride) { return (adapld::embed_ws_bytes(B, L_stride) + 15) / 16 * 16; }

// Host-side validation of each entry point (shared with adapld_step); B == 0
// is a valid, empty call.
int check_lexical(const int32_t* tokens, const int32_t* lens, int B, int L_stride, int n_max,
                  int32_t* cand_pos, int32_t* cand_count, int32_t* match_n) {
  if (B < 0) return ADAPLD_ERR_INVALID_ARG;
  if (B == 0) return ADAPLD_OK;
  if (!tokens || !lens || !cand_pos || !cand_count || !match_n) return ADAPLD_ERR_NULL_ARG;
  if (L_stride < 1) return ADAPLD_ERR_INVALID_ARG;
  if (n_max < 1 || n_max > ADAPLD_MAX_NMAX) return ADAPLD_ERR_UNSUPPORTED;
  return ADAPLD_OK;
}

int check_semantic(const uint16_t* bank, const uint16_t* query, const int32_t* lens,
                   const int32_t* cand_pos, const int32_t* cand_count, int B, int L_stride,
                   int d, int k, float tau, int32_t* topk_pos, float* topk_score,
                   int32_t* topk_count, int32_t* kind, void* ws, size_t ws_bytes) {
  if (B < 0) return ADAPLD_ERR_INVALID_ARG;
  if (B == 0) return ADAPLD_OK;
  if (!bank || !lens || !cand_pos || !cand_count || !topk_pos || !topk_score || !topk_count ||
      !kind || !ws)
    return ADAPLD_ERR_NULL_ARG;
  if (L_stride < 1 || d < 8 || d % 8 != 0 || k < 1) return ADAPLD_ERR_INVALID_ARG;
  if (d > ADAPLD_MAX_HIDDEN || k > ADAPLD_MAX_K || B > ADAPLD_MAX_SEMANTIC_BATCH ||
      (int64_t)B * L_stride > INT32_MAX)
    return ADAPLD_ERR_UNSUPPORTED;
  if (misaligned16(bank) || (query && misaligned16(query))) return ADAPLD_ERR_INVALID_ARG;
  if (ws_bytes < semantic_ws(B, L_stride, k)) return ADAPLD_ERR_WORKSPACE_TOO_SMALL;
  return ADAPLD_OK;
}

int check_tree(const int32_t* tokens, const int32_t* lens, const int32_t* topk_pos,
               const int32_t* topk_count, const int32_t* kind, int B, int L_stride,
               int k, int W, int S, int T_max, int32_t* node_token,
               int32_t* node_parent, int32_t* node_depth, int32_t* node_src,
               int32_t* node_count, uint64_t* tree_mask) {
  if (B < 0) return ADAPLD_ERR_INVALID_ARG;
  if (B == 0) return ADAPLD_OK;
  if (!tokens || !lens || !topk_pos || !topk_count || !kind || !node_token || !node_parent ||
      !node_depth || !node_src || !node_count || !tree_mask)
    return ADAPLD_ERR_NULL_ARG;
  if (L_stride < 1 || k < 1 || W < 1 || S < 0 || T_max < 1) return ADAPLD_ERR_INVALID_ARG;
  if (k > ADAPLD_MAX_K || T_max > ADAPLD_MAX_TREE_NODES) return ADAPLD_ERR_UNSUPPORTED;
  if ((long long)W * (S + 1LL) > T_max) return ADAPLD_ERR_INVALID_ARG;
  return ADAPLD_OK;
}

int check_verify(const uint16_t* q, const uint16_t* k_ctx, const uint16_t* v_ctx,
                 const uint16_t* k_tree, const uint16_t* v_tree, const int32_t* lens,
                 const int32_t* node_count, const uint64_t* tree_mask, int B,
                 int L_stride, int T_max, int Hq, int Hkv, int D, float scale,
                 uint16_t* out, float* lse, void* ws, size_t ws_bytes) {
  if (B < 0) return ADAPLD_ERR_INVALID_ARG;
  if (B == 0) return ADAPLD_OK;
  if (!q || !k_ctx || !v_ctx || !k_tree || !v_tree || !lens || !node_count || !tree_mask || !out)
    return ADAPLD_ERR_NULL_ARG;
  if (L_stride < 1 || T_max < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || !std::isfinite(scale) ||
      !(scale > 0.f))
    return ADAPLD_ERR_INVALID_ARG;
  if (D != ADAPLD_HEAD_DIM || T_max > ADAPLD_MAX_TREE_NODES) return ADAPLD_ERR_UNSUPPORTED;
  if (misaligned16(q) || misaligned16(k_ctx) || misaligned16(v_ctx) || misaligned16(k_tree) ||
      misaligned16(v_tree) || misaligned16(out))
    return ADAPLD_ERR_INVALID_ARG;
  const adapld::VerifyPlan p = adapld::plan_verify(B, L_stride, T_max, Hq, Hkv);
  const size_t need = adapld::verify_ws_bytes(p, B, Hkv);
  if (need > 0 && !ws) return ADAPLD_ERR_NULL_ARG;
  if (ws_bytes < need) return ADAPLD_ERR_WORKSPACE_TOO_SMALL;
  if (need > 0 && misaligned16(ws)) return ADAPLD_ERR_INVALID_ARG;
  return ADAPLD_OK;
}

}  // namespace

int adapld::record_hip_error(hipError_t e) {
  g_last_hip_error = static_cast<int>(e);
  return ADAPLD_ERR_HIP;
}

extern "C" {

const char* adapld_status_string(int status) {
  switch (status) {
    case ADAPLD_OK: return "ok";
    case ADAPLD_ERR_NULL_ARG: return "a required pointer argument is NULL";
    case ADAPLD_ERR_INVALID_ARG: return "invalid size, shape or alignment argument";
    case ADAPLD_ERR_UNSUPPORTED: return "argument outside the limits this library implements";
    case ADAPLD_ERR_WORKSPACE_TOO_SMALL: return "workspace smaller than adapld_workspace_bytes()";
    case ADAPLD_ERR_HIP: return "a HIP launch failed (see adapld_last_hip_error)";
    default: return "unknown status";
  }
}

int adapld_last_hip_error(void) { return g_last_hip_error; }

int adapld_version(void) { return kVersion; }

size_t adapld_workspace_bytes(int op, int B, int L_stride, int d, int k, int T_max, int Hq, int Hkv,
                              int D) {
  (void)D;
  if (B <= 0 || L_stride <= 0) return 0;
  switch (op) {
    case ADAPLD_OP_SEMANTIC_TOPK:
      if (k < 1 || k > ADAPLD_MAX_K) return 0;
      return semantic_ws(B, L_stride, k);
    case ADAPLD_OP_SEMANTIC_TOPK_EMBED:
      if (k < 1 || k > ADAPLD_MAX_K) return 0;
      return embed_head_ws(B, L_stride) + semantic_ws(B, L_stride, k);
    case ADAPLD_OP_BUILD_DRAFT_TREE_PAPER:   // k carries W
      if (k < 1 || k > 64 || d < 8 || d % 8 || (int64_t)B * k > ADAPLD_MAX_SEMANTIC_BATCH) return 0;
      return adapld::paper_tree_ws_bytes(B, L_stride, k, d);
    case ADAPLD_OP_STEP: {
      if (k < 1 || k > ADAPLD_MAX_K || T_max < 1 || T_max > ADAPLD_MAX_TREE_NODES || Hq < 1 || Hkv < 1 ||
          Hq % Hkv)
        return 0;
      const adapld::VerifyPlan p = adapld::plan_verify(B, L_stride, T_max, Hq, Hkv);
      return step_sem_part(B, L_stride, k) + adapld::verify_ws_bytes(p, B, Hkv);
    }
    case ADAPLD_OP_TREE_VERIFY_ATTN: {
      if (T_max < 1 || T_max > ADAPLD_MAX_TREE_NODES || Hq < 1 || Hkv < 1 || Hq % Hkv) return 0;
      const adapld::VerifyPlan p = adapld::plan_verify(B, L_stride, T_max, Hq, Hkv);
      return adapld::verify_ws_bytes(p, B, Hkv);
    }
    default:
      return 0;
  }
}

int adapld_verify_plan(int B, int L_stride, int T_max, int Hq, int Hkv, int32_t* info) {
  if (!info) return ADAPLD_ERR_NULL_ARG;
  if (B < 1 || L_stride < 1 || T_max < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv) return ADAPLD_ERR_INVALID_ARG;
  if (T_max > ADAPLD_MAX_TREE_NODES) return ADAPLD_ERR_UNSUPPORTED;
  const adapld::VerifyPlan p = adapld::plan_verify(B, L_stride, T_max, Hq, Hkv);
  info[0] = p.waves;
  info[1] = p.kh;
  info[2] = p.rows_per_wg;
  info[3] = p.rowgroups;
  info[4] = p.nsplit;
  info[5] = p.chunk;
  return ADAPLD_OK;
}

int adapld_lexical_match(const int32_t* tokens, const int32_t* lens, int B, int L_stride, int n_max,
                         int32_t* cand_pos, int32_t* cand_count, int32_t* match_n,
                         hipStream_t stream) {
  if (const int st = check_lexical(tokens, lens, B, L_stride, n_max, cand_pos, cand_count, match_n);
      st != ADAPLD_OK || B == 0)
    return st;
  return hip_status(adapld::launch_lexical_match(tokens, lens, B, L_stride, n_max, cand_pos,
                                                 cand_count, match_n, stream));
}

int adapld_semantic_topk(const uint16_t* bank, const uint16_t* query, const int32_t* lens,
                         const int32_t* cand_pos, const int32_t* cand_count, int B, int L_stride,
                         int d, int k, float tau, int preceding, int32_t* topk_pos, float* topk_score,
                         int32_t* topk_count, int32_t* kind, void* ws, size_t ws_bytes,
                         hipStream_t stream) {
  if (const int st = check_semantic(bank, query, lens, cand_pos, cand_count, B, L_stride, d, k,
                                    tau, topk_pos, topk_score, topk_count, kind, ws, ws_bytes);
      st != ADAPLD_OK || B == 0)
    return st;
  if (preceding != 0 && preceding != 1) return ADAPLD_ERR_INVALID_ARG;
  return hip_status(adapld::launch_semantic_topk(bank, query, lens, cand_pos, cand_count, B,
                                                 L_stride, d, k, tau, topk_pos, topk_score,
                                                 topk_count, kind, static_cast<uint64_t*>(ws),
                                                 nullptr, 0, stream, 1, nullptr, preceding));
}

int adapld_semantic_topk_embed(const uint16_t* bank, const uint16_t* query, const int32_t* tokens,
                               const int32_t* lens, const int32_t* cand_pos, const int32_t* cand_count,
                               const uint16_t* emb, int V, int B, int L_stride, int d, int k, float tau,
                               int preceding, int32_t* topk_pos, float* topk_score, int32_t* topk_count,
                               int32_t* kind, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (B < 0) return ADAPLD_ERR_INVALID_ARG;
  if (B == 0) return ADAPLD_OK;
  if (!bank || !tokens || !lens || !cand_pos || !cand_count || !emb || !topk_pos || !topk_score ||
      !topk_count || !kind || !ws)
    return ADAPLD_ERR_NULL_ARG;
  if (L_stride < 1 || d < 8 || d % 8 != 0 || k < 1 || V < 1 || !std::isfinite(tau) ||
      (preceding != 0 && preceding != 1))
    return ADAPLD_ERR_INVALID_ARG;
  if (d > ADAPLD_MAX_HIDDEN || k > ADAPLD_MAX_K || B > ADAPLD_MAX_SEMANTIC_BATCH ||
      (int64_t)B * L_stride > INT32_MAX)
    return ADAPLD_ERR_UNSUPPORTED;
  if (misaligned16(bank) || (query && misaligned16(query)) || misaligned16(emb) || misaligned16(ws))
    return ADAPLD_ERR_INVALID_ARG;
  const size_t head = embed_head_ws(B, L_stride);
  if (ws_bytes < head + semantic_ws(B, L_stride, k)) return ADAPLD_ERR_WORKSPACE_TOO_SMALL;
  int32_t *cands = nullptr, *counts = nullptr, *kinds = nullptr;
  hipError_t e = adapld::launch_embedding_fallback(tokens, lens, cand_pos, cand_count, emb, V, B, L_stride, d,
                                                   tau, ws, &cands, &counts, &kinds, stream);
  if (e != hipSuccess) return hip_status(e);
  uint64_t* keys = reinterpret_cast<uint64_t*>(static_cast<char*>(ws) + head);
  return hip_status(adapld::launch_semantic_topk(bank, query, lens, cands, counts, B, L_stride, d, k, NAN,
                                                 topk_pos, topk_score, topk_count, kind, keys, kinds, 1,
                                                 stream, 1, nullptr, preceding));
}

int adapld_build_draft_tree(const int32_t* tokens, const int32_t* lens, const int32_t* topk_pos,
                            const int32_t* topk_count, const int32_t* kind, int B, int L_stride,
                            int k, int W, int S, int T_max, int32_t* node_token,
                            int32_t* node_parent, int32_t* node_depth, int32_t* node_src,
                            int32_t* node_count, uint64_t* tree_mask, hipStream_t stream) {
  if (const int st = check_tree(tokens, lens, topk_pos, topk_count, kind, B, L_stride, k, W, S,
                                T_max, node_token, node_parent, node_depth, node_src, node_count,
                                tree_mask);
      st != ADAPLD_OK || B == 0)
    return st;
  return hip_status(adapld::launch_build_draft_tree(tokens, lens, topk_pos, topk_count, kind, B,
                                                    L_stride, k, W, S, T_max, node_token,
                                                    node_parent, node_depth, node_src, node_count,
                                                    tree_mask, stream));
}

int adapld_build_draft_tree_paper(const int32_t* tokens, const int32_t* lens, const uint16_t* bank,
                                  int d, const int32_t* topk_pos, const int32_t* topk_count,
                                  const int32_t* kind, int k, const int32_t* top_tokens, int W,
                                  int S, int succ_mode, const uint16_t* emb, int V, float tau,
                                  int B, int L_stride, int T_max, int32_t* node_token,
                                  int32_t* node_parent, int32_t* node_depth, int32_t* node_src,
                                  int32_t* node_count, uint64_t* tree_mask, void* ws,
                                  size_t ws_bytes, hipStream_t stream) {
  if (B < 0) return ADAPLD_ERR_INVALID_ARG;
  if (B == 0) return ADAPLD_OK;
  if (!tokens || !lens || !bank || !topk_pos || !topk_count || !kind || !top_tokens ||
      !node_token || !node_parent || !node_depth || !node_src || !node_count || !tree_mask || !ws)
    return ADAPLD_ERR_NULL_ARG;
  if (L_stride < 1 || d < 8 || d % 8 != 0 || k < 1 || W < 1 || S < 0 || T_max < 1)
    return ADAPLD_ERR_INVALID_ARG;
  if (k > ADAPLD_MAX_K || W > 64 || d > ADAPLD_MAX_HIDDEN || T_max > ADAPLD_MAX_TREE_NODES ||
      (int64_t)B * W > ADAPLD_MAX_SEMANTIC_BATCH || (int64_t)B * W * L_stride > INT32_MAX)
    return ADAPLD_ERR_UNSUPPORTED;
  if ((int64_t)S + 1 + 2LL * W > T_max) return ADAPLD_ERR_INVALID_ARG;
  if (succ_mode != ADAPLD_SUCC_EVERY_BRANCH && succ_mode != ADAPLD_SUCC_SEMANTIC_ONLY)
    return ADAPLD_ERR_INVALID_ARG;
  if (emb && (V < 1 || !std::isfinite(tau) || misaligned16(emb))) return ADAPLD_ERR_INVALID_ARG;
  if (misaligned16(bank) || misaligned16(ws)) return ADAPLD_ERR_INVALID_ARG;
  if (ws_bytes < adapld::paper_tree_ws_bytes(B, L_stride, W, d)) return ADAPLD_ERR_WORKSPACE_TOO_SMALL;
  return hip_status(adapld::launch_build_draft_tree_paper(
      tokens, lens, bank, d, topk_pos, topk_count, kind, k, top_tokens, W, S, succ_mode, emb, V, tau, B,
      L_stride, T_max, node_token, node_parent, node_depth, node_src, node_count, tree_mask, ws, stream));
}

int adapld_tree_verify_attn(const uint16_t* q, const uint16_t* k_ctx, const uint16_t* v_ctx,
                            const uint16_t* k_tree, const uint16_t* v_tree, const int32_t* lens,
                            const int32_t* node_count, const uint64_t* tree_mask, int B,
                            int L_stride, int T_max, int Hq, int Hkv, int D, float scale,
                            uint16_t* out, float* lse, void* ws, size_t ws_bytes,
                            hipStream_t stream) {
  if (const int st = check_verify(q, k_ctx, v_ctx, k_tree, v_tree, lens, node_count, tree_mask, B,
                                  L_stride, T_max, Hq, Hkv, D, scale, out, lse, ws, ws_bytes);
      st != ADAPLD_OK || B == 0)
    return st;
  const adapld::VerifyPlan p = adapld::plan_verify(B, L_stride, T_max, Hq, Hkv);
  return hip_status(adapld::launch_tree_verify_attn(q, k_ctx, v_ctx, k_tree, v_tree, lens,
                                                    node_count, tree_mask, B, L_stride, T_max, Hq,
                                                    Hkv, scale, out, lse, ws, p, stream));
}

int adapld_step(const int32_t* tokens, const int32_t* lens, const uint16_t* bank, const uint16_t* query,
                const uint16_t* q, const uint16_t* k_ctx, const uint16_t* v_ctx, const uint16_t* k_tree,
                const uint16_t* v_tree, int B, int L_stride, int d, int n_max, int k, int W, int S,
                int T_max, int Hq, int Hkv, int D, float tau, int preceding, float scale, int32_t* cand_pos,
                int32_t* cand_count, int32_t* match_n, int32_t* topk_pos, float* topk_score,
                int32_t* topk_count, int32_t* kind, int32_t* node_token, int32_t* node_parent,
                int32_t* node_depth, int32_t* node_src, int32_t* node_count, uint64_t* tree_mask,
                uint16_t* out, float* lse, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (B < 0) return ADAPLD_ERR_INVALID_ARG;
  if (B == 0) return ADAPLD_OK;
  if (preceding != 0 && preceding != 1) return ADAPLD_ERR_INVALID_ARG;
  if (!ws) return ADAPLD_ERR_NULL_ARG;
  if (misaligned16(ws)) return ADAPLD_ERR_INVALID_ARG;
  if (k < 1 || L_stride < 1) return ADAPLD_ERR_INVALID_ARG;
  if (k > ADAPLD_MAX_K) return ADAPLD_ERR_UNSUPPORTED;
  const size_t sem = step_sem_part(B, L_stride, k);
  if (ws_bytes < sem) return ADAPLD_ERR_WORKSPACE_TOO_SMALL;
  void* ws_ver = static_cast<char*>(ws) + sem;
  const size_t ver_bytes = ws_bytes - sem;
  // Every call is validated before the first is enqueued.
  int st = check_lexical(tokens, lens, B, L_stride, n_max, cand_pos, cand_count, match_n);
  if (st == ADAPLD_OK)
    st = check_semantic(bank, query, lens, cand_pos, cand_count, B, L_stride, d, k, tau, topk_pos,
                        topk_score, topk_count, kind, ws, sem);
  if (st == ADAPLD_OK)
    st = check_tree(tokens, lens, topk_pos, topk_count, kind, B, L_stride, k, W, S, T_max, node_token,
                    node_parent, node_depth, node_src, node_count, tree_mask);
  if (st == ADAPLD_OK)
    st = check_verify(q, k_ctx, v_ctx, k_tree, v_tree, lens, node_count, tree_mask, B, L_stride, T_max,
                      Hq, Hkv, D, scale, out, lse, ws_ver, ver_bytes);
  if (st != ADAPLD_OK) return st;
  hipError_t e = adapld::launch_lexical_match(tokens, lens, B, L_stride, n_max, cand_pos, cand_count,
                                              match_n, stream);
  // The rerank's merge kernel builds the tree right after ranking (the same
  // wave routine as adapld_build_draft_tree), which saves that launch.
  const adapld::TreeOut tree{tokens, W, S, T_max, node_token, node_parent, node_depth, node_src, node_count,
                             tree_mask};
  if (e == hipSuccess)
    e = adapld::launch_semantic_topk(bank, query, lens, cand_pos, cand_count, B, L_stride, d, k, tau,
                                     topk_pos, topk_score, topk_count, kind, static_cast<uint64_t*>(ws),
                                     nullptr, 0, stream, 1, &tree, preceding);
  if (e == hipSuccess)
    e = adapld::launch_tree_verify_attn(q, k_ctx, v_ctx, k_tree, v_tree, lens, node_count, tree_mask, B,
                                        L_stride, T_max, Hq, Hkv, scale, out, lse, ws_ver,
                                        adapld::plan_verify(B, L_stride, T_max, Hq, Hkv), stream);
  return hip_status(e);
}

size_t adapld_ngram_index_bytes(int B, int L_stride, int n_max) {
  if (B <= 0 || L_stride <= 0 || n_max < 1 || n_max > ADAPLD_MAX_NMAX) return 0;
  return (size_t)B * n_max * adapld::ngram_level_bytes(L_stride);
}

}  // extern "C"

namespace {

int check_ngram(const int32_t* tokens, const int32_t* lens, const void* index, size_t index_bytes, int B,
                int L_stride, int n_max) {
  if (B < 0) return ADAPLD_ERR_INVALID_ARG;
  if (B == 0) return ADAPLD_OK;
  if (!tokens || !lens || !index) return ADAPLD_ERR_NULL_ARG;
  if (L_stride < 1 || misaligned16(index)) return ADAPLD_ERR_INVALID_ARG;
  if (n_max < 1 || n_max > ADAPLD_MAX_NMAX || B > 65535 || L_stride > (1 << 24))
    return ADAPLD_ERR_UNSUPPORTED;
  if (index_bytes < adapld_ngram_index_bytes(B, L_stride, n_max)) return ADAPLD_ERR_WORKSPACE_TOO_SMALL;
  return ADAPLD_OK;
}

}  // namespace

extern "C" {

int adapld_ngram_index_build(const int32_t* tokens, const int32_t* lens, int B, int L_stride, int n_max,
                             void* index, size_t index_bytes, hipStream_t stream) {
  if (const int st = check_ngram(tokens, lens, index, index_bytes, B, L_stride, n_max); st != ADAPLD_OK || B == 0)
    return st;
  return hip_status(adapld::launch_ngram_update(tokens, lens, B, L_stride, n_max, index, 1, stream));
}

int adapld_ngram_index_append(const int32_t* tokens, const int32_t* lens, int B, int L_stride, int n_max,
                              void* index, size_t index_bytes, hipStream_t stream) {
  if (const int st = check_ngram(tokens, lens, index, index_bytes, B, L_stride, n_max); st != ADAPLD_OK || B == 0)
    return st;
  return hip_status(adapld::launch_ngram_append(tokens, lens, B, L_stride, n_max, index, nullptr, nullptr, nullptr,
                                                stream));
}

int adapld_ngram_index_append_match(const int32_t* tokens, const int32_t* lens, int B, int L_stride, int n_max,
                                    void* index, size_t index_bytes, int32_t* cand_pos, int32_t* cand_count,
                                    int32_t* match_n, hipStream_t stream) {
  if (const int st = check_ngram(tokens, lens, index, index_bytes, B, L_stride, n_max); st != ADAPLD_OK || B == 0)
    return st;
  if (!cand_pos || !cand_count || !match_n) return ADAPLD_ERR_NULL_ARG;
  return hip_status(adapld::launch_ngram_append(tokens, lens, B, L_stride, n_max, index, cand_pos, cand_count,
                                                match_n, stream));
}

int adapld_ngram_index_match(const int32_t* tokens, const int32_t* lens, const void* index, size_t index_bytes,
                             int B, int L_stride, int n_max, int32_t* cand_pos, int32_t* cand_count,
                             int32_t* match_n, hipStream_t stream) {
  if (const int st = check_ngram(tokens, lens, index, index_bytes, B, L_stride, n_max); st != ADAPLD_OK || B == 0)
    return st;
  if (!cand_pos || !cand_count || !match_n) return ADAPLD_ERR_NULL_ARG;
  return hip_status(adapld::launch_ngram_match(tokens, lens, index, B, L_stride, n_max, cand_pos, cand_count,
                                               match_n, stream));
}

int adapld_accept_greedy(const int32_t* node_token, const int32_t* node_parent,
                         const int32_t* node_depth, const int32_t* node_count,
                         const uint64_t* tree_mask, const int32_t* target_next, const int32_t* lens,
                         const uint16_t* k_tree, const uint16_t* v_tree, int B, int L_stride,
                         int T_max, int Hkv, int D, int32_t* accept_len, int32_t* accept_nodes,
                         int32_t* out_tokens, uint16_t* k_ctx, uint16_t* v_ctx,
                         hipStream_t stream) {
  if (B < 0) return ADAPLD_ERR_INVALID_ARG;
  if (B == 0) return ADAPLD_OK;
  if (!node_token || !node_parent || !node_depth || !node_count || !tree_mask || !target_next ||
      !lens || !accept_len || !accept_nodes || !out_tokens)
    return ADAPLD_ERR_NULL_ARG;
  const int n_kv = (k_tree != nullptr) + (v_tree != nullptr) + (k_ctx != nullptr) + (v_ctx != nullptr);
  if (n_kv != 0 && n_kv != 4) return ADAPLD_ERR_NULL_ARG;
  if (L_stride < 1 || T_max < 1) return ADAPLD_ERR_INVALID_ARG;
  if (T_max > ADAPLD_MAX_TREE_NODES || (int64_t)B * (T_max + 1) > INT32_MAX) return ADAPLD_ERR_UNSUPPORTED;
  if (n_kv == 4) {
    if (Hkv < 1) return ADAPLD_ERR_INVALID_ARG;
    if (D != ADAPLD_HEAD_DIM) return ADAPLD_ERR_UNSUPPORTED;
    if (misaligned16(k_tree) || misaligned16(v_tree) || misaligned16(k_ctx) || misaligned16(v_ctx))
      return ADAPLD_ERR_INVALID_ARG;
  }
  return hip_status(adapld::launch_accept_greedy(node_token, node_parent, node_depth, node_count,
                                                 tree_mask, target_next, lens, k_tree, v_tree, B,
                                                 L_stride, T_max, n_kv ? Hkv : 0, accept_len,
                                                 accept_nodes, out_tokens, k_ctx, v_ctx, stream));
}

}  // extern "C"
