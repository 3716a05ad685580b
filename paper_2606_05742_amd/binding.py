"""ctypes binding of libadapld (argument marshalling only).

Every function takes torch tensors that already live on the GPU, checks their
dtype, shape, contiguity and device, and passes raw device pointers plus the
current HIP stream to the C ABI declared in ``include/adapld.h``.  All
computation happens in the library's HIP kernels; nothing here computes a
result.  bf16 tensors may be ``torch.bfloat16`` or 16-bit integer views of
the same bits.  If the library is missing, every call raises AdapldError.
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass

import torch

KIND_NONE, KIND_LEX, KIND_SEM = 0, 1, 2
OP_LEXICAL_MATCH, OP_SEMANTIC_TOPK, OP_BUILD_DRAFT_TREE, OP_TREE_VERIFY_ATTN = 1, 2, 3, 4
OP_SEMANTIC_TOPK_EMBED = 5
OP_BUILD_DRAFT_TREE_PAPER = 6
OP_STEP = 7
SUCC_EVERY_BRANCH, SUCC_SEMANTIC_ONLY = 0, 1
HEAD_DIM = 128

# ADAPLD_LIB names another build of the library (the sanitized host test
# build); by default the in-tree libadapld.so.
LIB_PATH = os.environ.get("ADAPLD_LIB") or os.path.join(os.path.dirname(os.path.abspath(__file__)), "libadapld.so")

_c_i32p = ctypes.c_void_p
_lib = None


class AdapldError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(what)


# name -> (restype, argtypes) for every function include/adapld.h declares
SIGNATURES = {
    "adapld_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "adapld_last_hip_error": (ctypes.c_int, []),
    "adapld_version": (ctypes.c_int, []),
    "adapld_workspace_bytes": (ctypes.c_size_t, [ctypes.c_int] * 9),
    "adapld_verify_plan": (ctypes.c_int, [ctypes.c_int] * 5 + [ctypes.c_void_p]),
    "adapld_accept_greedy": (ctypes.c_int, [ctypes.c_void_p] * 9 + [ctypes.c_int] * 5 + [ctypes.c_void_p] * 6),
    "adapld_lexical_match": (ctypes.c_int, [
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_int,
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]),
    "adapld_semantic_topk": (ctypes.c_int, [
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_float, ctypes.c_int,
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    "adapld_semantic_topk_embed": (ctypes.c_int, [ctypes.c_void_p] * 7 + [ctypes.c_int] * 5 + [ctypes.c_float]
                                   + [ctypes.c_int] + [ctypes.c_void_p] * 5 + [ctypes.c_size_t, ctypes.c_void_p]),
    "adapld_build_draft_tree": (ctypes.c_int, [
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_void_p, ctypes.c_void_p]),
    "adapld_step": (ctypes.c_int, [ctypes.c_void_p] * 9 + [ctypes.c_int] * 11
                    + [ctypes.c_float, ctypes.c_int, ctypes.c_float]
                    + [ctypes.c_void_p] * 16 + [ctypes.c_size_t, ctypes.c_void_p]),
    "adapld_step_noalloc": (ctypes.c_int, [ctypes.c_void_p] * 9 + [ctypes.c_int] * 11
                            + [ctypes.c_float, ctypes.c_int, ctypes.c_float]
                            + [ctypes.c_void_p] * 15 + [ctypes.c_void_p]),
    "adapld_build_draft_tree_paper": (ctypes.c_int, [ctypes.c_void_p] * 3 + [ctypes.c_int] + [ctypes.c_void_p] * 3
                                      + [ctypes.c_int] + [ctypes.c_void_p] + [ctypes.c_int] * 3
                                      + [ctypes.c_void_p, ctypes.c_int, ctypes.c_float] + [ctypes.c_int] * 3
                                      + [ctypes.c_void_p] * 7 + [ctypes.c_size_t, ctypes.c_void_p]),
    "adapld_ngram_index_bytes": (ctypes.c_size_t, [ctypes.c_int] * 3),
    "adapld_ngram_index_build": (ctypes.c_int, [ctypes.c_void_p] * 2 + [ctypes.c_int] * 3
                                 + [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    "adapld_ngram_index_append": (ctypes.c_int, [ctypes.c_void_p] * 2 + [ctypes.c_int] * 3
                                  + [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    "adapld_ngram_index_match": (ctypes.c_int, [ctypes.c_void_p] * 3 + [ctypes.c_size_t] + [ctypes.c_int] * 3
                                 + [ctypes.c_void_p] * 4),
    "adapld_ngram_index_append_match": (ctypes.c_int, [ctypes.c_void_p] * 2 + [ctypes.c_int] * 3
                                        + [ctypes.c_void_p, ctypes.c_size_t] + [ctypes.c_void_p] * 4),
    "adapld_tree_verify_attn": (ctypes.c_int, [
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
        ctypes.c_float, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
        ctypes.c_void_p]),
}


def load_library(path: str = LIB_PATH):
    """Load libadapld.so (once).  Raises AdapldError when it is not built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise AdapldError(-100, f"{path} is missing: build it with `python -m paper_2606_05742_amd.build`")
    lib = ctypes.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(status: int, what: str):
    if status != 0:
        lib = load_library()
        msg = lib.adapld_status_string(status).decode()
        if status == -5:
            msg += f" (hipError {lib.adapld_last_hip_error()})"
        raise AdapldError(status, f"{what}: {msg}")


_BF16_DTYPES = (torch.bfloat16, torch.int16, torch.uint16)


def _ptr(t, name, dtypes, shape=None, nullable=False):
    if t is None:
        if nullable:
            return None
        raise AdapldError(-1, f"{name} is required")
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise AdapldError(-2, f"{name} must live on the GPU (got {t.device})")
    if t.dtype not in dtypes:
        raise AdapldError(-2, f"{name} has dtype {t.dtype}, expected one of {dtypes}")
    if not t.is_contiguous():
        raise AdapldError(-2, f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise AdapldError(-2, f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def workspace_bytes(op, B, L_stride, d=0, k=0, T_max=0, Hq=0, Hkv=0, D=0) -> int:
    return int(load_library().adapld_workspace_bytes(op, B, L_stride, d, k, T_max, Hq, Hkv, D))


def verify_plan(B, L_stride, T_max, Hq, Hkv) -> dict:
    """The verify kernel's decomposition for these sizes (host only)."""
    info = (ctypes.c_int32 * 6)()
    _check(load_library().adapld_verify_plan(B, L_stride, T_max, Hq, Hkv, info), "adapld_verify_plan")
    return dict(zip(("waves", "kh", "rows_per_wg", "rowgroups", "nsplit", "chunk"), list(info)))


def _i32(n, dev):
    return torch.empty(n, dtype=torch.int32, device=dev)


def lexical_match(tokens, lens, n_max, *, cand_pos=None, cand_count=None, match_n=None, stream=None):
    """Longest-suffix n-gram anchoring; returns (cand_pos, cand_count, match_n)."""
    lib = load_library()
    B, L_stride = tokens.shape
    dev = tokens.device
    cand_pos = torch.empty((B, L_stride), dtype=torch.int32, device=dev) if cand_pos is None else cand_pos
    cand_count = _i32(B, dev) if cand_count is None else cand_count
    match_n = _i32(B, dev) if match_n is None else match_n
    st = lib.adapld_lexical_match(
        _ptr(tokens, "tokens", (torch.int32,)), _ptr(lens, "lens", (torch.int32,), (B,)), B, L_stride,
        n_max, _ptr(cand_pos, "cand_pos", (torch.int32,), (B, L_stride)),
        _ptr(cand_count, "cand_count", (torch.int32,), (B,)), _ptr(match_n, "match_n", (torch.int32,), (B,)),
        _stream(stream))
    _check(st, "adapld_lexical_match")
    return cand_pos, cand_count, match_n


def semantic_topk(bank, lens, cand_pos, cand_count, k, *, tau=None, query=None, preceding=False, topk_pos=None,
                  topk_score=None, topk_count=None, kind=None, ws=None, stream=None):
    """Backoff + cosine reranking; returns (topk_pos, topk_score, topk_count, kind).
    preceding=True scores each candidate by the state before it against the
    state before the anchor (Eq. (6) as printed)."""
    lib = load_library()
    B, L_stride, d = bank.shape
    dev = bank.device
    topk_pos = torch.empty((B, k), dtype=torch.int32, device=dev) if topk_pos is None else topk_pos
    topk_score = torch.empty((B, k), dtype=torch.float32, device=dev) if topk_score is None else topk_score
    topk_count = _i32(B, dev) if topk_count is None else topk_count
    kind = _i32(B, dev) if kind is None else kind
    need = workspace_bytes(OP_SEMANTIC_TOPK, B, L_stride, d, k)
    if ws is None:
        ws = torch.empty(max(need, 16), dtype=torch.uint8, device=dev)
    st = lib.adapld_semantic_topk(
        _ptr(bank, "bank", _BF16_DTYPES), _ptr(query, "query", _BF16_DTYPES, (B, d), nullable=True),
        _ptr(lens, "lens", (torch.int32,), (B,)), _ptr(cand_pos, "cand_pos", (torch.int32,), (B, L_stride)),
        _ptr(cand_count, "cand_count", (torch.int32,), (B,)), B, L_stride, d, k,
        float("nan") if tau is None else float(tau), int(bool(preceding)),
        _ptr(topk_pos, "topk_pos", (torch.int32,), (B, k)), _ptr(topk_score, "topk_score", (torch.float32,), (B, k)),
        _ptr(topk_count, "topk_count", (torch.int32,), (B,)), _ptr(kind, "kind", (torch.int32,), (B,)),
        _ptr(ws, "ws", (torch.uint8,)), ws.numel(), _stream(stream))
    _check(st, "adapld_semantic_topk")
    return topk_pos, topk_score, topk_count, kind


def semantic_topk_embed(bank, tokens, lens, cand_pos, cand_count, emb, k, tau, *, query=None, preceding=False,
                        topk_pos=None, topk_score=None, topk_count=None, kind=None, ws=None, stream=None):
    """Backoff with the token-embedding fallback, then the hidden-state
    rerank; returns (topk_pos, topk_score, topk_count, kind)."""
    lib = load_library()
    B, L_stride, d = bank.shape
    V = emb.shape[0]
    dev = bank.device
    topk_pos = torch.empty((B, k), dtype=torch.int32, device=dev) if topk_pos is None else topk_pos
    topk_score = torch.empty((B, k), dtype=torch.float32, device=dev) if topk_score is None else topk_score
    topk_count = _i32(B, dev) if topk_count is None else topk_count
    kind = _i32(B, dev) if kind is None else kind
    need = workspace_bytes(OP_SEMANTIC_TOPK_EMBED, B, L_stride, d, k)
    if ws is None:
        ws = torch.empty(max(need, 16), dtype=torch.uint8, device=dev)
    st = lib.adapld_semantic_topk_embed(
        _ptr(bank, "bank", _BF16_DTYPES), _ptr(query, "query", _BF16_DTYPES, (B, d), nullable=True),
        _ptr(tokens, "tokens", (torch.int32,), (B, L_stride)), _ptr(lens, "lens", (torch.int32,), (B,)),
        _ptr(cand_pos, "cand_pos", (torch.int32,), (B, L_stride)), _ptr(cand_count, "cand_count", (torch.int32,), (B,)),
        _ptr(emb, "emb", _BF16_DTYPES, (V, d)), V, B, L_stride, d, k, float(tau), int(bool(preceding)),
        _ptr(topk_pos, "topk_pos", (torch.int32,), (B, k)), _ptr(topk_score, "topk_score", (torch.float32,), (B, k)),
        _ptr(topk_count, "topk_count", (torch.int32,), (B,)), _ptr(kind, "kind", (torch.int32,), (B,)),
        _ptr(ws, "ws", (torch.uint8,)), ws.numel(), _stream(stream))
    _check(st, "adapld_semantic_topk_embed")
    return topk_pos, topk_score, topk_count, kind


def build_draft_tree(tokens, lens, topk_pos, topk_count, kind, W, S, T_max=None, *, node_token=None,
                     node_parent=None, node_depth=None, node_src=None, node_count=None, tree_mask=None,
                     stream=None):
    """Draft tree from the ranked list; returns (token, parent, depth, src, count, mask)."""
    lib = load_library()
    B, L_stride = tokens.shape
    k = topk_pos.shape[1]
    T_max = W * (S + 1) if T_max is None else T_max
    nw = (T_max + 63) // 64
    dev = tokens.device
    mk = lambda t: torch.empty((B, T_max), dtype=torch.int32, device=dev) if t is None else t  # noqa: E731
    node_token, node_parent, node_depth, node_src = mk(node_token), mk(node_parent), mk(node_depth), mk(node_src)
    node_count = _i32(B, dev) if node_count is None else node_count
    tree_mask = torch.empty((B, T_max, nw), dtype=torch.int64, device=dev) if tree_mask is None else tree_mask
    i32 = (torch.int32,)
    st = lib.adapld_build_draft_tree(
        _ptr(tokens, "tokens", i32), _ptr(lens, "lens", i32, (B,)), _ptr(topk_pos, "topk_pos", i32, (B, k)),
        _ptr(topk_count, "topk_count", i32, (B,)), _ptr(kind, "kind", i32, (B,)), B, L_stride, k, W, S, T_max,
        _ptr(node_token, "node_token", i32, (B, T_max)), _ptr(node_parent, "node_parent", i32, (B, T_max)),
        _ptr(node_depth, "node_depth", i32, (B, T_max)), _ptr(node_src, "node_src", i32, (B, T_max)),
        _ptr(node_count, "node_count", i32, (B,)),
        _ptr(tree_mask, "tree_mask", (torch.int64, torch.uint64), (B, T_max, nw)), _stream(stream))
    _check(st, "adapld_build_draft_tree")
    return node_token, node_parent, node_depth, node_src, node_count, tree_mask


def build_draft_tree_paper(tokens, lens, bank, topk_pos, topk_count, kind, top_tokens, S, T_max=None, *,
                           succ_mode=SUCC_EVERY_BRANCH, emb=None, tau=None,
                           node_token=None, node_parent=None, node_depth=None, node_src=None, node_count=None,
                           tree_mask=None, ws=None, stream=None):
    """The paper's draft tree (main path, branch tokens from the target's top
    tokens, reranked successors); returns (token, parent, depth, src, count,
    mask).  top_tokens is int32 [B, L_stride, W]; succ_mode is
    SUCC_EVERY_BRANCH or SUCC_SEMANTIC_ONLY; emb (bf16 [V, d]) and tau turn on
    the successor retrieval's embedding backoff."""
    lib = load_library()
    B, L_stride, d = bank.shape
    k = topk_pos.shape[1]
    W = top_tokens.shape[2]
    T_max = S + 1 + 2 * W if T_max is None else T_max
    nw = (T_max + 63) // 64
    dev = bank.device
    mk = lambda t: torch.empty((B, T_max), dtype=torch.int32, device=dev) if t is None else t  # noqa: E731
    node_token, node_parent, node_depth, node_src = mk(node_token), mk(node_parent), mk(node_depth), mk(node_src)
    node_count = _i32(B, dev) if node_count is None else node_count
    tree_mask = torch.empty((B, T_max, nw), dtype=torch.int64, device=dev) if tree_mask is None else tree_mask
    need = workspace_bytes(OP_BUILD_DRAFT_TREE_PAPER, B, L_stride, d, W)
    if ws is None:
        ws = torch.empty(max(need, 16), dtype=torch.uint8, device=dev)
    i32 = (torch.int32,)
    if emb is not None:
        if tau is None:
            raise ValueError("the successor backoff needs tau")
        if emb.dim() != 2 or emb.shape[1] != d:
            raise ValueError(f"emb must be [V, {d}], got {tuple(emb.shape)}")
    st = lib.adapld_build_draft_tree_paper(
        _ptr(tokens, "tokens", i32, (B, L_stride)), _ptr(lens, "lens", i32, (B,)), _ptr(bank, "bank", _BF16_DTYPES),
        d, _ptr(topk_pos, "topk_pos", i32, (B, k)), _ptr(topk_count, "topk_count", i32, (B,)),
        _ptr(kind, "kind", i32, (B,)), k, _ptr(top_tokens, "top_tokens", i32, (B, L_stride, W)), W, S,
        int(succ_mode), _ptr(emb, "emb", _BF16_DTYPES, nullable=True), 0 if emb is None else emb.shape[0],
        float("nan") if tau is None else float(tau), B, L_stride, T_max,
        _ptr(node_token, "node_token", i32, (B, T_max)), _ptr(node_parent, "node_parent", i32, (B, T_max)),
        _ptr(node_depth, "node_depth", i32, (B, T_max)), _ptr(node_src, "node_src", i32, (B, T_max)),
        _ptr(node_count, "node_count", i32, (B,)),
        _ptr(tree_mask, "tree_mask", (torch.int64, torch.uint64), (B, T_max, nw)),
        _ptr(ws, "ws", (torch.uint8,)), ws.numel(), _stream(stream))
    _check(st, "adapld_build_draft_tree_paper")
    return node_token, node_parent, node_depth, node_src, node_count, tree_mask


def tree_verify_attn(q, k_ctx, v_ctx, k_tree, v_tree, lens, node_count, tree_mask, *, scale=None,
                     out=None, lse=None, ws=None, with_lse=True, stream=None):
    """Tree-masked attention of every draft node; returns (out, lse)."""
    lib = load_library()
    B, T_max, Hq, D = q.shape
    Hkv, L_stride = k_ctx.shape[1], k_ctx.shape[2]
    dev = q.device
    scale = 1.0 / math.sqrt(D) if scale is None else scale
    out = torch.empty((B, T_max, Hq, D), dtype=torch.bfloat16, device=dev) if out is None else out
    if lse is None and with_lse:
        lse = torch.empty((B, Hq, T_max), dtype=torch.float32, device=dev)
    need = workspace_bytes(OP_TREE_VERIFY_ATTN, B, L_stride, 0, 0, T_max, Hq, Hkv, D)
    if ws is None:
        ws = torch.empty(max(need, 16), dtype=torch.uint8, device=dev)
    nw = (T_max + 63) // 64
    st = lib.adapld_tree_verify_attn(
        _ptr(q, "q", _BF16_DTYPES), _ptr(k_ctx, "k_ctx", _BF16_DTYPES, (B, Hkv, L_stride, D)),
        _ptr(v_ctx, "v_ctx", _BF16_DTYPES, (B, Hkv, L_stride, D)),
        _ptr(k_tree, "k_tree", _BF16_DTYPES, (B, T_max, Hkv, D)),
        _ptr(v_tree, "v_tree", _BF16_DTYPES, (B, T_max, Hkv, D)),
        _ptr(lens, "lens", (torch.int32,), (B,)), _ptr(node_count, "node_count", (torch.int32,), (B,)),
        _ptr(tree_mask, "tree_mask", (torch.int64, torch.uint64), (B, T_max, nw)),
        B, L_stride, T_max, Hq, Hkv, D, float(scale),
        _ptr(out, "out", _BF16_DTYPES, (B, T_max, Hq, D)),
        _ptr(lse, "lse", (torch.float32,), (B, Hq, T_max), nullable=True),
        _ptr(ws, "ws", (torch.uint8,)), ws.numel(), _stream(stream))
    _check(st, "adapld_tree_verify_attn")
    return out, lse


def accept_greedy(node_token, node_parent, node_depth, node_count, tree_mask, target_next, lens, *,
                  k_tree=None, v_tree=None, k_ctx=None, v_ctx=None, accept_len=None, accept_nodes=None,
                  out_tokens=None, stream=None):
    """Greedy acceptance of the draft tree and, when the four K/V tensors are
    given, compaction of the kept nodes' K/V into k_ctx / v_ctx (in place).
    Returns (accept_len, accept_nodes, out_tokens)."""
    lib = load_library()
    B, T_max = node_token.shape
    dev = node_token.device
    nw = (T_max + 63) // 64
    kv = (k_tree, v_tree, k_ctx, v_ctx)
    if any(t is not None for t in kv) and not all(t is not None for t in kv):
        raise AdapldError(-1, "accept_greedy: give all of k_tree, v_tree, k_ctx, v_ctx or none")
    Hkv, D, L_stride = 0, HEAD_DIM, 1
    if k_ctx is not None:
        Hkv, L_stride, D = k_ctx.shape[1], k_ctx.shape[2], k_ctx.shape[3]
    accept_len = torch.empty(B, dtype=torch.int32, device=dev) if accept_len is None else accept_len
    accept_nodes = torch.empty((B, T_max), dtype=torch.int32, device=dev) if accept_nodes is None else accept_nodes
    out_tokens = torch.empty((B, T_max + 1), dtype=torch.int32, device=dev) if out_tokens is None else out_tokens
    i32 = (torch.int32,)
    st = lib.adapld_accept_greedy(
        _ptr(node_token, "node_token", i32, (B, T_max)), _ptr(node_parent, "node_parent", i32, (B, T_max)),
        _ptr(node_depth, "node_depth", i32, (B, T_max)), _ptr(node_count, "node_count", i32, (B,)),
        _ptr(tree_mask, "tree_mask", (torch.int64, torch.uint64), (B, T_max, nw)),
        _ptr(target_next, "target_next", i32, (B, T_max + 1)), _ptr(lens, "lens", i32, (B,)),
        _ptr(k_tree, "k_tree", _BF16_DTYPES, (B, T_max, Hkv, D), nullable=True),
        _ptr(v_tree, "v_tree", _BF16_DTYPES, (B, T_max, Hkv, D), nullable=True),
        B, L_stride, T_max, Hkv, D,
        _ptr(accept_len, "accept_len", i32, (B,)), _ptr(accept_nodes, "accept_nodes", i32, (B, T_max)),
        _ptr(out_tokens, "out_tokens", i32, (B, T_max + 1)),
        _ptr(k_ctx, "k_ctx", _BF16_DTYPES, (B, Hkv, L_stride, D), nullable=True),
        _ptr(v_ctx, "v_ctx", _BF16_DTYPES, (B, Hkv, L_stride, D), nullable=True),
        _stream(stream))
    _check(st, "adapld_accept_greedy")
    return accept_len, accept_nodes, out_tokens


class NgramIndex:
    """The incremental n-gram index of B contexts of capacity L_stride
    (adapld_ngram_index_*): build once, append after the contexts grow, match
    in place of lexical_match.  Holds the index's device buffer."""

    def __init__(self, B, L_stride, n_max, device="cuda"):
        self.B, self.L_stride, self.n_max = B, L_stride, n_max
        nbytes = load_library().adapld_ngram_index_bytes(B, L_stride, n_max)
        if nbytes == 0:
            raise AdapldError(-2, f"no index for B={B}, L_stride={L_stride}, n_max={n_max}")
        self.buf = torch.empty(nbytes, dtype=torch.uint8, device=device)

    def _args(self, tokens, lens):
        i32 = (torch.int32,)
        return (_ptr(tokens, "tokens", i32, (self.B, self.L_stride)), _ptr(lens, "lens", i32, (self.B,)))

    def build(self, tokens, lens, stream=None):
        st = load_library().adapld_ngram_index_build(*self._args(tokens, lens), self.B, self.L_stride, self.n_max,
                                                     self.buf.data_ptr(), self.buf.numel(), _stream(stream))
        _check(st, "adapld_ngram_index_build")
        return self

    def append(self, tokens, lens, stream=None):
        st = load_library().adapld_ngram_index_append(*self._args(tokens, lens), self.B, self.L_stride, self.n_max,
                                                      self.buf.data_ptr(), self.buf.numel(), _stream(stream))
        _check(st, "adapld_ngram_index_append")
        return self

    def _outs(self, dev, cand_pos, cand_count, match_n):
        B, Ls = self.B, self.L_stride
        cand_pos = torch.empty((B, Ls), dtype=torch.int32, device=dev) if cand_pos is None else cand_pos
        cand_count = _i32(B, dev) if cand_count is None else cand_count
        match_n = _i32(B, dev) if match_n is None else match_n
        i32 = (torch.int32,)
        ptrs = (_ptr(cand_pos, "cand_pos", i32, (B, Ls)), _ptr(cand_count, "cand_count", i32, (B,)),
                _ptr(match_n, "match_n", i32, (B,)))
        return (cand_pos, cand_count, match_n), ptrs

    def match(self, tokens, lens, *, cand_pos=None, cand_count=None, match_n=None, stream=None):
        """(cand_pos, cand_count, match_n), as lexical_match returns them."""
        outs, ptrs = self._outs(tokens.device, cand_pos, cand_count, match_n)
        st = load_library().adapld_ngram_index_match(*self._args(tokens, lens), self.buf.data_ptr(), self.buf.numel(),
                                                     self.B, self.L_stride, self.n_max, *ptrs, _stream(stream))
        _check(st, "adapld_ngram_index_match")
        return outs

    def append_match(self, tokens, lens, *, cand_pos=None, cand_count=None, match_n=None, stream=None):
        """append, then match, in one launch."""
        outs, ptrs = self._outs(tokens.device, cand_pos, cand_count, match_n)
        st = load_library().adapld_ngram_index_append_match(*self._args(tokens, lens), self.B, self.L_stride,
                                                            self.n_max, self.buf.data_ptr(), self.buf.numel(), *ptrs,
                                                            _stream(stream))
        _check(st, "adapld_ngram_index_append_match")
        return outs


@dataclass
class StepBuffers:
    """Outputs and workspaces of one step, allocated once and reused."""
    cand_pos: torch.Tensor
    cand_count: torch.Tensor
    match_n: torch.Tensor
    topk_pos: torch.Tensor
    topk_score: torch.Tensor
    topk_count: torch.Tensor
    kind: torch.Tensor
    node_token: torch.Tensor
    node_parent: torch.Tensor
    node_depth: torch.Tensor
    node_src: torch.Tensor
    node_count: torch.Tensor
    tree_mask: torch.Tensor
    out: torch.Tensor
    lse: torch.Tensor
    ws_sem: torch.Tensor
    ws_ver: torch.Tensor
    ws_step: torch.Tensor    # ws_sem and ws_ver are views of it (the layout adapld_step expects)

    @staticmethod
    def allocate(B, L_stride, d, k, T_max, Hq, Hkv, D=HEAD_DIM, device="cuda"):
        i32 = lambda *s: torch.empty(s, dtype=torch.int32, device=device)  # noqa: E731
        nw = (T_max + 63) // 64
        sem = (workspace_bytes(OP_SEMANTIC_TOPK, B, L_stride, d, k) + 255) // 256 * 256
        ver = workspace_bytes(OP_TREE_VERIFY_ATTN, B, L_stride, 0, 0, T_max, Hq, Hkv, D)
        ws_step = torch.empty(sem + max(ver, 16), dtype=torch.uint8, device=device)
        ws_sem, ws_ver = ws_step[:sem], ws_step[sem:]
        return StepBuffers(
            cand_pos=i32(B, L_stride), cand_count=i32(B), match_n=i32(B),
            topk_pos=i32(B, k), topk_score=torch.empty((B, k), dtype=torch.float32, device=device),
            topk_count=i32(B), kind=i32(B),
            node_token=i32(B, T_max), node_parent=i32(B, T_max), node_depth=i32(B, T_max),
            node_src=i32(B, T_max), node_count=i32(B),
            tree_mask=torch.empty((B, T_max, nw), dtype=torch.int64, device=device),
            out=torch.empty((B, T_max, Hq, D), dtype=torch.bfloat16, device=device),
            lse=torch.empty((B, Hq, T_max), dtype=torch.float32, device=device),
            ws_sem=ws_sem, ws_ver=ws_ver, ws_step=ws_step)


class StepCall:
    """One draft-and-verify step as a single native call (adapld_step, which
    enqueues the four kernels on one stream).  The tensors are checked and
    their pointers marshalled once, here; every call() then costs one C call.
    The stream is the one given, else the current stream at construction."""

    def __init__(self, tokens, lens, bank, q, k_ctx, v_ctx, k_tree, v_tree, *, n_max, k, W, S, tau=None,
                 query=None, preceding=False, scale=None, buffers: StepBuffers | None = None, stream=None,
                 noalloc=False):
        B, L_stride = tokens.shape
        _, _, d = bank.shape
        _, T_max, Hq, D = q.shape
        Hkv = k_ctx.shape[1]
        if buffers is None:
            buffers = StepBuffers.allocate(B, L_stride, d, k, T_max, Hq, Hkv, D, device=tokens.device)
        bf = self.buffers = buffers
        need = workspace_bytes(OP_STEP, B, L_stride, d, k, T_max, Hq, Hkv, D)
        if not noalloc and bf.ws_step.numel() < need:
            raise AdapldError(-4, f"buffers.ws_step holds {bf.ws_step.numel()} bytes, {need} needed")
        scale = 1.0 / math.sqrt(D) if scale is None else scale
        tau = float("nan") if tau is None else float(tau)
        i32, bf16 = (torch.int32,), _BF16_DTYPES
        nw = (T_max + 63) // 64
        self._name = "adapld_step_noalloc" if noalloc else "adapld_step"
        self._fn = getattr(load_library(), self._name)
        self._args = (
            _ptr(tokens, "tokens", i32, (B, L_stride)), _ptr(lens, "lens", i32, (B,)),
            _ptr(bank, "bank", bf16), _ptr(query, "query", bf16, (B, d), nullable=True),
            _ptr(q, "q", bf16), _ptr(k_ctx, "k_ctx", bf16, (B, Hkv, L_stride, D)),
            _ptr(v_ctx, "v_ctx", bf16, (B, Hkv, L_stride, D)), _ptr(k_tree, "k_tree", bf16, (B, T_max, Hkv, D)),
            _ptr(v_tree, "v_tree", bf16, (B, T_max, Hkv, D)),
            B, L_stride, d, n_max, k, W, S, T_max, Hq, Hkv, D, tau, int(bool(preceding)), scale,
            _ptr(bf.cand_pos, "cand_pos", i32, (B, L_stride)), _ptr(bf.cand_count, "cand_count", i32, (B,)),
            _ptr(bf.match_n, "match_n", i32, (B,)), _ptr(bf.topk_pos, "topk_pos", i32, (B, k)),
            _ptr(bf.topk_score, "topk_score", (torch.float32,), (B, k)),
            _ptr(bf.topk_count, "topk_count", i32, (B,)), _ptr(bf.kind, "kind", i32, (B,)),
            _ptr(bf.node_token, "node_token", i32, (B, T_max)), _ptr(bf.node_parent, "node_parent", i32, (B, T_max)),
            _ptr(bf.node_depth, "node_depth", i32, (B, T_max)), _ptr(bf.node_src, "node_src", i32, (B, T_max)),
            _ptr(bf.node_count, "node_count", i32, (B,)),
            _ptr(bf.tree_mask, "tree_mask", (torch.int64, torch.uint64), (B, T_max, nw)),
            _ptr(bf.out, "out", bf16, (B, T_max, Hq, D)), _ptr(bf.lse, "lse", (torch.float32,), (B, Hq, T_max)))
        # adapld_step_noalloc takes no workspace: its own device array serves
        self._args += (() if noalloc else (_ptr(bf.ws_step, "ws_step", (torch.uint8,)), bf.ws_step.numel()))
        self._args += (_stream(stream),)
        # keep every tensor alive as long as the call can be made
        self._keep = (tokens, lens, bank, query, q, k_ctx, v_ctx, k_tree, v_tree)

    def __call__(self) -> StepBuffers:
        _check(self._fn(*self._args), self._name)
        return self.buffers


def step(tokens, lens, bank, q, k_ctx, v_ctx, k_tree, v_tree, *, n_max, k, W, S, tau=None, query=None,
         preceding=False, scale=None, buffers: StepBuffers | None = None, stream=None, noalloc=False):
    """One draft-and-verify step: adapld_step, i.e. the four entry points
    back to back on one stream from one native call (adapld_step_noalloc
    with noalloc=True: the library's own device workspace, nothing allocated
    by the call).

    No host synchronisation happens inside; the lexical-hit / fallback decision
    is taken on the device.  Returns the StepBuffers holding every output.
    """
    return StepCall(tokens, lens, bank, q, k_ctx, v_ctx, k_tree, v_tree, n_max=n_max, k=k, W=W, S=S, tau=tau,
                    query=query, preceding=preceding, scale=scale, buffers=buffers, stream=stream,
                    noalloc=noalloc)()


def step_calls(tokens, lens, bank, q, k_ctx, v_ctx, k_tree, v_tree, *, n_max, k, W, S, tau=None, query=None,
               preceding=False, scale=None, buffers: StepBuffers | None = None, stream=None):
    """The same step as four separate entry-point calls (the route a caller
    takes to put its own work or events between them)."""
    B, L_stride = tokens.shape
    T_max = q.shape[1]
    if buffers is None:
        buffers = StepBuffers.allocate(B, L_stride, bank.shape[2], k, T_max, q.shape[2], k_ctx.shape[1],
                                       device=tokens.device)
    bf = buffers
    lexical_match(tokens, lens, n_max, cand_pos=bf.cand_pos, cand_count=bf.cand_count, match_n=bf.match_n,
                  stream=stream)
    semantic_topk(bank, lens, bf.cand_pos, bf.cand_count, k, tau=tau, query=query, preceding=preceding,
                  topk_pos=bf.topk_pos,
                  topk_score=bf.topk_score, topk_count=bf.topk_count, kind=bf.kind, ws=bf.ws_sem, stream=stream)
    build_draft_tree(tokens, lens, bf.topk_pos, bf.topk_count, bf.kind, W, S, T_max, node_token=bf.node_token,
                     node_parent=bf.node_parent, node_depth=bf.node_depth, node_src=bf.node_src,
                     node_count=bf.node_count, tree_mask=bf.tree_mask, stream=stream)
    tree_verify_attn(q, k_ctx, v_ctx, k_tree, v_tree, lens, bf.node_count, bf.tree_mask, scale=scale,
                     out=bf.out, lse=bf.lse, ws=bf.ws_ver, stream=stream)
    return bf
