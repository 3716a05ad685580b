"""Shared helpers of the GPU parity tests: uploads and the comparison rules.

Comparison rules (the bar the HIP path must meet against the oracle):
* lexical candidates, n*, kinds, tree arrays and masks: bit-exact;
* ranked lists: identical positions, except that two entries whose oracle
  scores are within 1e-5 relative (floor 1e-7 absolute, the size of the fp32
  accumulation error of a cosine over a few thousand bf16 products) may swap,
  and the last kept entry may be any of a near-tied group; the GPU's fp32
  scores within 1e-5 absolute of the oracle's float64 scores;
* the oracle tree is rebuilt from the GPU's ranked list and must match
  exactly (so near-tie swaps cannot hide a tree bug);
* verify output: max-abs <= 2e-2 (bf16 output), relative Frobenius error
  <= 1e-2, LSE max-abs <= 1e-4.
"""
from __future__ import annotations

import numpy as np
import torch

import oracle

SCORE_ATOL = 1e-5
TIE_RTOL = 1e-5
TIE_ATOL = 1e-7
O_ATOL = 2e-2
O_RTOL_FRO = 1e-2
LSE_ATOL = 1e-4


def dev_i32(x):
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.int32)).cuda()


def dev_bf16(bits):
    return torch.from_numpy(np.ascontiguousarray(bits, dtype=np.uint16).view(np.int16)).cuda().view(torch.bfloat16)


def bf16_to_np_bits(t):
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


class LazyBank:
    """bank[b] rows decoded to float64 only when indexed (the full bank can be GiBs)."""

    def __init__(self, bits, L):
        self.bits = bits
        self.shape = (L, bits.shape[1])

    def __getitem__(self, rows):
        return oracle.bf16_bits_to_f64(self.bits[rows])


def near_tie(a, b):
    return abs(a - b) <= TIE_RTOL * max(abs(a), abs(b)) + TIE_ATOL


def check_ranked(bank, query, cand, k, tau, g_kind, g_pos, g_score, ctx="", preceding=False):
    """Compare one sequence's GPU ranked list with the oracle; returns the oracle's record.
    preceding: the alignment of Eq. (6) as printed (position j scored by row j-1)."""
    o_kind, o_pos, o_score = oracle.semantic_topk(bank, query, cand, k, tau, preceding=preceding)
    assert g_kind == o_kind, f"{ctx}: kind {g_kind} != {o_kind}"
    L = bank.shape[0]
    sh = 1 if preceding else 0
    q = (bank[L - 1 - sh] if L - 1 - sh >= 0 else np.zeros(bank.shape[1])) if query is None else query
    if g_pos == o_pos:
        np.testing.assert_allclose(g_score, o_score, rtol=0, atol=SCORE_ATOL, err_msg=ctx)
        return o_kind, o_pos, o_score
    # Positions differ: every difference must be explained by near-ties.
    sig = list(oracle.cosine_rows(bank, [p - sh for p in g_pos], q)) if g_pos else []
    np.testing.assert_allclose(g_score, sig, rtol=0, atol=SCORE_ATOL, err_msg=ctx)
    pool = {c for c in cand if c >= sh} if len(cand) > 0 else set(range(sh, L - 1))
    assert set(g_pos) <= pool and len(set(g_pos)) == len(g_pos), ctx
    for i in range(len(sig)):
        for j in range(i + 1, len(sig)):
            assert sig[j] <= sig[i] or near_tie(sig[i], sig[j]), f"{ctx}: inversion {g_pos[i]},{g_pos[j]}"
    if len(g_pos) != len(o_pos):
        # only a tau boundary may change the count, and only by near-ties
        assert tau is not None and len(cand) == 0, ctx
        longer = o_score if len(o_pos) > len(g_pos) else sig
        for s in longer[min(len(o_pos), len(g_pos)):]:
            assert near_tie(s, tau), f"{ctx}: count differs away from tau"
    if sig:
        last = sig[-1]
        for p, s in zip(o_pos, o_score):
            if p not in g_pos and len(g_pos) == min(k, len(pool)):
                assert s <= last or near_tie(s, last), f"{ctx}: missed {p} ({s} > {last})"
    return o_kind, o_pos, o_score


def check_tree(tokens, kind, ranked, W, S, g, b, ctx=""):
    """The GPU tree of sequence b must equal the oracle tree built from the same ranked list."""
    t = oracle.build_draft_tree(tokens, kind, ranked, W, S)
    T = t["T"]
    assert int(g["node_count"][b]) == T, f"{ctx}: T {int(g['node_count'][b])} != {T}"
    for key in ("token", "parent", "depth", "src"):
        np.testing.assert_array_equal(g["node_" + key][b, :T], t[key], err_msg=f"{ctx}: {key}")
    T_max = g["node_token"].shape[1]
    nw = (T_max + 63) // 64
    ref = np.zeros((T_max, nw), dtype=np.uint64)
    for u in range(T):
        for v in range(T):
            if t["mask"][u, v]:
                ref[u, v // 64] |= np.uint64(1) << np.uint64(v % 64)
    np.testing.assert_array_equal(g["tree_mask"][b].view(np.uint64), ref, err_msg=f"{ctx}: mask")
    return t


def check_verify(O_g, LSE_g, O_o, LSE_o, ctx=""):
    O_g = np.asarray(O_g, dtype=np.float64)
    err = np.abs(O_g - O_o)
    assert err.max() <= O_ATOL, f"{ctx}: O max-abs {err.max():.3g}"
    rel = np.linalg.norm(O_g - O_o) / max(np.linalg.norm(O_o), 1e-30)
    assert rel <= O_RTOL_FRO, f"{ctx}: O relative error {rel:.3g}"
    lerr = np.abs(np.asarray(LSE_g, dtype=np.float64) - LSE_o)
    assert lerr.max() <= LSE_ATOL, f"{ctx}: LSE max-abs {lerr.max():.3g}"


def chain_subproblem(parent, u):
    """Node u's root-to-u path: verifying u against the full tree equals verifying
    the last node of this chain (same keys in the same ascending order)."""
    path = []
    v = u
    while v >= 0:
        path.append(v)
        v = parent[v]
    path = path[::-1]
    n = len(path)
    mask = np.tril(np.ones((n, n), dtype=bool))
    return path, mask
