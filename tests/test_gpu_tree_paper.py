"""GPU parity of adapld_build_draft_tree_paper (the paper's draft construction,
Sec. 3.5, Eqs. (8)-(15), Algorithm 1) against the oracle.

The retrieval outcome (ranked list and kind) comes from the GPU's own
lexical match and rerank, already checked elsewhere; the oracle builds its
tree from that same list and the same top-token table.  Tree structure,
branch tokens, main path and masks must match exactly; a successor may
differ only where two occurrences of its branch token have near-tied cosines
with the anchor (both sides then hold a valid argmax), the rule of the
ranked-list comparisons.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2606_05742_amd as adapld
from paper_2606_05742_amd.synth import CONFIGS, make_inputs, small_config
from parity_helpers import LazyBank, dev_bf16, dev_i32, near_tie

pytestmark = pytest.mark.gpu


def log(*a):
    print(*a, flush=True, file=sys.stderr)


def top_table(tokens, lens, W, seed, p_empty=0.15, p_dup=0.15, p_copy=0.5):
    """A synthetic top-W table [B, L_stride, W]: tokens drawn from the
    sequence's own context (so that most have occurrences), some slots empty
    (-1) or repeating an earlier slot, and slot 0 often the copy token M[j+1]
    (the target agreeing with the main path)."""
    rng = np.random.default_rng(seed)
    B, Ls = tokens.shape
    top = np.full((B, Ls, W), -1, np.int32)
    for b in range(B):
        L = int(lens[b])
        if L < 1:
            continue
        src = tokens[b, :L]
        top[b, :L] = src[rng.integers(0, L, size=(L, W))]
        if L > 1:
            copy = rng.random(L - 1) < p_copy
            top[b, :L - 1, 0] = np.where(copy, tokens[b, 1:L], top[b, :L - 1, 0])
        if W > 1:
            dup = rng.random((L, W - 1)) < p_dup
            top[b, :L, 1:] = np.where(dup, top[b, :L, :W - 1], top[b, :L, 1:])
        top[b, :L][rng.random((L, W)) < p_empty] = -1
    return top


def decode_mask(words, T_max):
    m = np.zeros((T_max, T_max), bool)
    w = words.view(np.uint64)
    for u in range(T_max):
        for v in range(T_max):
            m[u, v] = bool((int(w[u, v // 64]) >> (v % 64)) & 1)
    return m


def exact_emb(V, d, seed, nnz=4):
    """Token embeddings with exactly `nnz` entries of +-1 in the first 8
    dimensions (norm 2 for nnz = 4): every cosine is a multiple of 1/nnz and
    exact in fp32 and float64, so a threshold on such a value decides the same
    way on both sides.  Returns (float64 table, bf16 bits)."""
    rng = np.random.default_rng(seed)
    E = np.zeros((V, d))
    for r in range(V):
        cols = rng.choice(8, size=nnz, replace=False)
        E[r, cols] = rng.choice([-1.0, 1.0], size=nnz)
    return E, (E.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)


def check_paper_tree(M, bank, kind, ranked, top_row, W, S, g, b, ctx, succ_mode=0, emb=None, tau=None):
    """Sequence b's GPU tree against the oracle's, built from the same inputs."""
    t = oracle.build_draft_tree_paper(M, bank, kind, ranked, top_row, W, S, succ_mode=succ_mode, emb=emb, tau=tau)
    T = t["T"]
    assert int(g["node_count"][b]) == T, f"{ctx}: T {int(g['node_count'][b])} != {T}"
    for key in ("parent", "depth"):
        np.testing.assert_array_equal(g["node_" + key][b, :T], t[key], err_msg=f"{ctx}: {key}")
    L = len(M)
    j = int(ranked[0]) if T else -1
    for u in range(T):
        gt, gs = int(g["node_token"][b, u]), int(g["node_src"][b, u])
        ot, os_ = t["token"][u], t["src"][u]
        if t["depth"][u] == 1 and t["parent"][u] >= 0 and t["src"][t["parent"][u]] == -1 and gs != os_:
            # a successor: another candidate of the branch token with a near-tied cosine
            c = t["token"][t["parent"][u]]
            tg, to = gs - 1, os_ - 1
            cands = oracle.adapld_oracle.successor_candidates(M, c, emb, tau)
            assert tg in cands, f"{ctx}: node {u} src {gs} is no candidate of {c}"
            sg, so = oracle.cosine_rows(bank, [tg - 1, to - 1], bank[j])
            assert near_tie(sg, so), f"{ctx}: node {u} successor cos {sg} vs oracle {so}"
            assert gt == int(M[gs]), f"{ctx}: node {u} token"
            continue
        assert (gt, gs) == (ot, os_), f"{ctx}: node {u} (token, src) {(gt, gs)} != {(ot, os_)}"
    T_max = g["node_token"].shape[1]
    ref = np.zeros((T_max, T_max), bool)
    ref[:T, :T] = t["mask"]
    np.testing.assert_array_equal(decode_mask(g["tree_mask"][b], T_max), ref, err_msg=f"{ctx}: mask")
    return t


def run(x, cfg, top, W, S, T_max=None, seqs=None, dense_bank=True, ctx="", succ_mode=0, emb=None, tau=None):
    """emb: (float64 table, bf16 bits) or None."""
    tokens, lens, bank = dev_i32(x["tokens"]), dev_i32(x["lens"]), dev_bf16(x["bank"])
    cp, cc, _ = adapld.lexical_match(tokens, lens, cfg.n_max)
    pos, _, cnt, kind = adapld.semantic_topk(bank, lens, cp, cc, cfg.k)
    out = adapld.build_draft_tree_paper(tokens, lens, bank, pos, cnt, kind, dev_i32(top), S, T_max,
                                        succ_mode=succ_mode, emb=None if emb is None else dev_bf16(emb[1]), tau=tau)
    torch.cuda.synchronize()
    names = ("node_token", "node_parent", "node_depth", "node_src", "node_count", "tree_mask")
    g = {n: o.cpu().numpy() for n, o in zip(names, out)}
    pos, cnt, kind = pos.cpu().numpy(), cnt.cpu().numpy(), kind.cpu().numpy()
    kinds = []
    for b in (range(cfg.B) if seqs is None else seqs):
        L = int(x["lens"][b])
        M = x["tokens"][b, :L]
        bk = oracle.bf16_bits_to_f64(x["bank"][b, :L]) if dense_bank else LazyBank(x["bank"][b], L)
        ranked = [int(p) for p in pos[b, :int(cnt[b])]]
        j = ranked[0] if ranked else 0
        t = check_paper_tree(M, bk, int(kind[b]), ranked, top[b, j], W, S, g, b, f"{ctx} b={b}",
                             succ_mode=succ_mode, emb=None if emb is None else emb[0], tau=tau)
        kinds.append((int(kind[b]), t["T"]))
    return g, kinds


# L = 701 and 1503 give rows that do not start on 16 bytes (token-at-a-time
# loads); 9001 and 20000 take several passes of the setup kernel; W = 64 (the
# limit) fills every lane of the setup and assembly waves.
@pytest.mark.parametrize("succ_mode", [0, 1])
@pytest.mark.parametrize("L,d,W,S,seed", [(300, 128, 4, 12, 1), (2100, 256, 8, 6, 2), (701, 520, 1, 0, 3),
                                          (1503, 128, 16, 3, 4), (9001, 64, 4, 12, 5), (20000, 64, 8, 4, 6),
                                          (900, 64, 64, 20, 7)])
def test_paper_tree(L, d, W, S, seed, succ_mode):
    cfg = small_config(B=6, L=L, d=d, k=8, n_max=3, seed=200 + seed, V=40, forced_every=3)
    x = make_inputs(cfg, with_verify=False)
    top = top_table(x["tokens"], x["lens"], W, seed)
    g, kinds = run(x, cfg, top, W, S, ctx=f"L={L} W={W} S={S} mode={succ_mode}", succ_mode=succ_mode)
    if succ_mode == 1:   # Algorithm 1: a lexical anchor's tree holds no successor (no node under a branch token)
        for b, (k, T) in enumerate(kinds):
            if k == oracle.KIND_LEX:
                par, src = g["node_parent"][b, :T], g["node_src"][b, :T]
                assert all(src[p] != -1 for p in par if p >= 0), b
    ks = {k for k, _ in kinds}
    assert oracle.KIND_LEX in ks and oracle.KIND_SEM in ks, kinds
    assert any(T > 0 for _, T in kinds)


def test_paper_tree_ragged_and_degenerate():
    """Lengths 0, 1, 2, 3 and ragged ones; a T_max with spare rows (zero mask
    rows); a table with no usable token at some anchors."""
    cfg = small_config(B=8, L=400, d=64, k=4, n_max=2, seed=231, V=12, forced_every=2)
    lens = np.array([0, 1, 2, 3, 57, 400, 399, 130], np.int32)
    x = make_inputs(cfg, lens=lens, with_verify=False)
    top = top_table(x["tokens"], x["lens"], 4, 9)
    top[5] = -1                                     # no branch token anywhere in sequence 5
    top[6, :, 1:] = top[6, :, :1]                   # every slot repeats slot 0
    _, kinds = run(x, cfg, top, 4, 5, T_max=40, ctx="ragged")
    assert kinds[0] == (oracle.KIND_NONE, 0) and kinds[1] == (oracle.KIND_NONE, 0)


def test_paper_tree_no_occurrences():
    """Branch tokens that never occur in the context (ids outside its
    vocabulary) get no successor; the main path is unaffected."""
    cfg = small_config(B=4, L=500, d=128, k=8, n_max=3, seed=232, V=30, forced_every=2)
    x = make_inputs(cfg, with_verify=False)
    top = top_table(x["tokens"], x["lens"], 4, 10)
    top[:, :, 2:] = 1000 + np.arange(2, dtype=np.int32)
    run(x, cfg, top, 4, 12, ctx="absent")


def test_paper_tree_benchmark_workload():
    """b16_l8192_gqa32x8's context, bank and sizes (W=4, S=12), every
    sequence checked against the oracle."""
    cfg = CONFIGS["b16_l8192_gqa32x8"]
    log("[paper tree] generating b16_l8192_gqa32x8")
    x = make_inputs(cfg, with_verify=False)
    top = top_table(x["tokens"], x["lens"], cfg.W, 11)
    log("[paper tree] running and comparing")
    _, kinds = run(x, cfg, top, cfg.W, cfg.S, dense_bank=False, ctx="b16_l8192")
    assert {k for k, _ in kinds} >= {oracle.KIND_LEX, oracle.KIND_SEM}, kinds


@pytest.mark.parametrize("succ_mode", [0, 1])
@pytest.mark.parametrize("tau", [0.5, 0.25, 1.0])
def test_paper_tree_successor_backoff(succ_mode, tau):
    """Branch tokens absent from the context (ids 40..63 of a 64-row table;
    the context draws from 40 tokens) take their successor candidates from
    the embedding set, cos(e[M_t], e[c]) >= tau.  Every cosine of the table
    is a multiple of 1/4 and exact in fp32 and float64, so tau = 0.5, 0.25
    and 1.0 sit exactly on cosines present and the >= rule is compared as
    is."""
    cfg = small_config(B=6, L=700, d=64, k=8, n_max=3, seed=241, V=40, forced_every=2)
    x = make_inputs(cfg, with_verify=False)
    top = top_table(x["tokens"], x["lens"], 4, 12)
    rng = np.random.default_rng(13)
    top[:, :, 1:3] = rng.integers(40, 64, size=top[:, :, 1:3].shape)   # two absent tokens per anchor
    top[:, :, 3] = 70                                                   # outside the table: zero embedding
    emb = exact_emb(64, 64, 14)
    g, kinds = run(x, cfg, top, 4, 6, ctx=f"backoff tau={tau} mode={succ_mode}", succ_mode=succ_mode,
                   emb=emb, tau=tau)
    # below tau = 1 (identical embeddings only) the backoff produced successors for absent tokens
    n_succ = 0
    for b, (k, T) in enumerate(kinds):
        par, tok = g["node_parent"][b, :T], g["node_token"][b, :T]
        for u in range(T):
            p = par[u]
            if p >= 0 and g["node_src"][b, p] == -1 and 40 <= tok[p] < 64:
                n_succ += 1
    assert n_succ > 0 or tau == 1.0, kinds


def test_paper_tree_backoff_benchmark_workload():
    """b16_l8192_gqa32x8's contexts with every branch token absent from the
    context and an embedding table over its vocabulary (Algorithm 1: only
    the semantic anchors draft successors); every sequence checked."""
    cfg = CONFIGS["b16_l8192_gqa32x8"]
    log("[paper tree backoff] generating b16_l8192_gqa32x8")
    x = make_inputs(cfg, with_verify=False)
    B, Ls = x["tokens"].shape
    V = 4096   # the table covers the frequent ids; rarer context tokens have zero embeddings
    top = np.full((B, Ls, cfg.W), -1, np.int32)
    for b in range(B):
        absent = np.setdiff1d(np.arange(V), x["tokens"][b, :int(x["lens"][b])])
        top[b] = np.random.default_rng(b).choice(absent, size=(Ls, cfg.W), replace=True)
    emb = exact_emb(V, cfg.d, 15)
    log("[paper tree backoff] running and comparing")
    _, kinds = run(x, cfg, top, cfg.W, cfg.S, dense_bank=False, ctx="b16_l8192 backoff", succ_mode=1,
                   emb=emb, tau=0.75)
    assert {k for k, _ in kinds} >= {oracle.KIND_LEX, oracle.KIND_SEM}, kinds
