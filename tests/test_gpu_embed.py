"""GPU parity of adapld_semantic_topk_embed (the token-embedding fallback of
Sec. 3.3, Eqs. (4)-(5), then the hidden-state rerank of Sec. 3.4) against
the oracle: the kind of every sequence, and the ranked list of the
candidates the oracle's fallback keeps."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_05742_amd as adapld
from paper_2606_05742_amd.synth import f32_to_bf16_bits, make_inputs, small_config
from parity_helpers import check_ranked, dev_bf16, dev_i32

pytestmark = pytest.mark.gpu


def emb_table(V, d, clusters, seed, zero_rows=()):
    """Token embeddings in clusters (tokens t and t' of the same cluster
    t % clusters have a high cosine), bf16 bits."""
    rng = np.random.default_rng(seed)
    centers = rng.standard_normal((clusters, d))
    E = centers[np.arange(V) % clusters] + 0.35 * rng.standard_normal((V, d))
    for r in zero_rows:
        E[r] = 0.0
    return f32_to_bf16_bits(E.astype(np.float32))


def margin_ok(E, tokens, lens, tau, margin=1e-3):
    for b in range(tokens.shape[0]):
        L = int(lens[b])
        if L < 2:
            continue
        s = oracle.cosine_rows(E, tokens[b, :L - 1], E[int(tokens[b, L - 1])])
        if np.any(np.abs(s - tau) < margin):
            return False
    return True


def run_and_check(cfg, x, E_bits, tau, k, ctx, exact=False, preceding=False):
    """exact: the table's cosines are exact in fp32 (no margin around tau needed);
    preceding: the rerank's alignment (Eq. (6) as printed)."""
    E = oracle.bf16_bits_to_f64(E_bits)
    assert exact or margin_ok(E, x["tokens"], x["lens"], tau), "pick another tau: a cosine sits on it"
    tokens, lens = dev_i32(x["tokens"]), dev_i32(x["lens"])
    cp, cc, mn = adapld.lexical_match(tokens, lens, cfg.n_max)
    pos, sc, cnt, kind = adapld.semantic_topk_embed(dev_bf16(x["bank"]), tokens, lens, cp, cc, dev_bf16(E_bits),
                                                    k, tau, preceding=preceding)
    torch.cuda.synchronize()
    pos, sc, cnt, kind = (t.cpu().numpy() for t in (pos, sc, cnt, kind))
    kinds = []
    for b in range(cfg.B):
        L = int(x["lens"][b])
        M = x["tokens"][b, :L]
        _, C = oracle.lexical_match(M, cfg.n_max)
        ekind, Cs = oracle.embedding_fallback(M, E, C, tau)
        assert int(kind[b]) == ekind, (ctx, b, int(kind[b]), ekind)
        kinds.append(ekind)
        if ekind == oracle.KIND_NONE:
            assert int(cnt[b]) == 0, (ctx, b)
            continue
        n = int(cnt[b])
        check_ranked(oracle.bf16_bits_to_f64(x["bank"][b, :L]), None, Cs, k, None, oracle.KIND_LEX,
                     [int(p) for p in pos[b, :n]], [float(s) for s in sc[b, :n]], f"{ctx} b={b}",
                     preceding=preceding)
    return kinds


@pytest.mark.parametrize("L,d,k,tau", [(300, 256, 8, 0.5), (2100, 128, 64, 0.45), (700, 520, 16, 0.55)])
def test_embedding_fallback(L, d, k, tau):
    cfg = small_config(B=8, L=L, d=d, k=k, n_max=3, seed=140 + L % 97, V=60, forced_every=2)
    x = make_inputs(cfg, with_verify=False)
    E_bits = emb_table(cfg.V + 8, d, clusters=6, seed=L, zero_rows=(7,))   # ids reach V (c.17)
    kinds = run_and_check(cfg, x, E_bits, tau, k, f"L={L}")
    assert oracle.KIND_SEM in kinds and oracle.KIND_LEX in kinds, kinds


def test_embedding_fallback_preceding():
    """The embedding set ranked with Eq. (6)'s alignment (rows j-1, query row L-2)."""
    cfg = small_config(B=8, L=700, d=256, k=8, n_max=3, seed=147, V=60, forced_every=2)
    x = make_inputs(cfg, with_verify=False)
    E_bits = emb_table(cfg.V + 8, 256, clusters=6, seed=9, zero_rows=(7,))
    kinds = run_and_check(cfg, x, E_bits, 0.5, 8, "preceding", preceding=True)
    assert oracle.KIND_SEM in kinds and oracle.KIND_LEX in kinds, kinds


def test_embedding_fallback_nothing_kept():
    """tau above every cosine: each lexical miss is an autoregressive step."""
    cfg = small_config(B=4, L=400, d=128, k=8, n_max=3, seed=151, V=60, forced_every=1)
    x = make_inputs(cfg, with_verify=False)
    E_bits = emb_table(cfg.V + 8, 128, clusters=6, seed=3)
    kinds = run_and_check(cfg, x, E_bits, 1.01, 8, "tau>1")
    assert set(kinds) <= {oracle.KIND_NONE, oracle.KIND_LEX} and oracle.KIND_NONE in kinds


def test_embedding_fallback_two_pieces():
    """A context longer than one compaction piece (32768 positions)."""
    cfg = small_config(B=2, L=40000, d=64, k=16, n_max=3, seed=152, V=40, forced_every=1)
    x = make_inputs(cfg, with_verify=False)
    E_bits = emb_table(cfg.V + 8, 64, clusters=5, seed=9)
    kinds = run_and_check(cfg, x, E_bits, 0.6, 16, "L=40000")
    assert oracle.KIND_SEM in kinds


def test_embedding_fallback_out_of_range_tokens():
    """Token ids outside [0, V) have a zero embedding (cosine 0): kept for
    tau <= 0, dropped for tau > 0."""
    cfg = small_config(B=3, L=500, d=128, k=64, n_max=3, seed=153, V=50, forced_every=1)
    x = make_inputs(cfg, with_verify=False)
    V = cfg.V + 8   # table rows; generated ids reach cfg.V
    rng = np.random.default_rng(4)
    for b in range(cfg.B):
        L = int(x["lens"][b])
        idx = rng.choice(L - 1, size=12, replace=False)
        x["tokens"][b, idx] = np.where(rng.random(12) < 0.5, -3, V + 7)
    E_bits = emb_table(V, 128, clusters=5, seed=11)
    # the oracle sees the same ids mapped to an extra zero row
    E_ext = np.concatenate([E_bits, np.zeros((1, 128), dtype=np.uint16)])
    xm = dict(x)
    xm["tokens"] = np.where((x["tokens"] < 0) | (x["tokens"] >= V), V, x["tokens"])
    for tau in (-0.2, 0.5):
        E = oracle.bf16_bits_to_f64(E_ext)
        assert margin_ok(E, xm["tokens"], x["lens"], tau)
        tokens, lens = dev_i32(x["tokens"]), dev_i32(x["lens"])
        cp, cc, mn = adapld.lexical_match(tokens, lens, cfg.n_max)
        pos, sc, cnt, kind = adapld.semantic_topk_embed(dev_bf16(x["bank"]), tokens, lens, cp, cc, dev_bf16(E_bits),
                                                        64, tau)
        torch.cuda.synchronize()
        cnt, kind, pos = cnt.cpu().numpy(), kind.cpu().numpy(), pos.cpu().numpy()
        for b in range(cfg.B):
            L = int(x["lens"][b])
            # the lexical match runs on the original ids (they differ from every real id)
            _, C = oracle.lexical_match(x["tokens"][b, :L], cfg.n_max)
            ekind, Cs = oracle.embedding_fallback(xm["tokens"][b, :L], E, C, tau)
            assert int(kind[b]) == ekind, (tau, b)
            if ekind == oracle.KIND_SEM and len(Cs) <= 64:
                assert sorted(int(p) for p in pos[b, :int(cnt[b])]) == sorted(Cs), (tau, b)


@pytest.mark.parametrize("tau", [0.5, 0.25, 0.0, -0.5])
def test_embedding_fallback_threshold_equality(tau):
    """Eq. (4) keeps cos >= tau.  Embeddings of four +-1 entries among the
    first 8 dimensions (norm 2) have cosines that are multiples of 1/4, exact
    in fp32 and float64, so tau lands exactly on cosines present and the
    kind and the candidate set must follow the >= rule bit for bit."""
    cfg = small_config(B=8, L=600, d=128, k=64, n_max=3, seed=161, V=60, forced_every=1)
    x = make_inputs(cfg, with_verify=False)
    rng = np.random.default_rng(21)
    V = cfg.V + 8
    E = np.zeros((V, 128))
    for r in range(V):
        E[r, rng.choice(8, size=4, replace=False)] = rng.choice([-1.0, 1.0], size=4)
    E_bits = f32_to_bf16_bits(E.astype(np.float32))
    on = 0
    for b in range(cfg.B):
        L = int(x["lens"][b])
        s = oracle.cosine_rows(E, x["tokens"][b, :L - 1], E[int(x["tokens"][b, L - 1])])
        on += int(np.sum(s == tau))
    assert on > 0, "no cosine sits exactly on tau"
    kinds = run_and_check(cfg, x, E_bits, tau, 64, f"tau={tau} exact", exact=True)
    assert oracle.KIND_SEM in kinds or oracle.KIND_NONE in kinds


@pytest.mark.parametrize("V", [1 << 20, (1 << 20) + 5])
def test_embedding_fallback_vocabulary_edge(V):
    """The distinct-token path takes vocabularies of up to 2^20 tokens (a
    bitmap of them in LDS), larger ones the per-position path: both around
    that size, with ids at the last row of the table and just past it."""
    cfg = small_config(B=4, L=600, d=64, k=64, n_max=3, seed=171, V=50, forced_every=1)
    x = make_inputs(cfg, with_verify=False)
    small = emb_table(cfg.V + 8, 64, clusters=5, seed=13)
    E_bits = np.zeros((V, 64), dtype=np.uint16)
    E_bits[:small.shape[0]] = small
    E_bits[V - 1] = small[3]          # the last id is a near twin of id 3
    rng = np.random.default_rng(5)
    for b in range(cfg.B):
        L = int(x["lens"][b])
        idx = rng.choice(L - 1, size=16, replace=False)
        x["tokens"][b, idx[:8]] = V - 1
        x["tokens"][b, idx[8:]] = V   # outside the table: zero embedding
    tokens, lens = dev_i32(x["tokens"]), dev_i32(x["lens"])
    cp, cc, mn = adapld.lexical_match(tokens, lens, cfg.n_max)
    # the oracle sees the ids past the table mapped to an extra zero row
    E = oracle.bf16_bits_to_f64(np.concatenate([E_bits, np.zeros((1, 64), dtype=np.uint16)]))
    taus = [t for t in (0.6, 0.55, 0.65) if margin_ok(E, x["tokens"], x["lens"], t)][:1] + \
        [t for t in (-0.13, -0.27, -0.41, -0.07) if margin_ok(E, x["tokens"], x["lens"], t)][:1]
    assert len(taus) == 2, "no threshold clear of the cosines present"
    for tau in taus:
        pos, sc, cnt, kind = adapld.semantic_topk_embed(dev_bf16(x["bank"]), tokens, lens, cp, cc,
                                                        dev_bf16(E_bits), 64, tau)
        torch.cuda.synchronize()
        cnt, kind, pos = cnt.cpu().numpy(), kind.cpu().numpy(), pos.cpu().numpy()
        sem = 0
        for b in range(cfg.B):
            L = int(x["lens"][b])
            M = x["tokens"][b, :L]
            _, C = oracle.lexical_match(M, cfg.n_max)
            ekind, Cs = oracle.embedding_fallback(M, E, C, tau)
            assert int(kind[b]) == ekind, (V, tau, b)
            if ekind == oracle.KIND_SEM:
                sem += 1
                if len(Cs) <= 64:
                    assert sorted(int(p) for p in pos[b, :int(cnt[b])]) == sorted(Cs), (V, tau, b)
        assert sem > 0, (V, tau)
