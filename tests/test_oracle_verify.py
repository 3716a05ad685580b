"""Pins for the oracle's tree-masked verify attention (Sec. 3.6, tree attention).

Checks from outside the oracle: a hand-worked case, PyTorch's
scaled_dot_product_attention (CPU, float64) both with the tree as a boolean
mask and as independent per-path causal attention, the closed form of plain
decode attention for a one-node tree, and a mask-leak probe.
"""
import json
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import build_draft_tree, tree_verify_attn, KIND_LEX

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def test_golden_cases():
    d = json.load(open(os.path.join(GOLD, "verify_cases.json")))
    for c in d["cases"]:
        a = {k: np.array(c[k], dtype=np.float64) for k in ("Q", "Kc", "Vc", "Kt", "Vt")}
        par = c["parent"]
        T = len(par)
        mask = np.zeros((T, T), dtype=bool)
        for u in range(T):
            v = u
            while v >= 0:
                mask[u, v] = True
                v = par[v]
        O, LSE = tree_verify_attn(a["Q"], a["Kc"], a["Vc"], a["Kt"], a["Vt"], mask, c["L"], c["scale"])
        np.testing.assert_allclose(O, c["O"], rtol=0, atol=1e-12)
        np.testing.assert_allclose(LSE, c["LSE"], rtol=0, atol=1e-12)


def _random_tree(rng, T, branches):
    """Chains (branch-major), as the draft tree lays nodes out."""
    cuts = sorted(rng.choice(np.arange(1, T), size=branches - 1, replace=False).tolist()) if branches > 1 else []
    parent, start = [], 0
    for end in cuts + [T]:
        for u in range(start, end):
            parent.append(-1 if u == start else u - 1)
        start = end
    mask = np.zeros((T, T), dtype=bool)
    for u in range(T):
        v = u
        while v >= 0:
            mask[u, v] = True
            v = parent[v]
    return parent, mask


def _case(seed, T=9, Hq=8, Hkv=2, D=16, L=23, branches=3):
    rng = np.random.default_rng(seed)
    Q = rng.standard_normal((T, Hq, D))
    Kc = rng.standard_normal((Hkv, L + 5, D))
    Vc = rng.standard_normal((Hkv, L + 5, D))
    Kt = rng.standard_normal((T, Hkv, D))
    Vt = rng.standard_normal((T, Hkv, D))
    parent, mask = _random_tree(rng, T, branches)
    return Q, Kc, Vc, Kt, Vt, parent, mask, L


@pytest.mark.parametrize("seed", range(4))
def test_matches_torch_sdpa_with_tree_mask(seed):
    Q, Kc, Vc, Kt, Vt, parent, mask, L = _case(seed)
    T, Hq, D = Q.shape
    Hkv = Kc.shape[0]
    scale = 0.37
    O, LSE = tree_verify_attn(Q, Kc, Vc, Kt, Vt, mask, L, scale)
    t = torch.from_numpy
    # keys per kv head: context (L) then every tree node (T); GQA by repeating kv heads
    K = torch.cat([t(Kc[:, :L]), t(Kt).permute(1, 0, 2)], dim=1)      # (Hkv, L+T, D)
    V = torch.cat([t(Vc[:, :L]), t(Vt).permute(1, 0, 2)], dim=1)
    K = K.repeat_interleave(Hq // Hkv, dim=0)
    V = V.repeat_interleave(Hq // Hkv, dim=0)
    q = t(Q).permute(1, 0, 2)                                            # (Hq, T, D)
    am = torch.cat([torch.ones(T, L, dtype=torch.bool), t(mask)], dim=1)  # (T, L+T)
    ref = F.scaled_dot_product_attention(q, K, V, attn_mask=am, scale=scale)
    np.testing.assert_allclose(O, ref.permute(1, 0, 2).numpy(), rtol=0, atol=1e-12)
    logits = torch.einsum("htd,hkd->htk", q, K) * scale
    lse = torch.logsumexp(logits.masked_fill(~am, float("-inf")), dim=-1)
    np.testing.assert_allclose(LSE, lse.numpy(), rtol=0, atol=1e-12)


@pytest.mark.parametrize("seed", range(3))
def test_matches_per_path_causal_attention(seed):
    """Each node's output equals the last row of ordinary causal attention over
    the context followed by the path root -> node."""
    Q, Kc, Vc, Kt, Vt, parent, mask, L = _case(seed, T=8, branches=2)
    T, Hq, D = Q.shape
    Hkv = Kc.shape[0]
    G = Hq // Hkv
    scale = 1.0 / np.sqrt(D)
    O, LSE = tree_verify_attn(Q, Kc, Vc, Kt, Vt, mask, L, scale)
    for u in range(T):
        path = []
        v = u
        while v >= 0:
            path.append(v)
            v = parent[v]
        path = path[::-1]
        n = L + len(path)
        for h in range(Hq):
            g = h // G
            keys = torch.cat([torch.from_numpy(Kc[g, :L]), torch.from_numpy(Kt[path, g])])
            vals = torch.cat([torch.from_numpy(Vc[g, :L]), torch.from_numpy(Vt[path, g])])
            qs = torch.zeros(n, D, dtype=torch.float64)
            qs[L:] = torch.from_numpy(Q[path, h])
            out = F.scaled_dot_product_attention(qs[None], keys[None], vals[None], is_causal=True, scale=scale)
            np.testing.assert_allclose(O[u, h], out[0, -1].numpy(), rtol=0, atol=1e-12)


def test_single_node_is_decode_attention():
    rng = np.random.default_rng(5)
    D, L = 32, 40
    Q = rng.standard_normal((1, 2, D))
    Kc = rng.standard_normal((1, L, D))
    Vc = rng.standard_normal((1, L, D))
    Kt = rng.standard_normal((1, 1, D))
    Vt = rng.standard_normal((1, 1, D))
    O, LSE = tree_verify_attn(Q, Kc, Vc, Kt, Vt, np.ones((1, 1), bool), L, 0.2)
    for h in range(2):
        K = np.concatenate([Kc[0], Kt[0]])
        V = np.concatenate([Vc[0], Vt[0]])
        z = 0.2 * K @ Q[0, h]
        w = np.exp(z) / np.exp(z).sum()
        np.testing.assert_allclose(O[0, h], w @ V, rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(LSE[h, 0], np.log(np.exp(z).sum()), rtol=1e-12)


def test_mask_leak_probe():
    """A non-ancestor key aligned with a node's query must not move that node's output."""
    Q, Kc, Vc, Kt, Vt, parent, mask, L = _case(7, T=9, branches=3)
    O, _ = tree_verify_attn(Q, Kc, Vc, Kt, Vt, mask, L, 0.25)
    u = 8
    others = [v for v in range(9) if not mask[u, v]]
    assert others
    Kt2, Vt2 = Kt.copy(), Vt.copy()
    for v in others:
        Kt2[v, :] = 50.0 * Q[u, 0]
        Vt2[v, :] = 1e3
    O2, _ = tree_verify_attn(Q, Kc, Vc, Kt2, Vt2, mask, L, 0.25)
    np.testing.assert_array_equal(O[u], O2[u])
    # and the probe is live: the same keys do move a node that sees them
    w = others[0]
    assert not np.allclose(O[w], O2[w])
