"""Pins for the oracle's draft-tree construction (Sec. 3.5 reuse construction, Sec. 3.6 tree).

Checks from outside the oracle: hand-enumerated trees, the paper's main-path
formula in its own 1-based indexing, the branch-dedup rule, structural
invariants, and an ancestor relation computed by transitive closure of the
parent links (independent of the oracle's parent walk).
"""
import json
import os

import numpy as np
import pytest

from oracle import KIND_LEX, KIND_NONE, KIND_SEM, bf16_bits_to_f64, build_draft_tree, lexical_match, semantic_topk
from paper_2606_05742_amd.synth import make_inputs, small_config

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def closure_mask(parent):
    """Ancestor-or-self relation by Warshall's transitive closure of child -> parent edges."""
    T = len(parent)
    R = np.eye(T, dtype=bool)
    for u, p in enumerate(parent):
        if p >= 0:
            R[u, p] = True
    for m in range(T):
        R |= np.outer(R[:, m], R[m, :])
    return R


def test_golden_cases():
    d = json.load(open(os.path.join(GOLD, "tree_cases.json")))
    for c in d["cases"]:
        t = build_draft_tree(np.array(c["tokens"], dtype=np.int32), c["kind"], c["ranked"], c["W"], c["S"])
        for key in ("token", "parent", "depth", "src"):
            assert t[key] == c[key], (key, c)
        T = len(c["token"])
        ref = np.zeros((T, T), dtype=bool)
        for u, anc in enumerate(c["anc"]):
            ref[u, anc] = True
        np.testing.assert_array_equal(t["mask"], ref)


def _trees(seed, **kw):
    cfg = small_config(seed=seed, **kw)
    x = make_inputs(cfg, with_verify=False)
    for b in range(cfg.B):
        L = int(x["lens"][b])
        M = x["tokens"][b, :L]
        n, C = lexical_match(M, cfg.n_max)
        H = bf16_bits_to_f64(x["bank"][b, :L])
        kind, pos, sc = semantic_topk(H, None, C, cfg.k, None)
        yield cfg, M, C, kind, pos, build_draft_tree(M, kind, pos, cfg.W, cfg.S)


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_invariants(seed):
    for cfg, M, C, kind, pos, t in _trees(seed, B=10, L=150, V=60, W=4, S=6, k=10, forced_every=2):
        L = len(M)
        T = t["T"]
        assert T <= cfg.W * (cfg.S + 1)
        heads = [u for u in range(T) if t["depth"][u] == 0]
        firsts = [t["token"][u] for u in heads]
        assert len(set(firsts)) == len(firsts) <= cfg.W
        for u in range(T):
            assert t["token"][u] == M[t["src"][u]]
            assert 0 < t["src"][u] <= L - 1
            if t["depth"][u] > 0:
                p = t["parent"][u]
                assert p == u - 1 and t["src"][u] == t["src"][p] + 1
                assert t["depth"][u] == t["depth"][p] + 1
            else:
                assert t["parent"][u] == -1
        np.testing.assert_array_equal(t["mask"], closure_mask(t["parent"]))
        if kind == KIND_NONE:
            assert T == 0
        else:
            assert T >= 1


@pytest.mark.parametrize("seed", [4, 5])
def test_main_path_and_dedup(seed):
    """With a lexical hit, branch 0 is the main copy path M_{j*+1 : j*+l_i},
    l_i = min(l_m, |M| - j*) in the paper's 1-based positions, l_m = S + 1;
    no other branch starts with the main path's first token."""
    seen = 0
    for cfg, M, C, kind, pos, t in _trees(seed, B=12, L=150, V=40, W=4, S=6, k=10):
        if kind != KIND_LEX:
            continue
        seen += 1
        L = len(M)
        j1 = pos[0] + 1              # 1-based position of the selected anchor
        l_i = min(cfg.S + 1, L - j1)
        main = [int(M[p - 1]) for p in range(j1 + 1, j1 + l_i + 1)]   # 1-based -> 0-based read
        n0 = len(t["branches"][0])
        assert t["token"][:n0] == main
        others = [t["token"][u] for u in range(n0, t["T"]) if t["depth"][u] == 0]
        assert main[0] not in others
    assert seen >= 3


def test_fewer_distinct_successors_than_width():
    M = np.array([4, 9, 4, 9, 4, 9, 4], dtype=np.int32)
    t = build_draft_tree(M, KIND_LEX, [0, 2, 4], W=4, S=2)
    assert len(t["branches"]) == 1 and t["token"] == [9, 4, 9]
