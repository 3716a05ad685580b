"""Pins of the oracle's paper-faithful draft construction (Sec. 3.5,
Eqs. (8)-(15); Algorithm 1)."""
import json
import os

import numpy as np
import pytest
from scipy.spatial.distance import cosine as scipy_cosine_distance

import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "tree_paper_cases.json")


def test_golden_cases():
    cases = json.load(open(GOLDEN))["cases"]
    assert len(cases) >= 12
    for c in cases:
        L = len(c["tokens"])
        H = np.asarray(c["H"], dtype=np.float64) if "H" in c else np.eye(max(L, 1))
        emb = np.asarray(c["emb"], dtype=np.float64) if "emb" in c else None
        t = oracle.build_draft_tree_paper(c["tokens"], H, c["kind"], c["ranked"], c["top"], c["W"], c["S"],
                                          succ_mode=c.get("succ_mode", 0), emb=emb, tau=c.get("tau"))
        for key in ("token", "parent", "depth", "src"):
            assert t[key] == c[key], (c["why"], key, t[key])


def _cos(u, v):
    if not np.any(u) or not np.any(v):
        return 0.0
    return 1.0 - scipy_cosine_distance(u, v)


@pytest.mark.parametrize("seed", range(60))
def test_against_brute_force(seed):
    rng = np.random.default_rng(seed)
    V = int(rng.integers(2, 8))
    L = int(rng.integers(2, 50))
    M = rng.integers(0, V, size=L)
    H = rng.standard_normal((L, int(rng.integers(1, 6))))
    kind = int(rng.integers(0, 3))
    j = int(rng.integers(0, L - 1))
    ranked = [j] if kind else []
    top = list(rng.integers(-1, V + 2, size=int(rng.integers(0, 8))))
    W, S = int(rng.integers(1, 6)), int(rng.integers(0, 5))
    mode = int(rng.integers(0, 2))
    # half the cases carry an embedding table of V + 1 rows (so token V + 1
    # lies outside it), with small integer entries: equal cosines are exact
    emb = rng.integers(-2, 3, size=(V + 1, 2)).astype(np.float64) if seed % 2 else None
    tau = float(rng.choice([-0.5, 0.0, 0.5, 0.8])) if emb is not None else None
    t = oracle.build_draft_tree_paper(M, H, kind, ranked, top, W, S, succ_mode=mode, emb=emb, tau=tau)
    # the same tree built step by step from the equations
    want = []   # (token, parent, depth, src)
    if kind:
        if kind == oracle.KIND_LEX:
            l = min(S + 1, L - 1 - j)
            for dd in range(l):
                want.append((int(M[j + 1 + dd]), -1 if dd == 0 else len(want) - 1, dd, j + 1 + dd))
        excl = {int(M[j + 1])} if kind == oracle.KIND_LEX and L - 1 - j > 0 else set()
        seen = []
        for b in top:
            b = int(b)
            if b < 0 or b in seen or b in excl or len(seen) == W:
                continue
            seen.append(b)
        for b in seen:
            want.append((b, -1, 0, -1))
            u = len(want) - 1
            if mode == 1 and kind == oracle.KIND_LEX:
                continue   # Algorithm 1: no successor drafting in the strict branch
            occ = [tt for tt in range(1, L - 1) if int(M[tt]) == b]
            if not occ and emb is not None:
                eb = emb[b] if b < emb.shape[0] else np.zeros(2)
                occ = [tt for tt in range(1, L - 1)
                       if _cos(emb[int(M[tt])] if int(M[tt]) < emb.shape[0] else np.zeros(2), eb) >= tau]
            best, best_s = None, None
            for tt in occ:
                sc = _cos(H[tt - 1], H[j])
                if best is None or sc > best_s + 1e-12:
                    best, best_s = tt, sc
            if best is not None:
                want.append((int(M[best + 1]), u, 1, best + 1))
    assert [t["token"], t["parent"], t["depth"], t["src"]] == [[w[i] for w in want] for i in range(4)]


def test_invariants():
    rng = np.random.default_rng(1)
    for _ in range(300):
        L = int(rng.integers(2, 40))
        M = rng.integers(0, 5, size=L)
        H = rng.standard_normal((L, 3))
        kind = int(rng.integers(1, 3))
        j = int(rng.integers(0, L - 1))
        W, S = int(rng.integers(1, 5)), int(rng.integers(0, 4))
        top = list(rng.integers(0, 6, size=6))
        mode = int(rng.integers(0, 2))
        t = oracle.build_draft_tree_paper(M, H, kind, [j], top, W, S, succ_mode=mode)
        assert t["T"] <= (S + 1) + 2 * W
        if mode == 1 and kind == oracle.KIND_LEX:   # Algorithm 1: no successor after a lexical anchor
            assert all(t["src"][t["parent"][u]] != -1 for u in range(t["T"]) if t["parent"][u] >= 0)
        branch_tokens = [t["token"][u] for u in range(t["T"]) if t["src"][u] == -1]
        assert len(branch_tokens) == len(set(branch_tokens)) <= W
        if kind == oracle.KIND_LEX:
            assert int(M[j + 1]) not in branch_tokens
        for u in range(t["T"]):
            if t["src"][u] >= 0:
                assert t["token"][u] == int(M[t["src"][u]])
            if t["depth"][u] == 1 and t["src"][t["parent"][u]] == -1:   # a successor
                assert int(M[t["src"][u] - 1]) == t["token"][t["parent"][u]]
        # the mask is the ancestor-or-self relation of the parents
        for u in range(t["T"]):
            anc = set()
            v = u
            while v != -1:
                anc.add(v)
                v = t["parent"][v]
            assert set(np.nonzero(t["mask"][u])[0]) == anc
