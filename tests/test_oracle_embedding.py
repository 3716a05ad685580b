"""Pins of the oracle's token-embedding fallback (Sec. 3.3, Eqs. (4)-(5))."""
import json
import os

import numpy as np
import pytest
from scipy.spatial.distance import cosine as scipy_cosine_distance

import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "embedding_cases.json")


def test_golden_cases():
    g = json.load(open(GOLDEN))
    E = np.asarray(g["emb"], dtype=np.float64)
    assert len(g["cases"]) >= 6
    for c in g["cases"]:
        kind, pos = oracle.embedding_fallback(c["tokens"], E, c["cand"], c["tau"])
        assert kind == c["kind"] and pos == c["pos"], c["why"]


def _scipy_cos(u, v):
    if not np.any(u) or not np.any(v):
        return 0.0
    return 1.0 - scipy_cosine_distance(u, v)


@pytest.mark.parametrize("seed", range(12))
def test_against_scipy_cosine(seed):
    rng = np.random.default_rng(seed)
    V, d = int(rng.integers(3, 30)), int(rng.integers(2, 40))
    E = rng.standard_normal((V, d))
    E[rng.integers(0, V)] = 0.0                        # one zero row
    M = rng.integers(0, V, size=int(rng.integers(2, 60)))
    tau = float(rng.uniform(-0.5, 0.6))
    kind, pos = oracle.embedding_fallback(M, E, [], tau)
    a = E[M[-1]]
    want = [j for j in range(len(M) - 1) if _scipy_cos(E[M[j]], a) >= tau + 1e-12 or
            (abs(_scipy_cos(E[M[j]], a) - tau) <= 1e-12 and j in pos)]
    assert pos == want
    assert kind == (oracle.KIND_SEM if want else oracle.KIND_NONE)


def test_properties():
    rng = np.random.default_rng(3)
    for _ in range(200):
        V, d = int(rng.integers(2, 12)), int(rng.integers(1, 8))
        E = rng.standard_normal((V, d))
        M = rng.integers(0, V, size=int(rng.integers(1, 40)))
        L = len(M)
        lo, hi = sorted(rng.uniform(-1, 1, size=2))
        _, p_lo = oracle.embedding_fallback(M, E, [], lo)
        _, p_hi = oracle.embedding_fallback(M, E, [], hi)
        assert set(p_hi) <= set(p_lo)                                  # monotone in tau
        assert oracle.embedding_fallback(M, E, [], -1.0 - 1e-9)[1] == list(range(max(L - 1, 0)))
        assert oracle.embedding_fallback(M, E, [], 1.0 + 1e-9)[1] == []
        assert all(j < L - 1 for j in p_lo)
        # a decision belongs to the token: equal tokens are kept or dropped together
        for j in range(L - 1):
            for k in range(L - 1):
                if M[j] == M[k]:
                    assert (j in p_lo) == (k in p_lo)
        # every earlier copy of the anchor token has cosine 1 (a lexical hit
        # would have caught it, but the fallback's definition keeps it too)
        for j in range(L - 1):
            if M[j] == M[-1] and np.any(E[M[-1]]):
                assert j in p_lo
        # the backoff rule: a lexical list passes through untouched
        cand = sorted(set(int(c) for c in rng.integers(0, max(L - 1, 1), size=3)))
        assert oracle.embedding_fallback(M, E, cand, hi) == (oracle.KIND_LEX, cand)
