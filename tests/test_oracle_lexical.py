"""Pins for the oracle's lexical anchoring (Sec. 3.3, exact-match candidate set).

Each check comes from outside the oracle: hand-worked fixtures, an exhaustive
brute force by a different formulation (longest common suffix per position),
the paper's single-token equation, structure planted by the input generator,
and the nesting of n-gram levels.
"""
import itertools
import json
import os

import numpy as np
import pytest

from oracle import lexical_match
from paper_2606_05742_amd.synth import CONFIGS, make_inputs, small_config

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def test_golden_cases():
    d = json.load(open(os.path.join(GOLD, "lexical_cases.json")))
    for c in d["cases"]:
        n, C = lexical_match(np.array(c["tokens"], dtype=np.int32), c["n_max"])
        assert (n, C) == (c["n_star"], c["cand"]), c


def _lcs_brute(M, n_max):
    """Longest common suffix of M[:j+1] and M for every j <= L-2, by string reversal."""
    L = len(M)
    best, lcs = 0, []
    full = M[::-1]
    for j in range(L - 1):
        pre = M[: j + 1][::-1]
        m = len(os.path.commonprefix([list(pre), list(full)]))
        lcs.append(min(m, n_max))
    best = max(lcs) if lcs else 0
    if best == 0:
        return 0, []
    return best, [j for j, m in enumerate(lcs) if m == best]


@pytest.mark.parametrize("n_max", [1, 2, 3, 4])
def test_exhaustive_ternary(n_max):
    # every context over a 3-token vocabulary with L <= 8 (9 for n_max <= 2)
    top = 9 if n_max <= 2 else 8
    for L in range(0, top + 1):
        for M in itertools.product(range(3), repeat=L):
            got = lexical_match(np.array(M, dtype=np.int32), n_max)
            assert got == _lcs_brute(list(M), n_max), (M, n_max)


def test_single_token_is_paper_equation():
    # n_max = 1 is the paper's set {j : M_j = a_i}, j before the anchor.
    rng = np.random.default_rng(7)
    for _ in range(200):
        L = int(rng.integers(1, 60))
        M = rng.integers(0, 6, size=L).astype(np.int32)
        n, C = lexical_match(M, 1)
        ref = np.nonzero(M[:-1] == M[-1])[0].tolist()
        assert C == ref
        assert n == (1 if ref else 0)


def test_levels_nest():
    # j in C_n implies j in C_{n-1}: the level-n set is a subset of level n-1.
    rng = np.random.default_rng(3)
    for _ in range(300):
        L = int(rng.integers(2, 40))
        M = rng.integers(0, 3, size=L).astype(np.int32)
        for n in range(2, 6):
            ns, C = lexical_match(M, n)
            if ns == n:
                ns1, C1 = lexical_match(M, n - 1)
                assert ns1 == n - 1 and set(C) <= set(C1)


def _planted(log, n_max):
    """(context length, expected candidate) pairs planted by copy events.

    Truncating the context right after the copied token t+off (off >= n_max-1)
    makes its last n_max tokens a copy of the n_max tokens ending at s+off,
    provided no later event overwrote either range.
    """
    out = []
    for e, (s, t, ln) in enumerate(log):
        for off in range(n_max - 1, ln):
            src_rng = (s + off - n_max + 1, s + off)
            dst_rng = (t + off - n_max + 1, t + off)
            clean = all(not (t2 <= b and a < t2 + l2)
                        for (s2, t2, l2) in log[e + 1:] for a, b in (src_rng, dst_rng))
            if clean:
                out.append((t + off + 1, s + off))
    return out


def test_planted_copies_are_found():
    found = 0
    cfg = small_config(B=8, L=200, V=2000, copy_frac=0.5, span=(6, 20), seed=5)
    x = make_inputs(cfg, with_bank=False, with_verify=False)
    for b in range(cfg.B):
        M = x["tokens"][b]
        for Lp, j in _planted(x["copy_logs"][b], cfg.n_max):
            n, C = lexical_match(M[:Lp], cfg.n_max)
            assert n == cfg.n_max and j in C, (b, Lp, j)
            found += 1
    assert found >= 50


def test_forced_sequences_miss():
    cfg = CONFIGS["b16_l8192_gqa32x8"]
    x = make_inputs(cfg, with_bank=False, with_verify=False, seqs=[3, 7])
    for i in range(2):
        n, C = lexical_match(x["tokens"][i], cfg.n_max)
        assert (n, C) == (0, [])
