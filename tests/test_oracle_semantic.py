"""Pins for the oracle's backoff + reranking (Sec. 3.3 backoff rule, Sec. 3.4 scores).

Checks from outside the oracle: hand-worked fixtures, SciPy's cosine distance,
selection by repeated argmax (a different algorithm from the oracle's sort),
the backoff invariant, exact ties of duplicated rows, tau limits, and the
semantic neighbour the input generator plants in forced-miss sequences.
"""
import json
import os

import numpy as np
import pytest
from scipy.spatial.distance import cosine as scipy_cosine_distance

from oracle import (KIND_LEX, KIND_NONE, KIND_SEM, bf16_bits_to_f64, cosine_rows,
                    lexical_match, semantic_topk)
from paper_2606_05742_amd.synth import CONFIGS, f32_to_bf16_bits, make_inputs, small_config

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def test_golden_cases():
    d = json.load(open(os.path.join(GOLD, "semantic_cases.json")))
    for c in d["cases"]:
        H = np.array(d["banks"][c["bank"]], dtype=np.float64)
        q = None if c["query"] is None else np.array(c["query"], dtype=np.float64)
        kind, pos, sc = semantic_topk(H, q, c["cand"], c["k"], c["tau"], preceding=c.get("preceding", False))
        assert kind == c["kind"] and pos == c["pos"], c
        np.testing.assert_allclose(sc, c["score"], rtol=0, atol=1e-15)


def test_bf16_decode_exact():
    x = np.array([0.0, -0.0, 1.0, -2.5, 3.140625, 65280.0, 1e-38], dtype=np.float32)
    bits = f32_to_bf16_bits(x)
    y = bf16_bits_to_f64(bits)
    assert y[2] == 1.0 and y[3] == -2.5 and y[4] == 3.140625 and y[5] == 65280.0
    # every bf16 value round-trips through float32 unchanged
    allbits = np.arange(0, 65536, dtype=np.uint16)
    with np.errstate(invalid="ignore"):
        f = bf16_bits_to_f64(allbits)
    fin = np.isfinite(f)
    np.testing.assert_array_equal(f32_to_bf16_bits(f[fin].astype(np.float32)), allbits[fin])


def test_cosine_matches_scipy():
    rng = np.random.default_rng(0)
    H = rng.standard_normal((20, 37))
    q = rng.standard_normal(37)
    got = cosine_rows(H, range(20), q)
    ref = np.array([1.0 - scipy_cosine_distance(H[r], q) for r in range(20)])
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-14)


def _argmax_select(scores, rows, k):
    """Top k by repeated argmax; np.argmax returns the first (lowest-position) maximum."""
    s = np.array(scores, dtype=np.float64)
    out = []
    for _ in range(min(k, len(rows))):
        i = int(np.argmax(s))
        out.append(int(rows[i]))
        s[i] = -np.inf
    return out


@pytest.mark.parametrize("seed", range(5))
def test_selection_by_repeated_argmax(seed):
    rng = np.random.default_rng(seed)
    L, d = 50, 16
    # few distinct rows so that many scores tie exactly
    base = rng.integers(-2, 3, size=(6, d)).astype(np.float64)
    H = base[rng.integers(0, 6, size=L)]
    q = H[L - 1]
    rows = list(range(L - 1))
    s = [float(H[r] @ q / (np.linalg.norm(H[r]) * np.linalg.norm(q))) if np.linalg.norm(H[r]) > 0 else 0.0
         for r in rows]
    for k in (1, 5, 17, 64):
        kind, pos, _ = semantic_topk(H, None, [], k, None)
        assert kind == KIND_SEM and pos == _argmax_select(s, rows, k)
        cand = sorted(rng.choice(L - 1, size=9, replace=False).tolist())
        kind, pos, _ = semantic_topk(H, None, cand, k, None)
        assert kind == KIND_LEX and pos == _argmax_select([s[c] for c in cand], cand, k)


def test_backoff_invariant_and_sizes():
    cfg = small_config(B=12, L=120, V=400, forced_every=3, seed=9)
    x = make_inputs(cfg, with_verify=False)
    kinds = []
    for b in range(cfg.B):
        L = int(x["lens"][b])
        n, C = lexical_match(x["tokens"][b, :L], cfg.n_max)
        H = bf16_bits_to_f64(x["bank"][b, :L])
        kind, pos, sc = semantic_topk(H, None, C, cfg.k, None)
        kinds.append(kind)
        # the fallback fires iff the lexical set is empty
        assert (kind in (KIND_SEM, KIND_NONE)) == (len(C) == 0)
        if kind == KIND_LEX:
            assert len(pos) == min(cfg.k, len(C)) and set(pos) <= set(C)
        else:
            # tau disabled: the fallback keeps min(k, L-1) rows
            assert len(pos) == min(cfg.k, L - 1)
        assert all(a >= b_ for a, b_ in zip(sc, sc[1:]))
        # tau above any cosine empties the fallback; it never empties a lexical hit
        k2, p2, _ = semantic_topk(H, None, C, cfg.k, 1.01)
        assert (k2 == KIND_NONE) == (len(C) == 0)
    assert KIND_LEX in kinds and KIND_SEM in kinds


def test_zero_norm_rows_score_zero():
    H = np.array([[0.0, 0.0], [1.0, 0.0], [0.0, 0.0], [-1.0, 0.0], [0.0, 0.0]])
    kind, pos, sc = semantic_topk(H, np.array([1.0, 0.0]), [], 4, None)
    assert pos == [1, 0, 2, 3] and sc == [1.0, 0.0, 0.0, -1.0]
    kind, pos, sc = semantic_topk(H, np.array([0.0, 0.0]), [], 3, None)
    assert pos == [0, 1, 2] and sc == [0.0, 0.0, 0.0]


def _copy_family(log, src):
    fam = {src}
    changed = True
    while changed:
        changed = False
        for s, t, ln in log:
            for i in range(ln):
                a, b = s + i, t + i
                if (a in fam) != (b in fam):
                    fam |= {a, b}
                    changed = True
    return fam


def test_planted_neighbour_ranks_first():
    cfg = CONFIGS["b16_l8192_gqa32x8"]
    x = make_inputs(cfg, with_verify=False, seqs=[3, 11])
    for i in range(2):
        L = int(x["lens"][i])
        tok, src = x["forced"][i]
        n, C = lexical_match(x["tokens"][i, :L], cfg.n_max)
        assert C == []
        H = bf16_bits_to_f64(x["bank"][i, :L])
        kind, pos, sc = semantic_topk(H, None, C, cfg.k, None)
        assert kind == KIND_SEM
        # the noisy copy has cosine ~ 1/sqrt(1.01); unrelated N(0,1) rows ~ 0
        assert pos[0] in _copy_family(x["copy_logs"][i], src)
        assert sc[0] > 0.95


@pytest.mark.parametrize("seed", range(4))
def test_preceding_alignment_against_scipy(seed):
    """Eq. (6) as printed, from SciPy: candidate j >= 1 scored by
    1 - cosine distance(H[j-1], H[L-2]), ranked by repeated argmax."""
    rng = np.random.default_rng(100 + seed)
    L, d = 40, 12
    base = rng.integers(-2, 3, size=(5, d)).astype(np.float64)
    H = base[rng.integers(0, 5, size=L)]
    H[rng.integers(0, L, size=3)] = 0.0
    q = H[L - 2]

    def sc(j):
        return 0.0 if not H[j - 1].any() or not q.any() else 1.0 - scipy_cosine_distance(H[j - 1], q)

    for k in (1, 4, 39):
        rows = list(range(1, L - 1))
        kind, pos, got = semantic_topk(H, None, [], k, None, preceding=True)
        assert kind == KIND_SEM and pos == _argmax_select([sc(j) for j in rows], rows, k)
        np.testing.assert_allclose(got, [sc(j) for j in pos], rtol=0, atol=1e-12)
        cand = sorted(rng.choice(L - 1, size=8, replace=False).tolist())
        kind, pos, _ = semantic_topk(H, None, cand, k, None, preceding=True)
        kept = [c for c in cand if c >= 1]
        assert kind == KIND_LEX and pos == _argmax_select([sc(j) for j in kept], kept, k)


def test_preceding_is_the_row_alignment_one_step_back():
    """Scoring H[j-1] equals scoring the rows of a bank moved down one row
    (H'[j] = H[j-1]) with the default alignment, position 0 left out, and the
    query H[L-2] passed explicitly."""
    rng = np.random.default_rng(7)
    L, d = 60, 9
    H = rng.standard_normal((L, d))
    Hs = np.vstack([rng.standard_normal((1, d)), H[:-1]])
    # the fallback's candidates are every position 1..L-2 of the moved bank
    a = semantic_topk(H, None, [], 6, None, preceding=True)
    b = semantic_topk(Hs, H[L - 2], list(range(1, L - 1)), 6, None)
    assert a[0] == KIND_SEM and a[1] == b[1]
    np.testing.assert_allclose(a[2], b[2], rtol=0, atol=1e-15)
    a = semantic_topk(H, None, [0, 5, 9, 30, 58], 6, None, preceding=True)
    b = semantic_topk(Hs, H[L - 2], [5, 9, 30, 58], 6, None)
    assert a[0] == KIND_LEX and a[1] == b[1]
    assert semantic_topk(H, None, [0], 6, None, preceding=True) == (KIND_LEX, [], [])
