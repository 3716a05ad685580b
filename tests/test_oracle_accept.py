"""Pins of the oracle's greedy acceptance and KV compaction (Sec. 3.6;
Appendix C: with greedy decoding a draft token is kept when it equals the
target's own choice, and the first mismatch ends verification).

The central pin is the property the paper relies on: the tokens a step emits
are exactly the target's own greedy continuation of the context, and the
number of draft tokens kept is the longest prefix of that continuation that
some tree path spells.  It is checked against a synthetic deterministic
"target" (a hash of the prefix), computed by decoding it token by token.
"""
import json
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "accept_cases.json")


def test_golden_cases():
    cases = json.load(open(GOLDEN))["cases"]
    assert len(cases) >= 6
    for c in cases:
        path, emitted = oracle.accept_greedy(c["token"], c["parent"], c["root_next"], c["node_next"])
        assert path == c["path"], c["why"]
        assert emitted == c["emitted"], c["why"]


def _target(prefix, V):
    """A deterministic stand-in for the target's greedy choice after a prefix."""
    h = 1469598103934665603
    for t in prefix:
        h = ((h ^ (int(t) + 1)) * 1099511628211) & ((1 << 64) - 1)
    return int((h >> 17) % V)


def _random_tree(rng, ctx, V, T, follow):
    """A random tree (parent index below the child's); with probability
    `follow` a node takes the target's own token after its parent's path."""
    token, parent, paths = [], [], []
    for u in range(T):
        p = -1 if u == 0 or rng.random() < 0.3 else int(rng.integers(0, u))
        prefix = list(ctx) + (paths[p] if p >= 0 else [])
        t = _target(prefix, V) if rng.random() < follow else int(rng.integers(0, V))
        token.append(t)
        parent.append(p)
        paths.append((paths[p] if p >= 0 else []) + [t])
    return token, parent, paths


@pytest.mark.parametrize("seed", range(40))
def test_emitted_tokens_are_the_targets_greedy_continuation(seed):
    rng = np.random.default_rng(seed)
    V = int(rng.integers(2, 6))
    ctx = list(rng.integers(0, V, size=int(rng.integers(1, 6))))
    T = int(rng.integers(0, 14))
    token, parent, paths = _random_tree(rng, ctx, V, T, follow=0.7)
    root_next = _target(ctx, V)
    node_next = [_target(ctx + paths[u], V) for u in range(T)]
    path, emitted = oracle.accept_greedy(token, parent, root_next, node_next)
    # decode the target greedily, one token at a time
    greedy = []
    for _ in range(T + 1):
        greedy.append(_target(ctx + greedy, V))
    longest = max([len(p) for p in paths if p == greedy[:len(p)]], default=0)
    assert len(path) == longest
    assert emitted == greedy[:longest + 1]
    # the path is a root path of the tree, listed from depth 0 down
    for i, u in enumerate(path):
        assert parent[u] == (path[i - 1] if i else -1)


def test_sequential_greedy_walk_on_trees_with_distinct_siblings():
    """On trees whose siblings carry distinct tokens (every tree the builder
    makes), walking down from the root and taking the child that carries the
    target's next token gives the same path."""
    rng = np.random.default_rng(5)
    for _ in range(300):
        V = int(rng.integers(2, 5))
        T = int(rng.integers(0, 12))
        token, parent = [], []
        for u in range(T):
            p = -1 if u == 0 or rng.random() < 0.3 else int(rng.integers(0, u))
            taken = {token[v] for v in range(u) if parent[v] == p}
            free = [t for t in range(V) if t not in taken]
            if not free:
                break
            token.append(int(rng.choice(free)))
            parent.append(p)
        T = len(token)
        root_next = int(rng.integers(0, V))
        node_next = [int(rng.integers(0, V)) for _ in range(T)]
        walk, cur, want = [], -1, root_next
        while True:
            kids = [v for v in range(T) if parent[v] == cur and token[v] == want]
            if not kids:
                break
            cur = kids[0]
            walk.append(cur)
            want = node_next[cur]
        path, emitted = oracle.accept_greedy(token, parent, root_next, node_next)
        assert path == walk
        assert emitted == [token[v] for v in walk] + [want]


def test_builder_trees_keep_at_most_one_branch():
    """Branch tokens are distinct, so at most one depth-0 node matches and the
    kept path lies on one branch."""
    rng = np.random.default_rng(11)
    for _ in range(200):
        M = rng.integers(0, 6, size=int(rng.integers(3, 40)))
        ranked = list(rng.permutation(len(M) - 1)[:8])
        tree = oracle.build_draft_tree(M, oracle.KIND_LEX, ranked, W=4, S=3)
        T = tree["T"]
        root_next = int(rng.integers(0, 6))
        node_next = [int(rng.integers(0, 6)) for _ in range(T)]
        path, emitted = oracle.accept_greedy(tree["token"], tree["parent"], root_next, node_next)
        assert len(emitted) == len(path) + 1
        if path:
            br = [i for i, b in enumerate(tree["branches"]) if b[0] == tree["src"][path[0]]]
            assert len(br) == 1
            assert [tree["src"][u] for u in path] == tree["branches"][br[0]][:len(path)]


def test_compact_kv():
    rng = np.random.default_rng(3)
    Hkv, cap, D, T = 3, 20, 8, 6
    kc = rng.integers(0, 1 << 16, size=(Hkv, cap, D), dtype=np.uint16)
    vc = rng.integers(0, 1 << 16, size=(Hkv, cap, D), dtype=np.uint16)
    kt = rng.integers(0, 1 << 16, size=(T, Hkv, D), dtype=np.uint16)
    vt = rng.integers(0, 1 << 16, size=(T, Hkv, D), dtype=np.uint16)
    path = [1, 3, 4]
    K, V = oracle.compact_kv(kc, vc, kt, vt, 15, path)
    for i, u in enumerate(path):
        np.testing.assert_array_equal(K[:, 15 + i], kt[u])
        np.testing.assert_array_equal(V[:, 15 + i], vt[u])
    untouched = [j for j in range(cap) if not 15 <= j < 18]
    np.testing.assert_array_equal(K[:, untouched], kc[:, untouched])
    np.testing.assert_array_equal(V[:, untouched], vc[:, untouched])
    # rows past the capacity are dropped
    K, V = oracle.compact_kv(kc, vc, kt, vt, 18, path)
    np.testing.assert_array_equal(K[:, 18], kt[1])
    np.testing.assert_array_equal(K[:, 19], kt[3])
    np.testing.assert_array_equal(K[:, :18], kc[:, :18])
