"""The oracle's pins catch plausible mistakes.

Each mutant changes one spot of the oracle (a dropped term, an off-by-one, a
wrong sign, a transposed operand, a wrong tie order) in a child process and
runs the pin suite against it; every mutant must make the suite fail.
"""
import json
import os
import subprocess
import sys

from concurrent.futures import ThreadPoolExecutor

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
# fastest first: with -x a caught mutant stops at its first failing pin
PINS = ["tests/test_oracle_accept.py", "tests/test_oracle_embedding.py", "tests/test_oracle_step.py",
        "tests/test_oracle_tree_paper.py", "tests/test_oracle_verify.py", "tests/test_oracle_tree.py",
        "tests/test_oracle_lexical.py", "tests/test_oracle_semantic.py"]

MUTANTS = [
    ("js = np.arange(n - 1, L - 1)", "js = np.arange(n - 1, L)"),              # anchor counts itself
    ("js = np.arange(n - 1, L - 1)", "js = np.arange(n, L - 1)"),              # drops the first window
    ("hit &= M[js - i] == M[L - 1 - i]", "hit &= M[js - i] == M[L - 2 - i]"),  # suffix off by one
    ("for n in range(n_max, 0, -1):", "for n in range(1, n_max + 1):"),        # shortest level first
    ("order = np.lexsort((rows, -s))", "order = np.lexsort((-rows, -s))"),    # ties to highest position
    ("order = np.lexsort((rows, -s))", "order = np.lexsort((rows, s))"),      # ascending scores
    ("nx = np.sqrt(np.einsum(\"ij,ij->i\", X, X))", "nx = np.einsum(\"ij,ij->i\", X, X)"),  # norm not rooted
    ("rows = np.arange(0, max(L - 1, 0), dtype=np.int64)", "rows = np.arange(0, L, dtype=np.int64)"),  # query row scored
    ("if sc[i] >= tau]", "if sc[i] > tau]"),                                   # tau boundary
    ("    if lexical:\n        return KIND_LEX, pos, sc\n", "    if lexical:\n        pass\n"),  # tau applied to lexical hits
    ("branches.append(list(range(o, min(o + S, L - 1) + 1)))", "branches.append(list(range(o, min(o + S, L - 1))))"),
    ("            if b in used:\n                continue\n", "            pass\n"),            # no dedup
    ("parent.append(-1 if dpt == 0 else u - 1)", "parent.append(-1)"),        # flat tree
    ("            o = int(r) + 1\n", "            o = int(r)\n"),                # copies the anchor, not its successor
    ("keys = np.concatenate([Kc[g, :L], Kt[anc, g]], axis=0)", "keys = np.concatenate([Kc[g, :L], Kt[:len(anc), g]], axis=0)"),
    ("z = scale * (keys @ Q[u, h])", "z = (keys @ Q[u, h])"),                   # scale dropped
    ("LSE[h, u] = m + np.log(l)", "LSE[h, u] = np.log(l)"),                   # max dropped
    ("heads = range(g * G, (g + 1) * G)", "heads = range(g, Hq, Hkv)"),       # wrong GQA grouping
    ("O[u, h] = (e @ vals) / l", "O[u, h] = (e @ vals)"),                       # no normalisation
    ("            expected = int(node_next[v])\n", "            expected = int(node_next[u])\n"),  # end node's choice
    ("        if ok and len(chain) > best_len:", "        if ok and len(chain) >= best_len:"),  # ties to the last end
    ("    bonus = int(node_next[best]) if best is not None else int(root_next)", "    bonus = int(root_next)"),
    ("        chain.reverse()\n", ""),                                         # walks the path bottom-up
    ("        K[:, L + i] = kt_bits[u]", "        K[:, L + i] = kt_bits[i]"),  # rows by rank, not node
    ("    C = [j for j in range(L - 1) if s[j] >= tau]", "    C = [j for j in range(L - 1) if s[j] > tau]"),
    ("    s = cosine_rows(emb, M[:L - 1], emb[int(M[L - 1])])", "    s = cosine_rows(emb, M[:L - 1], emb[int(M[L - 2])])"),
    ("        return KIND_LEX, [int(j) for j in cand]\n", "        pass\n"),   # semantic set despite a hit
    ("    C = [j for j in range(L - 1) if s[j] >= tau]", "    C = [j for j in range(L - 2) if s[j] >= tau]"),
    ("                token.append(int(M[best + 1]))", "                token.append(int(M[best]))"),   # the branch token again
    ("                s_b = cosine_rows(bank, [t - 1 for t in C], bank[j])", "                s_b = cosine_rows(bank, C, bank[j])"),
    ("            if b < 0 or b in branches or b == first:", "            if b < 0 or b in branches:"),  # main token kept as a branch
    ("    ts = list(range(1, L - 1))", "    ts = list(range(0, L - 1))"),          # an occurrence with no preceding state
    ("        drafts_successors = succ_mode == SUCC_EVERY_BRANCH or kind == KIND_SEM",
     "        drafts_successors = True"),                                          # Algorithm 1's strict branch ignored
    ("        drafts_successors = succ_mode == SUCC_EVERY_BRANCH or kind == KIND_SEM",
     "        drafts_successors = succ_mode == SUCC_EVERY_BRANCH or kind == KIND_LEX"),  # the two branches swapped
    ("    if C or emb is None or not ts:\n        return C\n", "    return C\n"),       # no successor backoff
    ("    if C or emb is None or not ts:\n", "    if emb is None or not ts:\n"),        # semantic set despite occurrences
    ("    return [t for i, t in enumerate(ts) if s[i] >= tau]", "    return [t for i, t in enumerate(ts) if s[i] > tau]"),
    ("    s = cosine_rows(E, np.arange(len(ts)), row(b))", "    s = cosine_rows(E, np.arange(len(ts)), row(int(M[L - 1])))"),
    ("            Vc = bf16_bits_to_f64(vc_bits[b, :, :L])", "            Vc = bf16_bits_to_f64(kc_bits[b, :, :L])"),   # values read from the keys
    ("            sc_ = (1.0 / np.sqrt(Q.shape[-1])) if scale is None else scale",
     "            sc_ = (1.0 / Q.shape[-1]) if scale is None else scale"),
    ("        qv = None if query_bits is None else bf16_bits_to_f64(query_bits[b])", "        qv = None"),
    ("        kind, pos, sc = semantic_topk(H, qv, C, k, tau, preceding=preceding)",
     "        kind, pos, sc = semantic_topk(H, qv, C, k, None, preceding=preceding)"),
    ("        kind, pos, sc = semantic_topk(H, qv, C, k, tau, preceding=preceding)",
     "        kind, pos, sc = semantic_topk(H, qv, C, k, tau)"),                   # step ignores the alignment
    ("    s = cosine_rows(bank, rows - sh, q)", "    s = cosine_rows(bank, rows, q)"),   # Eq. (6) rows not moved back
    ("        q = bank[L - 1 - sh] if L - 1 - sh >= 0 else np.zeros(bank.shape[1])",
     "        q = bank[L - 1] if L - 1 >= 0 else np.zeros(bank.shape[1])"),      # query not moved back
    ("    rows = rows[rows >= sh]\n", ""),                                       # position 0 scored
    ("    seqs = range(B) if seqs is None else seqs", "    seqs = range(B)"),
    ("        main = list(range(j + 1, j + 1 + min(S + 1, L - 1 - j))) if kind == KIND_LEX else []",
     "        main = list(range(j + 1, j + 1 + min(S, L - 1 - j))) if kind == KIND_LEX else []"),
]


def _run(mutant):
    env = dict(os.environ, ADAPLD_ORACLE_MUTANT=json.dumps(list(mutant)))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", *PINS],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    return r.returncode


def test_pins_catch_every_mutant():
    workers = max(1, min(8, len(os.sched_getaffinity(0))))
    with ThreadPoolExecutor(workers) as ex:
        codes = list(ex.map(_run, MUTANTS))
    survivors = [m for m, c in zip(MUTANTS, codes) if c != 1]
    assert not survivors, survivors


def test_unmutated_oracle_passes_pins():
    assert _run(("KIND_NONE = 0", "KIND_NONE = 0")) == 0
