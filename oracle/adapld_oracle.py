"""CPU oracle for the AdaPLD draft-and-verify step (test infrastructure only).

This module is a plain, slow, float64 statement of what one decoding iteration
of AdaPLD computes between the target model's forward passes.  It exists to
check the HIP path: only the test suite, the package smoke check and the
benchmark's CPU-baseline leg may import it.  It shares no code with the HIP
path and imports nothing from it; its inputs are plain NumPy arrays (bf16
values arrive as their uint16 bit patterns and are decoded here, exactly, to
float64).

Four steps, per sequence, in the paper's order (Sec. 3.3 - 3.6, Algorithm 1):

``lexical_match``   -- lexical anchoring (Sec. 3.3, the exact-match set), read
                       as a longest-suffix n-gram match, n = n_max .. 1.
``semantic_topk``   -- the lexical/semantic backoff (Sec. 3.3) and the
                       hidden-state reranking (Sec. 3.4): cosine scores, ranked
                       by (score desc, position asc), top k kept.
``build_draft_tree``-- reuse construction (Sec. 3.5) organised as a draft tree
                       (Sec. 3.6): one branch per distinct successor token,
                       each a copied span; an ancestor-or-self mask.
``build_draft_tree_paper`` -- the paper's own construction (Sec. 3.5,
                       Algorithm 1): the main copy path of a lexical anchor,
                       branch tokens from the target's top tokens after the
                       anchor, and one successor token per branch retrieved
                       by a lexical match of the branch token (with the
                       token-embedding backoff when it never occurs) and a
                       hidden-state rerank against the anchor.
``tree_verify_attn``-- tree-masked attention over the KV cache (Sec. 3.6,
                       tree attention after Medusa), softmax in float64.
``embedding_fallback`` -- the lexical/semantic backoff with the paper's own
                       semantic signal (Sec. 3.3, Eqs. (4)-(5)): on a
                       lexical miss, every earlier position whose token
                       embedding has cosine >= tau with the last token's.
``accept_greedy``   -- greedy verification of the tree (Sec. 3.6 and the
                       speculative-decoding background of Appendix C: with
                       greedy decoding a draft token is kept when it equals
                       the target's own choice, up to the first mismatch),
                       and ``compact_kv`` -- the accepted nodes' K/V moved to
                       consecutive cache positions after the context.

Readings of the paper used here (where it is silent, ambiguous or where the
reproduced workload differs from its text):

* positions are 0-based; candidates j lie in [n-1, L-2], so every candidate
  has a following token (Sec. 3.3 uses 1 <= j < |M|);
* only the longest non-empty n-gram level is kept (n_max = 1 is exactly the
  paper's single-token match);
* the semantic score is the cosine between bank rows and an explicit query
  vector (by default the bank row of the last position), over candidate rows
  r (lexical hit) or all rows [0, L-2] (fallback); a zero norm gives cosine 0;
* tau, when given, filters fallback scores below it; it never filters a
  lexical hit;
* branch tokens are the first W distinct successor tokens M[r+1] along the
  ranked list; each branch is M[r+1 .. min(r+1+S, L-1)] (the branch token
  followed by up to S copied tokens).  With a lexical hit, branch 0 is the
  paper's main copy path with maximum copy length S+1;
* the tree is stored branch-major, depth-major within a branch; the parent of
  a depth-0 node is -1 (the root, the last context token, lives in the KV
  cache and is not a query row);
* verification keys for node u are all context keys 0..L-1 followed by the
  tree keys of u's ancestors-or-self in ascending node order;
* in the paper's construction the anchor j* is the top of the ranked list;
  the main path (lexical hit only) is M[j*+1 .. j*+l] with
  l = min(S+1, L-1-j*); the branch tokens are the given top tokens after the
  anchor in their order, without negatives, repeats and (lexical hit) the
  main path's first token, at most W of them; a branch token b gets the
  successor M[t*+1] where t* maximises cos(H[t-1], H[j*]) over its
  candidate positions t in [1, L-2] (lowest t among equal scores): those
  with M_t = b, or, when b never occurs there and an embedding table is
  given, those whose token embedding has cosine >= tau with b's (the
  lexical-first backoff of Sec. 3.3 with b as the query); a token with no
  candidate gets no successor; whether a lexical anchor's branches get
  successors is an argument, since the text of Sec. 3.5 drafts them for
  every branch and Algorithm 1 only after a semantic hit; nodes: the main
  path as a chain, then each branch token (depth 0) followed by its
  successor (depth 1);
* the token-embedding fallback scores positions j in [0, L-2] (the paper's
  1 <= j < |M|, 1-based) by cos(e[M_j], e[M_{L-1}]) (a zero norm gives 0),
  keeps those >= tau in ascending order, and is used only when the lexical
  set is empty (then kind SEM if anything is kept, else NONE); the selection
  among the kept positions is the hidden-state rerank of Sec. 3.4;
* greedy acceptance takes the target's greedy token after the context (the
  root) and after every node as given (no model here); node u is accepted
  when its token equals the target's token after its parent and every
  ancestor is accepted; the accepted path ends at the deepest accepted node
  (lowest index among equally deep ones, which only duplicate sibling tokens
  can produce); the emitted tokens are the path's tokens followed by the
  target's token after its last node (the bonus token; the target's token
  after the context when nothing is accepted);
* the accepted nodes' K/V go to cache positions L, L+1, ... in path order;
  positions at or beyond the cache capacity are not written.  The bonus
  token's K/V come from the next forward pass, outside this step.

Parity unpinned: none of the paper's printed numbers can pin these functions
(the paper prints no worked example); every function is pinned by brute force,
library routines, closed forms and invariants in the test suite instead.
"""
from __future__ import annotations

import numpy as np

KIND_NONE = 0
KIND_LEX = 1
KIND_SEM = 2


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact decode of bf16 bit patterns (uint16) to float64."""
    b = np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


# --------------------------------------------------------------------------
# Step 1: lexical anchoring (Sec. 3.3, exact-match candidate set; Alg. 1 ExactMatch)
# --------------------------------------------------------------------------

def lexical_match(tokens: np.ndarray, n_max: int):
    """Longest-suffix n-gram candidates of one context.

    For n = n_max down to 1, C_n holds every j in [n-1, L-2] whose n tokens
    ending at j equal the last n tokens of the context.  The first non-empty
    level wins.  Returns (n_star, C) with C ascending; (0, []) when no level
    has a candidate.
    """
    M = np.asarray(tokens)
    L = int(M.shape[0])
    assert n_max >= 1
    for n in range(n_max, 0, -1):
        if L < n + 1:
            continue
        js = np.arange(n - 1, L - 1)
        hit = np.ones(js.shape[0], dtype=bool)
        for i in range(n):
            hit &= M[js - i] == M[L - 1 - i]
        C = js[hit]
        if C.size > 0:
            return n, [int(j) for j in C]
    return 0, []


# --------------------------------------------------------------------------
# Step 2: backoff + hidden-state reranking (Sec. 3.3 backoff rule; Sec. 3.4 scores)
# --------------------------------------------------------------------------

def cosine_rows(H: np.ndarray, rows, q: np.ndarray) -> np.ndarray:
    """cos(H[r], q) for r in rows, float64; 0 where either norm is 0."""
    rows = np.asarray(rows, dtype=np.int64)
    X = H[rows]
    dots = X @ q
    nx = np.sqrt(np.einsum("ij,ij->i", X, X))
    nq = np.sqrt(q @ q)
    den = nx * nq
    out = np.zeros(rows.shape[0], dtype=np.float64)
    ok = den > 0
    out[ok] = dots[ok] / den[ok]
    return out


def semantic_topk(bank: np.ndarray, query, cand, k: int, tau=None, preceding=False):
    """Rank the retrieval candidates of one sequence.

    bank: (L, d) float64 hidden states; query: (d,) float64 or None.
    cand: the lexical candidate list (possibly empty).  With candidates (a
    lexical hit) the scored positions are the candidates and kind = LEX;
    otherwise every position in [0, L-2] is a candidate (semantic fallback),
    entries below tau are dropped when tau is given, and kind = SEM if any
    entry remains, else NONE.

    The score of position j (Sec. 3.4, Eq. (6)):
    - preceding=True, the equation as printed: the state before the candidate
      against the state before the anchor, cos(H[j-1], q) with q = H[L-2] by
      default; position 0 has no earlier state and is not scored (a lexical
      hit whose only candidate is 0 keeps kind LEX with nothing ranked);
    - preceding=False: cos(H[j], q) with q = H[L-1] by default (reading c.5).
    Ranking: score descending, then position ascending; the first
    min(k, #scored) are kept.  Returns (kind, positions, scores).
    """
    L = int(bank.shape[0])
    sh = 1 if preceding else 0
    if query is not None:
        q = np.asarray(query, dtype=np.float64)
    else:
        q = bank[L - 1 - sh] if L - 1 - sh >= 0 else np.zeros(bank.shape[1])
    if len(cand) > 0:
        rows = np.asarray(cand, dtype=np.int64)
        lexical = True
    else:
        rows = np.arange(0, max(L - 1, 0), dtype=np.int64)
        lexical = False
    rows = rows[rows >= sh]
    if rows.size == 0:
        return (KIND_LEX if lexical else KIND_NONE), [], []
    s = cosine_rows(bank, rows - sh, q)
    order = np.lexsort((rows, -s))
    top = order[: min(k, rows.size)]
    pos = [int(rows[i]) for i in top]
    sc = [float(s[i]) for i in top]
    if lexical:
        return KIND_LEX, pos, sc
    if tau is not None:
        keep = [i for i in range(len(sc)) if sc[i] >= tau]
        pos = [pos[i] for i in keep]
        sc = [sc[i] for i in keep]
    return (KIND_SEM if pos else KIND_NONE), pos, sc


def embedding_fallback(tokens: np.ndarray, emb: np.ndarray, cand, tau: float):
    """The lexical/semantic backoff rule with token-embedding similarity
    (Sec. 3.3, Eqs. (4)-(5)).

    tokens: (L,) ints; emb: (V, d) float64 token embeddings; cand: the lexical
    candidate list.  A non-empty lexical list is the result (kind LEX).
    Otherwise the result is every position j in [0, L-2] with
    cos(emb[M_j], emb[M_{L-1}]) >= tau, ascending: kind SEM if non-empty,
    else NONE.  Returns (kind, positions).
    """
    M = np.asarray(tokens)
    L = int(M.shape[0])
    if len(cand) > 0:
        return KIND_LEX, [int(j) for j in cand]
    if L < 2:
        return KIND_NONE, []
    s = cosine_rows(emb, M[:L - 1], emb[int(M[L - 1])])
    C = [j for j in range(L - 1) if s[j] >= tau]
    return (KIND_SEM if C else KIND_NONE), C


# --------------------------------------------------------------------------
# Step 3: reuse construction as a draft tree (Sec. 3.5, Sec. 3.6; Alg. 1 BuildDraftTree)
# --------------------------------------------------------------------------

def build_draft_tree(tokens: np.ndarray, kind: int, ranked, W: int, S: int):
    """Branches from the ranked retrieval list, as a tree.

    Walks the ranked positions r in order; the successor token M[r+1] opens a
    new branch unless an earlier branch already starts with it; at most W
    branches.  A branch copies M[r+1 .. min(r+1+S, L-1)].  Returns a dict with
    per-node lists token, parent, depth, src (the memory position the node
    copies), the node count T, the branch list, and the (T, T) boolean
    ancestor-or-self mask.
    """
    M = np.asarray(tokens)
    L = int(M.shape[0])
    branches = []
    if kind != KIND_NONE:
        used = set()
        for r in ranked:
            o = int(r) + 1
            b = int(M[o])
            if b in used:
                continue
            used.add(b)
            branches.append(list(range(o, min(o + S, L - 1) + 1)))
            if len(branches) == W:
                break
    token, parent, depth, src = [], [], [], []
    for br in branches:
        for dpt, p in enumerate(br):
            u = len(token)
            token.append(int(M[p]))
            parent.append(-1 if dpt == 0 else u - 1)
            depth.append(dpt)
            src.append(p)
    T = len(token)
    mask = np.zeros((T, T), dtype=bool)
    for u in range(T):
        v = u
        while v != -1:
            mask[u, v] = True
            v = parent[v]
    return dict(token=token, parent=parent, depth=depth, src=src, T=T,
                branches=branches, mask=mask)


SUCC_EVERY_BRANCH = 0    # Sec. 3.5 text: successor drafting for every branch token
SUCC_SEMANTIC_ONLY = 1   # Algorithm 1: no successors when the anchor is a lexical hit


def successor_candidates(tokens: np.ndarray, b: int, emb=None, tau=None):
    """The candidate set of a branch token used as a secondary query (Sec. 3.5,
    successor drafting, with the lexical-first backoff rule of Sec. 3.3).

    Positions t in [1, L-2] (a preceding hidden state and a following token).
    Lexical set: M_t == b.  When it is empty and an embedding table is given,
    the semantic set instead: cos(emb[M_t], emb[b]) >= tau (a token id outside
    the table has a zero embedding, cosine 0).  Returns the positions,
    ascending.
    """
    M = np.asarray(tokens)
    L = int(M.shape[0])
    ts = list(range(1, L - 1))
    C = [t for t in ts if int(M[t]) == b]
    if C or emb is None or not ts:
        return C
    V, d = emb.shape
    def row(tok):
        return emb[tok] if 0 <= tok < V else np.zeros(d)
    E = np.stack([row(int(M[t])) for t in ts])
    s = cosine_rows(E, np.arange(len(ts)), row(b))
    return [t for i, t in enumerate(ts) if s[i] >= tau]


def build_draft_tree_paper(tokens: np.ndarray, bank: np.ndarray, kind: int, ranked, top_tokens, W: int, S: int,
                           succ_mode: int = SUCC_EVERY_BRANCH, emb=None, tau=None):
    """The paper's draft construction (Sec. 3.5, Eqs. (8)-(15); Algorithm 1).

    tokens: (L,) ints; bank: (L, d) float64 hidden states; kind and ranked:
    the retrieval outcome (ranked positions, best first); top_tokens: the
    target's top tokens after the anchor j* = ranked[0], best first.
    succ_mode: SUCC_EVERY_BRANCH drafts a successor for every branch token
    (the text of Sec. 3.5); SUCC_SEMANTIC_ONLY only when the anchor came from
    the semantic fallback (Algorithm 1 leaves d_succ empty in its strict
    branch).  emb, tau: the token-embedding table (V, d) and threshold of the
    successor retrieval's semantic backoff; None keeps successor retrieval
    lexical only.
    Returns the same dict as build_draft_tree; src is the memory position a
    node copies, or -1 for a branch token (it comes from the model).
    """
    M = np.asarray(tokens)
    L = int(M.shape[0])
    token, parent, depth, src = [], [], [], []
    if kind != KIND_NONE and len(ranked) > 0:
        j = int(ranked[0])
        main = list(range(j + 1, j + 1 + min(S + 1, L - 1 - j))) if kind == KIND_LEX else []
        for dpt, p in enumerate(main):
            token.append(int(M[p]))
            parent.append(-1 if dpt == 0 else len(token) - 2)
            depth.append(dpt)
            src.append(p)
        first = int(M[j + 1]) if main else None
        branches = []
        for b in top_tokens:
            b = int(b)
            if b < 0 or b in branches or b == first:
                continue
            branches.append(b)
            if len(branches) == W:
                break
        drafts_successors = succ_mode == SUCC_EVERY_BRANCH or kind == KIND_SEM
        for b in branches:
            u = len(token)
            token.append(b)
            parent.append(-1)
            depth.append(0)
            src.append(-1)
            C = successor_candidates(M, b, emb, tau) if drafts_successors else []
            if C:
                s_b = cosine_rows(bank, [t - 1 for t in C], bank[j])
                best = C[int(np.argmax(s_b))]   # first maximum: the lowest t
                token.append(int(M[best + 1]))
                parent.append(u)
                depth.append(1)
                src.append(best + 1)
    T = len(token)
    mask = np.zeros((T, T), dtype=bool)
    for u in range(T):
        v = u
        while v != -1:
            mask[u, v] = True
            v = parent[v]
    return dict(token=token, parent=parent, depth=depth, src=src, T=T, mask=mask)


# --------------------------------------------------------------------------
# Step 4: tree-masked verify attention (Sec. 3.6)
# --------------------------------------------------------------------------

def tree_verify_attn(Q, Kc, Vc, Kt, Vt, mask, L: int, scale: float):
    """Attention of every tree node's query against context + ancestor keys.

    Q: (T, Hq, D); Kc, Vc: (Hkv, >=L, D); Kt, Vt: (T, Hkv, D); mask: (T, T)
    ancestor-or-self booleans; all float64.  Query head h reads kv head
    h // (Hq // Hkv).  For node u the keys are Kc[g, 0..L-1] followed by
    Kt[v, g] for every v with mask[u, v], v ascending; values likewise.
    Returns O (T, Hq, D) and LSE (Hq, T) (natural log of the softmax
    denominator of the scaled logits).
    """
    T, Hq, D = Q.shape
    Hkv = Kc.shape[0]
    G = Hq // Hkv
    O = np.zeros((T, Hq, D), dtype=np.float64)
    LSE = np.zeros((Hq, T), dtype=np.float64)
    for u in range(T):
        anc = [v for v in range(T) if mask[u, v]]
        for g in range(Hkv):
            keys = np.concatenate([Kc[g, :L], Kt[anc, g]], axis=0)
            vals = np.concatenate([Vc[g, :L], Vt[anc, g]], axis=0)
            heads = range(g * G, (g + 1) * G)
            for h in heads:
                z = scale * (keys @ Q[u, h])
                m = z.max()
                e = np.exp(z - m)
                l = e.sum()
                O[u, h] = (e @ vals) / l
                LSE[h, u] = m + np.log(l)
    return O, LSE


# --------------------------------------------------------------------------
# Step 5: greedy acceptance and KV compaction (Sec. 3.6; Appendix C)
# --------------------------------------------------------------------------

def accept_greedy(token, parent, root_next: int, node_next):
    """Greedy verification of a draft tree.

    token[u], parent[u]: the tree (parent -1 for depth-0 nodes).  root_next:
    the target's greedy token after the context; node_next[u]: its greedy
    token after node u's path.  Every root-to-node path is walked from the
    root: it survives while each node's token equals the target's token after
    the previous node.  Returns (path, emitted): the node list of the deepest
    surviving path (depth 0 first; lowest end index among equally deep ones)
    and the emitted tokens, the path's tokens followed by the bonus token.
    """
    T = len(token)
    best, best_len = None, 0
    for u in range(T):
        chain = []
        v = u
        while v != -1:
            chain.append(v)
            v = int(parent[v])
        chain.reverse()
        expected = int(root_next)
        ok = True
        for v in chain:
            if int(token[v]) != expected:
                ok = False
                break
            expected = int(node_next[v])
        if ok and len(chain) > best_len:
            best, best_len = u, len(chain)
    path = []
    v = best if best is not None else -1
    while v != -1:
        path.append(v)
        v = int(parent[v])
    path.reverse()
    bonus = int(node_next[best]) if best is not None else int(root_next)
    emitted = [int(token[v]) for v in path] + [bonus]
    return path, emitted


def compact_kv(kc_bits, vc_bits, kt_bits, vt_bits, L: int, path):
    """The cache after acceptance: copies of Kc, Vc ((Hkv, L_stride, D) bit
    patterns) with row L+i of every kv head replaced by Kt[path[i]], Vt[path[i]]
    ((T, Hkv, D)), for L+i < L_stride."""
    K = np.array(kc_bits, copy=True)
    V = np.array(vc_bits, copy=True)
    cap = K.shape[1]
    for i, u in enumerate(path):
        if L + i >= cap:
            break
        K[:, L + i] = kt_bits[u]
        V[:, L + i] = vt_bits[u]
    return K, V


# --------------------------------------------------------------------------
# One whole step over a batch (Alg. 1, one loop iteration up to verification)
# --------------------------------------------------------------------------

def step(tokens, lens, bank_bits, query_bits, n_max, k, W, S, tau=None,
         q_bits=None, kc_bits=None, vc_bits=None, kt_bits=None, vt_bits=None,
         scale=None, seqs=None, verify=True, preceding=False):
    """Run the four steps for the sequences in ``seqs`` (default: all).

    tokens: (B, L_stride) int; lens: (B,); bank_bits: (B, L_stride, d) uint16;
    query_bits: None (the default query of semantic_topk) or (B, d) uint16;
    preceding: the score alignment of semantic_topk.  Verify tensors are
    bf16 bit patterns in the layouts Q (B, T_max, Hq, D), Kc/Vc
    (B, Hkv, L_stride, D), Kt/Vt (B, T_max, Hkv, D).  Returns one dict per
    sequence with every intermediate and output.
    """
    B = tokens.shape[0]
    seqs = range(B) if seqs is None else seqs
    out = []
    for b in seqs:
        L = int(lens[b])
        M = np.asarray(tokens[b, :L])
        n_star, C = lexical_match(M, n_max)
        H = bf16_bits_to_f64(bank_bits[b, :L])
        qv = None if query_bits is None else bf16_bits_to_f64(query_bits[b])
        kind, pos, sc = semantic_topk(H, qv, C, k, tau, preceding=preceding)
        tree = build_draft_tree(M, kind, pos, W, S)
        rec = dict(b=b, n_star=n_star, cand=C, kind=kind, topk_pos=pos, topk_score=sc, tree=tree)
        if verify and tree["T"] > 0:
            T = tree["T"]
            Q = bf16_bits_to_f64(q_bits[b, :T])
            Kc = bf16_bits_to_f64(kc_bits[b, :, :L])
            Vc = bf16_bits_to_f64(vc_bits[b, :, :L])
            Kt = bf16_bits_to_f64(kt_bits[b, :T])
            Vt = bf16_bits_to_f64(vt_bits[b, :T])
            sc_ = (1.0 / np.sqrt(Q.shape[-1])) if scale is None else scale
            O, LSE = tree_verify_attn(Q, Kc, Vc, Kt, Vt, tree["mask"], L, sc_)
            rec.update(O=O, LSE=LSE)
        out.append(rec)
    return out
