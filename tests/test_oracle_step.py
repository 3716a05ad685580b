"""Pin of the oracle's whole-step composition (Algorithm 1, one iteration up
to verification): ``oracle.step`` must equal the four pinned oracle steps
applied by hand to each sequence's own slice of the batch.

The test slices every batched tensor itself (context length, tree size,
kv-head axis), decodes the bf16 patterns with its own decoder and passes the
verify scale explicitly, so a slip in step's slicing, default scale, query or
tau handling, or sequence selection shows up as a mismatch.
"""
import numpy as np
import pytest

import oracle


def _bf16_bits(x):
    return (np.asarray(x, dtype=np.float32).view(np.uint32) >> 16).astype(np.uint16)


def _decode(bits):
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _batch(seed, B=4, L_stride=48, d=16, Hq=4, Hkv=2, D=8, W=3, S=2):
    rng = np.random.default_rng(seed)
    T_max = W * (S + 1)
    tokens = rng.integers(0, 6, size=(B, L_stride)).astype(np.int32)
    lens = np.array([L_stride, 17, 5, 30][:B], dtype=np.int32)
    tokens[2, lens[2] - 1] = 99          # a lexical miss: the semantic fallback runs
    bank = _bf16_bits(rng.standard_normal((B, L_stride, d)))
    query = _bf16_bits(rng.standard_normal((B, d)))
    q = _bf16_bits(rng.standard_normal((B, T_max, Hq, D)))
    kc = _bf16_bits(rng.standard_normal((B, Hkv, L_stride, D)))
    vc = _bf16_bits(rng.standard_normal((B, Hkv, L_stride, D)))
    kt = _bf16_bits(rng.standard_normal((B, T_max, Hkv, D)))
    vt = _bf16_bits(rng.standard_normal((B, T_max, Hkv, D)))
    return dict(tokens=tokens, lens=lens, bank=bank, query=query, q=q, kc=kc, vc=vc, kt=kt, vt=vt,
                W=W, S=S, D=D)


def _by_hand(x, b, n_max, k, tau, explicit_query, scale, verify, preceding=False):
    L = int(x["lens"][b])
    M = x["tokens"][b, :L]
    n_star, C = oracle.lexical_match(M, n_max)
    H = _decode(x["bank"][b, :L])
    # the default query: the anchor's own state, or (Eq. (6)) the one before it
    qv = _decode(x["query"][b]) if explicit_query else H[L - 2 if preceding else L - 1]
    kind, pos, sc = oracle.semantic_topk(H, qv, C, k, tau, preceding=preceding)
    tree = oracle.build_draft_tree(M, kind, pos, x["W"], x["S"])
    rec = dict(n_star=n_star, cand=C, kind=kind, topk_pos=pos, topk_score=sc, tree=tree)
    T = tree["T"]
    if verify and T > 0:
        O, LSE = oracle.tree_verify_attn(
            _decode(x["q"][b, :T]), _decode(x["kc"][b, :, :L]), _decode(x["vc"][b, :, :L]),
            _decode(x["kt"][b, :T]), _decode(x["vt"][b, :T]), tree["mask"], L, scale)
        rec.update(O=O, LSE=LSE)
    return rec


@pytest.mark.parametrize("preceding", [False, True])
@pytest.mark.parametrize("explicit_query", [False, True])
@pytest.mark.parametrize("tau", [None, 0.05])
def test_step_equals_the_pinned_steps(explicit_query, tau, preceding):
    x = _batch(3)
    n_max, k = 3, 5
    seqs = [0, 2, 3]
    got = oracle.step(x["tokens"], x["lens"], x["bank"], x["query"] if explicit_query else None, n_max, k,
                      x["W"], x["S"], tau=tau, q_bits=x["q"], kc_bits=x["kc"], vc_bits=x["vc"],
                      kt_bits=x["kt"], vt_bits=x["vt"], seqs=seqs, preceding=preceding)
    assert [r["b"] for r in got] == seqs
    kinds = set()
    for r in got:
        want = _by_hand(x, r["b"], n_max, k, tau, explicit_query, 1.0 / np.sqrt(x["D"]), True, preceding)
        kinds.add(want["kind"])
        for key in ("n_star", "cand", "kind", "topk_pos"):
            assert r[key] == want[key], (r["b"], key)
        np.testing.assert_array_equal(r["topk_score"], want["topk_score"])
        for key in ("token", "parent", "depth", "src", "T"):
            assert r["tree"][key] == want["tree"][key]
        assert ("O" in r) == ("O" in want)
        if "O" in want:
            np.testing.assert_array_equal(r["O"], want["O"])
            np.testing.assert_array_equal(r["LSE"], want["LSE"])
    assert oracle.KIND_LEX in kinds and (oracle.KIND_SEM in kinds or oracle.KIND_NONE in kinds)


def test_step_explicit_scale_and_no_verify():
    x = _batch(5)
    got = oracle.step(x["tokens"], x["lens"], x["bank"], None, 2, 4, x["W"], x["S"], q_bits=x["q"],
                      kc_bits=x["kc"], vc_bits=x["vc"], kt_bits=x["kt"], vt_bits=x["vt"], scale=0.7)
    assert [r["b"] for r in got] == [0, 1, 2, 3]
    for r in got:
        want = _by_hand(x, r["b"], 2, 4, None, False, 0.7, True)
        assert r["tree"]["token"] == want["tree"]["token"]
        if "O" in want:
            np.testing.assert_array_equal(r["O"], want["O"])
            np.testing.assert_array_equal(r["LSE"], want["LSE"])
    bare = oracle.step(x["tokens"], x["lens"], x["bank"], None, 2, 4, x["W"], x["S"], verify=False)
    for r in bare:
        assert "O" not in r and "LSE" not in r
        want = _by_hand(x, r["b"], 2, 4, None, False, 0.7, False)
        assert r["topk_pos"] == want["topk_pos"] and r["tree"]["token"] == want["tree"]["token"]


def test_default_scale_is_inverse_sqrt_head_dim():
    """With scale omitted the verify logits use 1/sqrt(D) (the usual attention
    scale; D = 8 here), not 1/D or 1."""
    x = _batch(7)
    got = oracle.step(x["tokens"], x["lens"], x["bank"], None, 3, 4, x["W"], x["S"], q_bits=x["q"],
                      kc_bits=x["kc"], vc_bits=x["vc"], kt_bits=x["kt"], vt_bits=x["vt"], seqs=[0])
    r = got[0]
    assert "LSE" in r
    for scale, same in ((1.0 / np.sqrt(8.0), True), (1.0 / 8.0, False), (1.0, False)):
        want = _by_hand(x, 0, 3, 4, None, False, scale, True)
        assert np.array_equal(r["LSE"], want["LSE"]) == same, scale
