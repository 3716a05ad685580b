"""The C-ABI library loads, exports every declared symbol and validates
arguments on the host (no compute call is made: every call below carries an
invalid argument, which the library rejects before enqueueing anything)."""
import ctypes
import math
import os
import re

import pytest

from paper_2606_05742_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "adapld.h")
OK, NULL, INVALID, UNSUPPORTED, WS_SMALL = 0, -1, -2, -3, -4
P = ctypes.c_void_p(0x10000)  # never dereferenced: validation fails first
N = None


@pytest.fixture(scope="module")
def lib():
    return binding.load_library()


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(adapld_[a-z_]+)\s*\(", src)))


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert len(names) == 19
    for n in names:
        assert hasattr(lib, n), n
        assert n in binding.SIGNATURES, n


def test_status_strings(lib):
    for code in (OK, NULL, INVALID, UNSUPPORTED, WS_SMALL, -5, 123):
        assert lib.adapld_status_string(code)
    assert lib.adapld_version() == 20000
    assert lib.adapld_last_hip_error() == 0


def test_workspace_sizes(lib):
    ws = lib.adapld_workspace_bytes
    assert ws(1, 16, 8192, 4096, 8, 52, 32, 8, 128) == 0          # lexical needs none
    sem = ws(2, 16, 8192, 4096, 8, 0, 0, 0, 0)
    assert sem == 16 * 1024 * 8 * 8                                # one list per scan wave (1024) and sequence
    assert ws(2, 16, 300, 4096, 8, 0, 0, 0, 0) == 16 * 300 * 8 * 8  # at most one per row
    assert ws(2, 16, 8192, 4096, 65, 0, 0, 0, 0) == 0              # k beyond the limit
    assert ws(4, 1, 4096, 0, 0, 44, 32, 8, 128) > 0                # split context
    assert ws(4, 16, 2048, 0, 0, 52, 32, 8, 128) == 0              # one split: no partials
    assert ws(4, 16, 8192, 0, 0, 52, 32, 7, 128) == 0              # Hq % Hkv != 0
    assert ws(9, 16, 8192, 0, 0, 52, 32, 8, 128) == 0


def test_verify_plan(lib):
    info = (ctypes.c_int32 * 6)()
    f = lib.adapld_verify_plan
    assert f(16, 8192, 52, 32, 8, N) == NULL
    assert f(0, 8192, 52, 32, 8, info) == INVALID
    assert f(16, 8192, 52, 32, 7, info) == INVALID
    assert f(16, 8192, 257, 32, 8, info) == UNSUPPORTED
    assert f(16, 8192, 52, 32, 8, info) == OK
    waves, kh, rows_per_wg, rowgroups, nsplit, chunk = list(info)
    assert rows_per_wg == waves // kh * 32 and rowgroups * rows_per_wg >= 52 * 4
    assert nsplit * chunk >= 8192 and chunk % 64 == 0
    # the shapes of test_verify_variants (tests/test_gpu_parity.py) take all
    # four decompositions: (waves per row block, split context)
    seen = set()
    for B, L, T, Hq, Hkv in ((12, 300, 52, 40, 8), (6, 1200, 36, 32, 8), (1, 300, 20, 8, 2), (1, 1200, 20, 8, 2)):
        p = binding.verify_plan(B, L, T, Hq, Hkv)
        seen.add((p["kh"], p["nsplit"] > 1))
    assert seen == {(1, False), (1, True), (2, False), (2, True)}


def test_embed_validation(lib):
    f = lib.adapld_semantic_topk_embed
    nan = float("nan")
    args = lambda **kw: [kw.get(n, v) for n, v in (  # noqa: E731
        ("bank", P), ("query", N), ("tokens", P), ("lens", P), ("cand_pos", P), ("cand_count", P), ("emb", P),
        ("V", 100), ("B", 2), ("L_stride", 64), ("d", 128), ("k", 8), ("tau", 0.5), ("pre", 1),
        ("pos", P), ("score", P), ("count", P), ("kind", P), ("ws", P), ("ws_bytes", 1 << 30), ("stream", N))]
    assert f(*args(B=0)) == OK
    assert f(*args(B=-1)) == INVALID
    assert f(*args(emb=N)) == NULL
    assert f(*args(tokens=N)) == NULL
    assert f(*args(ws=N)) == NULL
    assert f(*args(tau=nan)) == INVALID                 # the threshold is required
    assert f(*args(pre=2)) == INVALID                   # the alignment is 0 or 1
    assert f(*args(V=0)) == INVALID
    assert f(*args(d=12)) == INVALID
    assert f(*args(k=65)) == UNSUPPORTED
    assert f(*args(emb=ctypes.c_void_p(0x10008))) == INVALID
    need = lib.adapld_workspace_bytes(5, 2, 64, 128, 8, 0, 0, 0, 0)
    assert need >= lib.adapld_workspace_bytes(2, 2, 64, 128, 8, 0, 0, 0, 0) + 2 * 64 * 5
    assert f(*args(ws_bytes=need - 1)) == WS_SMALL


def test_step_validation(lib):
    f = lib.adapld_step
    nan = float("nan")
    args = lambda **kw: [kw.get(n, v) for n, v in (  # noqa: E731
        ("tokens", P), ("lens", P), ("bank", P), ("query", N), ("q", P), ("k_ctx", P), ("v_ctx", P),
        ("k_tree", P), ("v_tree", P), ("B", 2), ("L_stride", 64), ("d", 128), ("n_max", 3), ("k", 8),
        ("W", 4), ("S", 4), ("T_max", 20), ("Hq", 8), ("Hkv", 2), ("D", 128), ("tau", nan), ("pre", 1),
        ("scale", 0.1), *[(f"o{i}", P) for i in range(15)], ("ws", P), ("ws_bytes", 1 << 30), ("stream", N))]
    assert f(*args(B=0)) == OK
    assert f(*args(B=-1)) == INVALID
    assert f(*args(ws=N)) == NULL
    assert f(*args(ws=ctypes.c_void_p(0x10008))) == INVALID
    assert f(*args(pre=-1)) == INVALID
    assert f(*args(tokens=N)) == NULL                 # the lexical call's check
    assert f(*args(n_max=65)) == UNSUPPORTED
    assert f(*args(d=12)) == INVALID                  # the rerank's
    assert f(*args(bank=ctypes.c_void_p(0x10008))) == INVALID
    assert f(*args(W=0)) == INVALID                   # the tree's
    assert f(*args(T_max=19)) == INVALID              # below W*(S+1)
    assert f(*args(D=64)) == UNSUPPORTED              # the verify's
    assert f(*args(scale=0.0)) == INVALID
    assert f(*args(Hq=6, Hkv=4)) == INVALID
    need = lib.adapld_workspace_bytes(7, 2, 64, 128, 8, 20, 8, 2, 128)
    sem = lib.adapld_workspace_bytes(2, 2, 64, 128, 8, 0, 0, 0, 0)
    ver = lib.adapld_workspace_bytes(4, 2, 64, 0, 0, 20, 8, 2, 128)
    assert need == (sem + 255) // 256 * 256 + ver
    assert f(*args(ws_bytes=(sem + 255) // 256 * 256 - 1)) == WS_SMALL
    split = lib.adapld_workspace_bytes(7, 1, 4096, 128, 8, 20, 8, 2, 128)   # a split verify: partials too
    assert split > lib.adapld_workspace_bytes(2, 1, 4096, 128, 8, 0, 0, 0, 0) + 255
    assert f(*args(B=1, L_stride=4096, T_max=20, ws_bytes=split - 1)) == WS_SMALL


def test_paper_tree_validation(lib):
    f = lib.adapld_build_draft_tree_paper
    args = lambda **kw: [kw.get(n, v) for n, v in (  # noqa: E731
        ("tokens", P), ("lens", P), ("bank", P), ("d", 128), ("pos", P), ("count", P), ("kind", P), ("k", 8),
        ("top", P), ("W", 4), ("S", 12), ("succ_mode", 0), ("emb", N), ("V", 0), ("tau", float("nan")),
        ("B", 2), ("L_stride", 64), ("T_max", 21),
        ("nt", P), ("np", P), ("nd", P), ("ns", P), ("nc", P), ("mask", P), ("ws", P), ("ws_bytes", 1 << 30),
        ("stream", N))]
    assert f(*args(B=0)) == OK
    assert f(*args(B=-1)) == INVALID
    assert f(*args(bank=N)) == NULL
    assert f(*args(top=N)) == NULL
    assert f(*args(ws=N)) == NULL
    assert f(*args(d=12)) == INVALID
    assert f(*args(W=0)) == INVALID
    assert f(*args(S=-1)) == INVALID
    assert f(*args(T_max=20)) == INVALID                  # below (S+1) + 2W
    assert f(*args(W=65, T_max=256)) == UNSUPPORTED
    assert f(*args(k=65)) == UNSUPPORTED
    assert f(*args(T_max=257)) == UNSUPPORTED
    assert f(*args(B=513)) == UNSUPPORTED                 # B*W lists > 2048
    assert f(*args(bank=ctypes.c_void_p(0x10008))) == INVALID
    assert f(*args(ws=ctypes.c_void_p(0x10008))) == INVALID
    assert f(*args(B=0, succ_mode=2)) == OK               # B = 0 returns before any check
    assert f(*args(succ_mode=2)) == INVALID               # neither reading
    assert f(*args(succ_mode=-1)) == INVALID
    assert f(*args(emb=P, V=0, tau=0.5)) == INVALID        # an embedding table needs rows
    assert f(*args(emb=P, V=10, tau=float("nan"))) == INVALID
    assert f(*args(emb=P, V=10, tau=float("inf"))) == INVALID
    assert f(*args(emb=ctypes.c_void_p(0x10008), V=10, tau=0.5)) == INVALID
    need = lib.adapld_workspace_bytes(6, 2, 64, 128, 4, 0, 0, 0, 0)
    assert need >= 2 * 4 * 64 * 4 + 2 * 4 * 128 * 2     # candidate lists + queries
    assert f(*args(ws_bytes=need - 1)) == WS_SMALL
    assert lib.adapld_workspace_bytes(6, 2, 64, 12, 4, 0, 0, 0, 0) == 0


def test_accept_validation(lib):
    f = lib.adapld_accept_greedy
    A = [P] * 7            # node_token, node_parent, node_depth, node_count, tree_mask, target_next, lens
    O = [P, P, P]          # accept_len, accept_nodes, out_tokens
    assert f(*A, N, N, 0, 0, 0, 0, 0, *O, N, N, N) == OK                 # B = 0: nothing to do
    assert f(*A, N, N, -1, 8, 8, 0, 0, *O, N, N, N) == INVALID
    assert f(N, *A[1:], N, N, 2, 8, 8, 0, 0, *O, N, N, N) == NULL
    assert f(*A, N, N, 2, 8, 8, 0, 0, P, P, N, N, N, N) == NULL          # out_tokens missing
    assert f(*A, P, N, 2, 8, 8, 2, 128, *O, P, P, N) == NULL             # some but not all K/V
    assert f(*A, N, N, 2, 0, 8, 0, 0, *O, N, N, N) == INVALID           # L_stride < 1
    assert f(*A, N, N, 2, 8, 0, 0, 0, *O, N, N, N) == INVALID           # T_max < 1
    assert f(*A, N, N, 2, 8, 257, 0, 0, *O, N, N, N) == UNSUPPORTED
    assert f(*A, P, P, 2, 8, 8, 0, 128, *O, P, P, N) == INVALID          # Hkv < 1 with K/V
    assert f(*A, P, P, 2, 8, 8, 2, 64, *O, P, P, N) == UNSUPPORTED       # D != 128
    Q = ctypes.c_void_p(0x10008)                                          # 8-byte aligned only
    assert f(*A, Q, P, 2, 8, 8, 2, 128, *O, P, P, N) == INVALID


def test_lexical_validation(lib):
    f = lib.adapld_lexical_match
    assert f(N, N, 0, 0, 0, N, N, N, N) == OK                      # B = 0: nothing to do
    assert f(N, P, 2, 16, 3, P, P, P, N) == NULL
    assert f(P, P, -1, 16, 3, P, P, P, N) == INVALID
    assert f(P, P, 2, 0, 3, P, P, P, N) == INVALID
    assert f(P, P, 2, 16, 0, P, P, P, N) == UNSUPPORTED
    assert f(P, P, 2, 16, 65, P, P, P, N) == UNSUPPORTED


def test_semantic_validation(lib):
    f = lib.adapld_semantic_topk
    nan = float("nan")
    args = lambda **kw: [kw.get(n, v) for n, v in [  # noqa: E731
        ("bank", P), ("query", N), ("lens", P), ("cand_pos", P), ("cand_count", P), ("B", 2), ("L", 64),
        ("d", 256), ("k", 8), ("tau", nan), ("pre", 0), ("tp", P), ("ts", P), ("tc", P), ("kind", P), ("ws", P),
        ("wsb", 1 << 20), ("st", N)]]
    assert f(*args(bank=N)) == NULL
    assert f(*args(ws=N)) == NULL
    assert f(*args(d=12)) == INVALID
    assert f(*args(d=0)) == INVALID
    assert f(*args(k=0)) == INVALID
    assert f(*args(k=65)) == UNSUPPORTED
    assert f(*args(d=8200)) == UNSUPPORTED
    assert f(*args(bank=ctypes.c_void_p(0x10008))) == INVALID      # misaligned bf16 rows
    assert f(*args(wsb=16)) == WS_SMALL
    assert f(*args(pre=2)) == INVALID                              # the alignment is 0 or 1
    assert f(*args(B=2049)) == UNSUPPORTED                         # sequence offsets live in LDS
    assert f(*args(B=2048, L=1 << 20)) == UNSUPPORTED              # B * L_stride beyond int32


def test_tree_validation(lib):
    f = lib.adapld_build_draft_tree
    args = lambda **kw: [kw.get(n, v) for n, v in [  # noqa: E731
        ("tok", P), ("lens", P), ("tp", P), ("tc", P), ("kind", P), ("B", 2), ("L", 64), ("k", 8),
        ("W", 4), ("S", 5), ("T", 24), ("nt", P), ("np", P), ("nd", P), ("ns", P), ("nc", P),
        ("mask", P), ("st", N)]]
    assert f(*args(mask=N)) == NULL
    assert f(*args(W=0)) == INVALID
    assert f(*args(S=-1)) == INVALID
    assert f(*args(T=23)) == INVALID                               # T_max < W(S+1)
    assert f(*args(k=65)) == UNSUPPORTED
    assert f(*args(T=257, W=1, S=0)) == UNSUPPORTED


def test_verify_validation(lib):
    f = lib.adapld_tree_verify_attn
    args = lambda **kw: [kw.get(n, v) for n, v in [  # noqa: E731
        ("q", P), ("kc", P), ("vc", P), ("kt", P), ("vt", P), ("lens", P), ("nc", P), ("mask", P),
        ("B", 2), ("L", 64), ("T", 24), ("Hq", 8), ("Hkv", 2), ("D", 128), ("scale", 0.1), ("out", P),
        ("lse", N), ("ws", P), ("wsb", 1 << 30), ("st", N)]]
    assert f(*args(out=N)) == NULL
    assert f(*args(Hkv=3)) == INVALID
    assert f(*args(D=64)) == UNSUPPORTED
    assert f(*args(T=300)) == UNSUPPORTED
    assert f(*args(scale=float("inf"))) == INVALID
    assert f(*args(scale=0.0)) == INVALID
    assert f(*args(scale=-0.1)) == INVALID
    assert f(*args(q=ctypes.c_void_p(0x10002))) == INVALID
    # L = 8192 splits the context, so a workspace is required
    assert lib.adapld_workspace_bytes(4, 2, 8192, 0, 0, 24, 8, 2, 128) > 0
    assert f(*args(L=8192, wsb=0)) == WS_SMALL


def test_binding_refuses_cpu_tensors():
    import torch
    t = torch.zeros((2, 8), dtype=torch.int32)
    with pytest.raises(binding.AdapldError):
        binding.lexical_match(t, torch.zeros(2, dtype=torch.int32), 2)


def test_step_noalloc_validation(lib):
    """The allocation-free step refuses, before any HIP call, sizes whose
    workspace exceeds its device array (host-only checks: no GPU needed)."""
    f = lib.adapld_step_noalloc
    cap = 64 << 20
    args = lambda **kw: [kw.get(n, v) for n, v in (  # noqa: E731
        *((f"p{i}", P) for i in range(9)), ("B", 2), ("L_stride", 64), ("d", 128), ("n_max", 3), ("k", 8),
        ("W", 4), ("S", 4), ("T_max", 20), ("Hq", 8), ("Hkv", 2), ("D", 128), ("tau", float("nan")), ("pre", 0),
        ("scale", 0.1), *((f"o{i}", P) for i in range(15)), ("stream", N))]
    assert f(*args(B=0)) == OK
    assert f(*args(B=-1)) == INVALID
    big = dict(B=2048, L_stride=4096, k=64)   # the rerank's lists alone: 2048 * 1024 * 64 * 8 bytes
    assert lib.adapld_workspace_bytes(7, 2048, 4096, 128, 64, 20, 8, 2, 128) > cap
    assert f(*args(**big)) == WS_SMALL


def test_ngram_index_validation(lib):
    """Host checks of the n-gram index calls (nothing is launched)."""
    need = lib.adapld_ngram_index_bytes(2, 64, 4)
    assert need > 0 and lib.adapld_ngram_index_bytes(2, 64, 65) == 0 and lib.adapld_ngram_index_bytes(0, 64, 4) == 0
    for f in (lib.adapld_ngram_index_build, lib.adapld_ngram_index_append):
        assert f(P, P, 0, 64, 4, P, need, N) == OK
        assert f(P, P, -1, 64, 4, P, need, N) == INVALID
        assert f(N, P, 2, 64, 4, P, need, N) == NULL
        assert f(P, P, 2, 64, 4, N, need, N) == NULL
        assert f(P, P, 2, 0, 4, P, need, N) == INVALID
        assert f(P, P, 2, 64, 0, P, need, N) == UNSUPPORTED
        assert f(P, P, 2, 64, 65, P, need, N) == UNSUPPORTED
        assert f(P, P, 2, 64, 4, ctypes.c_void_p(0x10008), need, N) == INVALID
        assert f(P, P, 2, 64, 4, P, need - 1, N) == WS_SMALL
    am = lib.adapld_ngram_index_append_match
    assert am(P, P, 0, 64, 4, P, need, P, P, P, N) == OK
    assert am(P, P, 2, 64, 4, P, need, P, N, P, N) == NULL
    assert am(P, P, 2, 1 << 25, 4, P, 1 << 60, P, P, P, N) == UNSUPPORTED
    m = lib.adapld_ngram_index_match
    assert m(P, P, P, need, 0, 64, 4, P, P, P, N) == OK
    assert m(P, P, P, need, 2, 64, 4, N, P, P, N) == NULL
    assert m(P, P, P, need - 1, 2, 64, 4, P, P, P, N) == WS_SMALL
