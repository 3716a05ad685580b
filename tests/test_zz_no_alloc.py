"""adapld_step_noalloc (the step with the library's own device workspace,
for callers that cannot allocate) against adapld_step with a caller
workspace: every output bit for bit, on two calls in a row, the second with
a smaller input (the array keeps the first call's contents), then the
smaller input again with Eq. (6)'s alignment of the rerank."""
import numpy as np
import pytest
import torch

import paper_2606_05742_amd as adapld
from paper_2606_05742_amd.synth import make_inputs, small_config
from parity_helpers import dev_bf16, dev_i32

pytestmark = pytest.mark.gpu

FIELDS = ("cand_pos", "cand_count", "match_n", "topk_pos", "topk_score", "topk_count", "kind", "node_token",
          "node_parent", "node_depth", "node_src", "node_count", "tree_mask", "out", "lse")


def _step(x, cfg, noalloc, preceding=False):
    args = [dev_i32(x["tokens"]), dev_i32(x["lens"]), dev_bf16(x["bank"]), dev_bf16(x["q"]),
            dev_bf16(x["k_ctx"]), dev_bf16(x["v_ctx"]), dev_bf16(x["k_tree"]), dev_bf16(x["v_tree"])]
    bufs = adapld.StepBuffers.allocate(cfg.B, cfg.L, cfg.d, cfg.k, cfg.T_max, cfg.Hq, cfg.Hkv, cfg.D)
    for name in FIELDS:   # outputs start as garbage that differs between the two runs
        t = getattr(bufs, name)
        t.view(torch.uint8).fill_(0x5A if noalloc else 0xA5)
    adapld.step(*args, n_max=cfg.n_max, k=cfg.k, W=cfg.W, S=cfg.S, buffers=bufs, noalloc=noalloc,
                preceding=preceding)
    torch.cuda.synchronize()
    return bufs


def _compare(x, cfg, ctx, preceding=False):
    ref = _step(x, cfg, False, preceding)
    got = _step(x, cfg, True, preceding)
    B, L = cfg.B, cfg.L
    lens = np.clip(x["lens"], 0, L)
    cc = ref.cand_count.cpu().numpy()
    tc = ref.topk_count.cpu().numpy()
    nc = ref.node_count.cpu().numpy()
    for name in ("cand_count", "match_n", "topk_count", "kind", "node_count", "tree_mask"):
        assert torch.equal(getattr(got, name), getattr(ref, name)), (ctx, name)
    for name, per in (("cand_pos", cc), ("topk_pos", tc), ("topk_score", tc), ("node_token", nc),
                      ("node_parent", nc), ("node_depth", nc), ("node_src", nc)):
        g, r = getattr(got, name).cpu(), getattr(ref, name).cpu()
        for b in range(B):
            n = int(per[b])
            assert torch.equal(g[b, :n].view(torch.int32), r[b, :n].view(torch.int32)), (ctx, name, b)
    go, ro = got.out.cpu().view(torch.int16), ref.out.cpu().view(torch.int16)
    gl, rl = got.lse.cpu().view(torch.int32), ref.lse.cpu().view(torch.int32)
    for b in range(B):
        n = int(nc[b])
        assert torch.equal(go[b, :n], ro[b, :n]), (ctx, "out", b)
        assert torch.equal(gl[b, :, :n], rl[b, :, :n]), (ctx, "lse", b)
    assert int(nc.sum()) > 0 and int(lens.sum()) > 0


def test_noalloc_step_two_calls():
    # first call: a split verify (one long sequence, GQA), so the array holds
    # the rerank's lists and the verify's partials
    big = small_config(B=1, L=4096, d=512, k=8, n_max=4, seed=301, V=200, Hq=32, Hkv=8, W=4, S=10,
                       forced_every=1)
    info = adapld.verify_plan(big.B, big.L, big.T_max, big.Hq, big.Hkv)
    assert info["nsplit"] > 1, info
    _compare(make_inputs(big), big, "first (split verify)")
    # second call: smaller, ragged, lexical hits and misses
    small = small_config(B=3, L=700, d=256, k=4, n_max=3, seed=302, V=40, Hq=8, Hkv=2, W=3, S=4,
                         forced_every=2)
    xs = make_inputs(small, lens=np.array([700, 333, 2], np.int32))
    _compare(xs, small, "second (smaller)")
    _compare(xs, small, "third (smaller, rows j-1 against row L-2)", preceding=True)
