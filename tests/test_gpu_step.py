"""adapld_step (the four calls from one native call) against the same step
as four separate entry-point calls: the outputs must be identical bit for
bit (the same kernels on the same inputs; every kernel is deterministic).
The step's results themselves are compared with the oracle in
test_gpu_parity.py, which runs the step through adapld_step."""
import numpy as np
import pytest
import torch

import paper_2606_05742_amd as adapld
from paper_2606_05742_amd.synth import make_inputs, small_config
from parity_helpers import dev_bf16, dev_i32

pytestmark = pytest.mark.gpu

FIELDS = ("cand_pos", "cand_count", "match_n", "topk_pos", "topk_score", "topk_count", "kind", "node_token",
          "node_parent", "node_depth", "node_src", "node_count", "tree_mask", "out", "lse")


def host(bf):
    return {f: getattr(bf, f).view(torch.int16).cpu().numpy() if f == "out" else getattr(bf, f).cpu().numpy()
            for f in FIELDS}


@pytest.mark.parametrize("kw,split,preceding", [
    (dict(B=3, L=300, d=256, k=6, W=3, S=5, seed=301, forced_every=2), False, False),
    (dict(B=2, L=3000, d=128, Hq=8, Hkv=2, k=8, W=4, S=8, seed=302, forced_every=2), True, False),
    (dict(B=3, L=300, d=256, k=6, W=3, S=5, seed=303, forced_every=2), False, True),
])
def test_native_step_matches_four_calls(kw, split, preceding):
    cfg = small_config(**kw)
    plan = adapld.verify_plan(cfg.B, cfg.L, cfg.T_max, cfg.Hq, cfg.Hkv)
    assert (plan["nsplit"] > 1) == split, plan
    x = make_inputs(cfg)
    t = dict(tokens=dev_i32(x["tokens"]), lens=dev_i32(x["lens"]), bank=dev_bf16(x["bank"]), q=dev_bf16(x["q"]),
             k_ctx=dev_bf16(x["k_ctx"]), v_ctx=dev_bf16(x["v_ctx"]), k_tree=dev_bf16(x["k_tree"]),
             v_tree=dev_bf16(x["v_tree"]))
    args = (t["tokens"], t["lens"], t["bank"], t["q"], t["k_ctx"], t["v_ctx"], t["k_tree"], t["v_tree"])
    kw2 = dict(n_max=cfg.n_max, k=cfg.k, W=cfg.W, S=cfg.S, preceding=preceding)
    ref = host(adapld.step_calls(*args, **kw2))
    call = adapld.StepCall(*args, **kw2)
    for rep in range(2):   # the marshalled call replayed
        got = host(call())
        torch.cuda.synchronize()
        for f in FIELDS:
            np.testing.assert_array_equal(got[f], ref[f], err_msg=f"{f} (call {rep})")
    assert int(ref["node_count"].sum()) > 0
