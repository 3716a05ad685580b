"""The root (the last context token) verified with its tree in the same call,
as query row 0 (the verification of the bonus token, Sec. 3.6).

The verify takes any ancestor mask, so the root needs no layout of its own: row
0 holds the root's query with an empty mask row (its keys are the context
keys 0..L-1, its own key at L-1 included), and the tree's nodes follow in rows
1..T with their mask bits shifted by one (no node sees tree row 0, whose key
is the cache's row L-1).  The test builds that layout from the step's own
trees and compares every row, the root's included, with the oracle's
attention (also for sequences with an empty tree, where only the root row is
live)."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2606_05742_amd as adapld
from paper_2606_05742_amd.synth import f32_to_bf16_bits, make_inputs, small_config
from parity_helpers import check_verify, dev_bf16, dev_i32

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("kw", [
    dict(B=4, L=700, d=256, Hq=8, Hkv=2, k=8, W=3, S=4, n_max=3, seed=151, forced_every=2),
    dict(B=2, L=3000, d=128, Hq=8, Hkv=2, k=8, W=4, S=8, n_max=3, seed=152, forced_every=2),   # split context
])
def test_root_as_row_zero(kw):
    cfg = small_config(**kw)
    x = make_inputs(cfg)
    t = dict(tokens=dev_i32(x["tokens"]), lens=dev_i32(x["lens"]), bank=dev_bf16(x["bank"]), q=dev_bf16(x["q"]),
             k_ctx=dev_bf16(x["k_ctx"]), v_ctx=dev_bf16(x["v_ctx"]), k_tree=dev_bf16(x["k_tree"]),
             v_tree=dev_bf16(x["v_tree"]))
    bf = adapld.step(t["tokens"], t["lens"], t["bank"], t["q"], t["k_ctx"], t["v_ctx"], t["k_tree"], t["v_tree"],
                     n_max=cfg.n_max, k=cfg.k, W=cfg.W, S=cfg.S)
    torch.cuda.synchronize()
    T_of = bf.node_count.cpu().numpy()
    words = bf.tree_mask.cpu().numpy().view(np.uint64)

    # Layout with the root as row 0.
    B, Tm = cfg.B, cfg.T_max
    T1 = Tm + 1
    rng = np.random.default_rng(kw["seed"])
    root_q = f32_to_bf16_bits(rng.standard_normal((B, 1, cfg.Hq, cfg.D)).astype(np.float32))
    q1 = np.concatenate([root_q, x["q"]], axis=1)
    kt1 = np.concatenate([np.zeros_like(x["k_tree"][:, :1]), x["k_tree"]], axis=1)
    vt1 = np.concatenate([np.zeros_like(x["v_tree"][:, :1]), x["v_tree"]], axis=1)
    nw1 = (T1 + 63) // 64
    mask1 = np.zeros((B, T1, nw1), np.uint64)
    dense = np.zeros((B, T1, T1), bool)
    for b in range(B):
        for u in range(int(T_of[b])):
            for v in range(int(T_of[b])):
                if (int(words[b, u, v // 64]) >> (v % 64)) & 1:
                    mask1[b, u + 1, (v + 1) // 64] |= np.uint64(1) << np.uint64((v + 1) % 64)
                    dense[b, u + 1, v + 1] = True
    count1 = (T_of + 1).astype(np.int32)
    out, lse = adapld.tree_verify_attn(dev_bf16(q1), t["k_ctx"], t["v_ctx"], dev_bf16(kt1), dev_bf16(vt1), t["lens"],
                                       dev_i32(count1), torch.from_numpy(mask1.view(np.int64)).cuda())
    torch.cuda.synchronize()
    out, lse = out.float().cpu().numpy(), lse.cpu().numpy()
    scale = 1.0 / math.sqrt(cfg.D)
    for b in range(B):
        L = int(x["lens"][b])
        n = int(count1[b])
        O, LSE = oracle.tree_verify_attn(oracle.bf16_bits_to_f64(q1[b, :n]),
                                         oracle.bf16_bits_to_f64(x["k_ctx"][b, :, :L]),
                                         oracle.bf16_bits_to_f64(x["v_ctx"][b, :, :L]),
                                         oracle.bf16_bits_to_f64(kt1[b, :n]), oracle.bf16_bits_to_f64(vt1[b, :n]),
                                         dense[b, :n, :n], L, scale)
        check_verify(out[b, :n], lse[b, :, :n], O, LSE, f"b={b} T={n - 1}")
