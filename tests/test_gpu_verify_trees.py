"""GPU parity of adapld_tree_verify_attn against the oracle's tree attention
(Sec. 3.6) on every node of every sequence, on random branching trees (each
node's parent any earlier node or the root), so that masks are arbitrary
ancestor-or-self relations rather than the builder's chains.  Node counts
and context lengths mix sequences whose stacked rows fill two row groups,
one row group or none, ragged last tiles, contexts shorter than one tile or
empty, and a batch with almost no work; the shape is the benchmark's
(16 sequences, 32 query heads over 8 kv heads, T_max = 52), and three more
shapes take the other decompositions: 40 query heads over 8 with T_max = 137
(every wave its own block, three row groups), 64 over 8 with T_max = 72 and
a split context (five row groups, two splits), and 32 heads without
grouping (one row group, four splits); two cases at 8192 keys take
whole-workgroup row blocks in one row group with four and eight splits,
and one whole-workgroup row blocks in five row groups with three splits;
the last case is the largest tree the
boundary takes (256 nodes)."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2606_05742_amd as adapld
from paper_2606_05742_amd.synth import f32_to_bf16_bits
from parity_helpers import check_verify, dev_bf16, dev_i32

pytestmark = pytest.mark.gpu

D = 128


def random_tree(rng, T):
    parent = np.full(T, -1, dtype=np.int64)
    for u in range(1, T):
        parent[u] = rng.integers(-1, u)
    mask = np.zeros((T, T), dtype=bool)
    for u in range(T):
        v = u
        while v >= 0:
            mask[u, v] = True
            v = parent[v]
    return mask


def run_case(L_stride, lens, counts, seed, B=16, HQ=32, HKV=8, T_MAX=52, plan_is=(2, 2, 1)):
    """plan_is: the decomposition the case must take (waves per row block,
    row groups, splits; None for splits: more than one)."""
    rng = np.random.default_rng(seed)
    plan = adapld.verify_plan(B, L_stride, T_MAX, HQ, HKV)
    kh, rgs, ns = plan_is
    assert (plan["kh"], plan["rowgroups"]) == (kh, rgs) and (plan["nsplit"] > 1 if ns is None else plan["nsplit"] == ns), plan
    bits = lambda shape: f32_to_bf16_bits(rng.standard_normal(shape).astype(np.float32))  # noqa: E731
    q = bits((B, T_MAX, HQ, D))
    kc = bits((B, HKV, L_stride, D))
    vc = bits((B, HKV, L_stride, D))
    kt = bits((B, T_MAX, HKV, D))
    vt = bits((B, T_MAX, HKV, D))
    nw = (T_MAX + 63) // 64
    masks = []
    words = np.zeros((B, T_MAX, nw), dtype=np.uint64)
    for b in range(B):
        m = random_tree(rng, counts[b])
        masks.append(m)
        for u in range(counts[b]):
            for v in range(counts[b]):
                if m[u, v]:
                    words[b, u, v // 64] |= np.uint64(1) << np.uint64(v % 64)
    out, lse = adapld.tree_verify_attn(dev_bf16(q), dev_bf16(kc), dev_bf16(vc), dev_bf16(kt), dev_bf16(vt),
                                       dev_i32(np.asarray(lens)), dev_i32(np.asarray(counts)),
                                       torch.from_numpy(words.view(np.int64)).cuda())
    torch.cuda.synchronize()
    out = out.float().cpu().numpy()
    lse = lse.cpu().numpy()
    scale = 1.0 / math.sqrt(D)
    for b in range(B):
        T, L = counts[b], lens[b]
        if T == 0:
            continue
        O, LSE = oracle.tree_verify_attn(
            oracle.bf16_bits_to_f64(q[b, :T]), oracle.bf16_bits_to_f64(kc[b, :, :L]),
            oracle.bf16_bits_to_f64(vc[b, :, :L]), oracle.bf16_bits_to_f64(kt[b, :T]),
            oracle.bf16_bits_to_f64(vt[b, :T]), masks[b], L, scale)
        check_verify(out[b, :T], lse[b, :, :T], O, LSE, f"seed={seed} b={b} T={T} L={L}")


def test_random_trees_mixed_sizes():
    # 208 and 140 stacked rows (two row groups), 128, 104 and 4 (one), none
    counts = [52, 52, 35, 32, 26, 1, 0, 52, 13, 52, 40, 26, 33, 0, 52, 7]
    lens = [700, 699, 640, 65, 64, 700, 700, 1, 0, 333, 700, 129, 700, 5, 700, 700]
    run_case(700, lens, counts, seed=1)


def test_random_trees_two_row_groups():
    counts = [52] * 16
    lens = [2048] * 16
    run_case(2048, lens, counts, seed=2)


def test_random_trees_almost_no_work():
    """Two live sequences, contexts of 130 and 64 keys."""
    counts = [33, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 20]
    lens = [130, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 64]
    run_case(200, lens, counts, seed=3)


def test_random_trees_every_wave_its_block():
    """40 query heads over 8: up to 685 stacked rows in row groups of 256."""
    counts = [137, 1, 0, 64, 100, 137, 52, 77]
    lens = [1500, 1500, 700, 1, 64, 1499, 900, 1500]
    run_case(1500, lens, counts, seed=4, B=8, HQ=40, HKV=8, T_MAX=137, plan_is=(1, 3, 1))


def test_random_trees_split_context():
    """64 query heads over 8, five row groups, the context split in two."""
    counts = [72, 9, 0]
    lens = [5000, 4999, 5000]
    run_case(5000, lens, counts, seed=5, B=3, HQ=64, HKV=8, T_MAX=72, plan_is=(2, 5, None))


def test_random_trees_one_row_group_streaming():
    """The benchmark's heads at 8192 keys and 8 sequences: whole-workgroup row
    blocks, one row group (its tiles loaded with the streaming hint), the
    context split in four, ragged last tiles, a context that ends inside the
    first split (three splits with no key)."""
    counts = [52, 52, 30, 1, 52, 17, 0, 52]
    lens = [8192, 8191, 4097, 100, 2048, 6000, 8192, 1]
    run_case(8192, lens, counts, seed=8, B=8, HQ=32, HKV=8, T_MAX=52, plan_is=(1, 1, 4))


def test_random_trees_eight_splits():
    """4 sequences of 8192 keys: eight splits."""
    counts = [52, 40, 1, 52]
    lens = [8192, 8000, 64, 1000]
    run_case(8192, lens, counts, seed=9, B=4, HQ=32, HKV=8, T_MAX=52, plan_is=(1, 1, 8))


def test_random_trees_row_groups_and_odd_splits():
    """64 query heads over 8 with T_max = 137: whole-workgroup row blocks in
    five row groups (L2-shared tiles) and the context in three splits, the
    second sequence's context ending inside the second split."""
    counts = [137, 90]
    lens = [1500, 700]
    run_case(1500, lens, counts, seed=10, B=2, HQ=64, HKV=8, T_MAX=137, plan_is=(1, 5, 3))


def test_random_trees_no_grouping():
    """32 heads, each its own kv head (G = 1), split context."""
    counts = [30, 17]
    lens = [900, 300]
    run_case(900, lens, counts, seed=6, B=2, HQ=32, HKV=32, T_MAX=30, plan_is=(2, 1, None))


def test_random_trees_largest():
    """T_max = 256, the largest tree the boundary takes: four tree tiles and
    four mask words per row, a 256-node tree beside smaller ones."""
    counts = [256, 200, 65]
    lens = [700, 0, 64]
    run_case(700, lens, counts, seed=7, B=3, HQ=16, HKV=16, T_MAX=256, plan_is=(2, 2, 1))
