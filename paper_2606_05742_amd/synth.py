"""Seeded synthetic inputs for the AdaPLD draft-and-verify step.

This module only draws random data; it holds none of the method's arithmetic.
It is the single source of inputs for both the HIP path and the CPU oracle.

The recipe stands in for the paper's workloads (Spec-Bench, CodeEditorBench and
the reasoning suites of Sec. 4.1), whose texts and model weights are not used
here.  Each sequence b draws from two streams, so that a draw of the tokens
alone gives the same tokens as a full draw:

``PCG64(SeedSequence([seed, b]))`` -- the tokens and the copy events:
1. tokens: L uniforms mapped through the CDF of a Zipf(a) law truncated to
   ranks 1..V; token id = 0-based rank;
2. span copies until at least ceil(p*L) positions are covered: span length
   l ~ U{lo..hi}, destination t ~ U{l..L-l}, source s ~ U{0..t-l};
3. optional forced lexical miss: the last token becomes the smallest id absent
   from the rest of the context; a source row src ~ U{0..L-2} is drawn.

``PCG64(SeedSequence([seed, b, 2]))`` -- the hidden bank:
4. standard normal ``(L, d)`` float32, then per copy event (in event order)
   the copied rows become source + 0.1*N(0,1); a forced sequence's last row
   becomes row src + 0.1*N(0,1) (a planted semantic neighbour);
5. the bank is rounded to bf16 (round-to-nearest-even) and stored as uint16.

The verify tensors (Q, K/V of the context, K/V of the tree nodes) come from
``PCG64(SeedSequence([seed, b, 1]))``, all bf16-rounded N(0,1).

The copy structure mimics the reuse statistics of the paper's appendix
(retrieval hit-rate and reuse-length tables): copied spans of a few to a few
hundred tokens make lexical hits common, and a fraction of sequences miss.
"""
from __future__ import annotations

import dataclasses
import math
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

__all__ = ["SeqConfig", "CONFIGS", "make_inputs", "f32_to_bf16_bits", "zipf_cdf"]


@dataclasses.dataclass(frozen=True)
class SeqConfig:
    """One workload: sizes of the context, the bank, the tree and attention."""

    name: str
    B: int
    L: int
    V: int
    zipf_a: float
    copy_frac: float
    span: tuple            # (lo, hi) copied-span length, inclusive
    d: int                 # hidden size of the bank
    Hq: int
    Hkv: int
    D: int
    n_max: int             # longest n-gram tried by the lexical match
    k: int                 # ranked candidates kept by the semantic/rerank step
    W: int                 # branch width
    S: int                 # tokens copied after each branch token
    seed: int
    forced_every: int = 0  # sequence b is forced to miss when b % forced_every == forced_every - 1
    prompt_len: int = 0    # >0: two-part context (prompt passages, then generated tail)
    prompt_span: tuple = (0, 0)
    prompt_copy_frac: float = 0.0

    @property
    def T_max(self) -> int:
        return self.W * (self.S + 1)

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv


# The five workloads.  Names state what they are; shapes follow the target
# models the paper evaluates (Vicuna-7B-like MHA, Llama-3-8B-like GQA, a 14B
# class and a 70B class model).
CONFIGS = {
    "b1_l512_mha32": SeqConfig(
        name="b1_l512_mha32", B=1, L=512, V=32000, zipf_a=1.1, copy_frac=0.30,
        span=(4, 32), d=4096, Hq=32, Hkv=32, D=128, n_max=3, k=4, W=4, S=8, seed=0),
    "b1_l4096_gqa32x8": SeqConfig(
        name="b1_l4096_gqa32x8", B=1, L=4096, V=128256, zipf_a=1.1, copy_frac=0.30,
        span=(4, 32), d=4096, Hq=32, Hkv=8, D=128, n_max=4, k=8, W=4, S=10, seed=2),
    "b16_l8192_gqa32x8": SeqConfig(
        name="b16_l8192_gqa32x8", B=16, L=8192, V=128256, zipf_a=1.1, copy_frac=0.40,
        span=(8, 64), d=4096, Hq=32, Hkv=8, D=128, n_max=4, k=8, W=4, S=12, seed=3,
        forced_every=4),
    "b64_l2048_gqa40x8": SeqConfig(
        name="b64_l2048_gqa40x8", B=64, L=2048, V=152064, zipf_a=1.05, copy_frac=0.50,
        span=(4, 48), d=5120, Hq=40, Hkv=8, D=128, n_max=5, k=8, W=8, S=16, seed=4),
    "b8_l32768_gqa64x8": SeqConfig(
        name="b8_l32768_gqa64x8", B=8, L=32768, V=128256, zipf_a=1.1, copy_frac=0.30,
        span=(4, 32), d=8192, Hq=64, Hkv=8, D=128, n_max=4, k=16, W=8, S=8, seed=5,
        prompt_len=28672, prompt_span=(64, 512), prompt_copy_frac=0.50),
}

# The workload the step is timed on: 16 sequences of 8192 tokens, 8B-class shapes.
BENCH_CONFIG = "b16_l8192_gqa32x8"


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (nearest, ties to even); return the uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return (rounded >> np.uint32(16)).astype(np.uint16)


def zipf_cdf(V: int, a: float) -> np.ndarray:
    ranks = np.arange(1, V + 1, dtype=np.float64)
    w = ranks ** (-a)
    c = np.cumsum(w)
    return c / c[-1]


def _span_events(rng, L, frac, lo, hi, t_lo, t_end, log):
    """Draw copy events for destinations in [t_lo, t_end) until frac of it is covered."""
    n = t_end - t_lo
    target = math.ceil(frac * n)
    covered = np.zeros(max(n, 0), dtype=bool)
    while int(covered.sum()) < target:
        ln = int(rng.integers(lo, hi + 1))
        t_min = max(t_lo, ln)
        t_max = t_end - ln
        if t_max < t_min:
            break
        t = int(rng.integers(t_min, t_max + 1))
        s = int(rng.integers(0, t - ln + 1))
        covered[t - t_lo:t - t_lo + ln] = True
        log.append((s, t, ln))


def _make_sequence(cfg: SeqConfig, b: int, L: int, d: int, cdf: np.ndarray, with_bank: bool):
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([cfg.seed, b])))
    u = rng.random(L)
    tokens = np.minimum(np.searchsorted(cdf, u, side="right"), cfg.V - 1).astype(np.int32)
    log = []
    if cfg.prompt_len > 0:
        P = min(cfg.prompt_len, L)
        _span_events(rng, L, cfg.prompt_copy_frac, *cfg.prompt_span, 0, P, log)
        if P < L:
            _span_events(rng, L, cfg.copy_frac, *cfg.span, P, L, log)
    else:
        _span_events(rng, L, cfg.copy_frac, *cfg.span, 0, L, log)
    for s, t, ln in log:
        tokens[t:t + ln] = tokens[s:s + ln]
    forced = None
    if cfg.forced_every and (b % cfg.forced_every == cfg.forced_every - 1) and L >= 2:
        present = np.zeros(cfg.V + 1, dtype=bool)
        present[tokens[:L - 1]] = True
        tok = int(np.flatnonzero(~present)[0])
        tokens[L - 1] = tok
        src = int(rng.integers(0, L - 1))
        forced = (tok, src)
    bank = None
    if with_bank:
        hrng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([cfg.seed, b, 2])))
        hidden = hrng.standard_normal((L, d), dtype=np.float32)
        for s, t, ln in log:
            noise = hrng.standard_normal((ln, d), dtype=np.float32)
            hidden[t:t + ln] = hidden[s:s + ln] + np.float32(0.1) * noise
        if forced is not None:
            noise = hrng.standard_normal(d, dtype=np.float32)
            hidden[L - 1] = hidden[forced[1]] + np.float32(0.1) * noise
        bank = f32_to_bf16_bits(hidden)
    return tokens, bank, log, forced


def _verify_tensors(cfg: SeqConfig, b: int, L: int):
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([cfg.seed, b, 1])))
    T = cfg.T_max
    q = f32_to_bf16_bits(rng.standard_normal((T, cfg.Hq, cfg.D), dtype=np.float32))
    kc = f32_to_bf16_bits(rng.standard_normal((cfg.Hkv, L, cfg.D), dtype=np.float32))
    vc = f32_to_bf16_bits(rng.standard_normal((cfg.Hkv, L, cfg.D), dtype=np.float32))
    kt = f32_to_bf16_bits(rng.standard_normal((T, cfg.Hkv, cfg.D), dtype=np.float32))
    vt = f32_to_bf16_bits(rng.standard_normal((T, cfg.Hkv, cfg.D), dtype=np.float32))
    return q, kc, vc, kt, vt


def make_inputs(cfg: SeqConfig, *, lens=None, with_bank=True, with_verify=True, seqs=None):
    """Draw the inputs of one step.

    ``lens`` optionally gives a per-sequence context length <= cfg.L (ragged
    batches); rows past a sequence's length are zero.  ``seqs`` restricts the
    draw to a subset of sequence indices (the arrays then hold only those, in
    the given order).  Returns a dict of numpy arrays plus the copy logs.
    """
    seqs = list(range(cfg.B)) if seqs is None else list(seqs)
    nb = len(seqs)
    L = cfg.L
    if lens is None:
        lens = [L] * nb
    lens = np.asarray(lens, dtype=np.int32)
    assert lens.shape == (nb,) and (lens >= 0).all() and (lens <= L).all()
    cdf = zipf_cdf(cfg.V, cfg.zipf_a)
    tokens = np.zeros((nb, L), np.int32)
    bank = np.zeros((nb, L, cfg.d), np.uint16) if with_bank else None
    logs, forced = [None] * nb, [None] * nb
    T = cfg.T_max
    if with_verify:
        q = np.zeros((nb, T, cfg.Hq, cfg.D), np.uint16)
        kc = np.zeros((nb, cfg.Hkv, L, cfg.D), np.uint16)
        vc = np.zeros_like(kc)
        kt = np.zeros((nb, T, cfg.Hkv, cfg.D), np.uint16)
        vt = np.zeros_like(kt)

    def one(i):
        b, Lb = seqs[i], int(lens[i])
        tok, bk, log, frc = _make_sequence(cfg, b, Lb, cfg.d, cdf, with_bank)
        tokens[i, :Lb] = tok
        if with_bank:
            bank[i, :Lb] = bk
        logs[i], forced[i] = log, frc
        if with_verify:
            q[i], kc[i, :, :Lb], vc[i, :, :Lb], kt[i], vt[i] = _verify_tensors(cfg, b, Lb)

    # Each sequence owns its streams, so the draw is the same for any thread count.
    workers = max(1, min(nb, _threads()))
    if workers == 1:
        for i in range(nb):
            one(i)
    else:
        with ThreadPoolExecutor(workers) as ex:
            list(ex.map(one, range(nb)))
    out = dict(cfg=cfg, tokens=tokens, lens=lens, bank=bank, copy_logs=logs, forced=forced)
    if with_verify:
        out.update(q=q, k_ctx=kc, v_ctx=vc, k_tree=kt, v_tree=vt)
    return out


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return min(n, 16)


def small_config(**kw) -> SeqConfig:
    """A small workload for tests: defaults suit an oracle run of a second or so."""
    base = dict(name="small", B=3, L=300, V=50, zipf_a=1.1, copy_frac=0.3, span=(4, 16),
                d=256, Hq=8, Hkv=2, D=128, n_max=3, k=6, W=3, S=5, seed=11)
    base.update(kw)
    return SeqConfig(**base)
