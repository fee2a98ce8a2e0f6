"""Seeded synthetic workloads for the HyperDFlash drafter step.

This module only draws random inputs. It holds none of the method's
arithmetic: no reduction, no normalisation, no attention, no projection.
Both sides of every parity check (the CPU oracle and the HIP library) are fed
the very same bits that these functions return.

Shapes follow the paper's setting: a DeepSeek-V4-Flash-class target whose
Hyper-Connection residual has m = 4 paths of width d = 4096 (the two parameter
counts of Table 1, m*m*d = 65,536 and m*d*d = 67,108,864, force these values),
and a DFlash-style block drafter that drafts one block of B slots per step
(Sec. 1; Sec. 2.3 for the slot/position alignment).  The paper's own workloads
(public benchmark suites served through vLLM with the real target and trained
drafter weights, Sec. 3.2) are not available; these seeded tensors of the same
shapes stand in for them.

Random numbers come from torch generators seeded per (case seed, tensor id),
so drawing order never matters.  Floating-point draws are made in fp32 and,
for bf16 workloads, rounded once to bf16 (round-to-nearest-even, torch's own
conversion).  Generation may run on the CPU or on a GPU (a GPU generator is
much faster for the multi-GB tensors); whichever device drew a tensor, the
oracle receives a host copy of exactly those bits.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

# Fixed tensor ids: every tensor has its own stream, independent of call order.
_TID = {
    "H": 1, "W_g": 2, "b_g": 3, "path_scale": 4,
    "tok_emb": 10, "w_qkv": 11, "w_o": 12, "w_gate_up": 13, "w_down": 14, "w_lm": 15,
    "ctx_norm": 20, "attn_norm": 21, "mlp_norm": 22, "final_norm": 23,
    "H_ctx": 30, "kv_prefix": 31, "anchor": 40, "ctx_len": 41, "match_p": 42,
    "targets": 43,
}


def _gen(seed: int, tid: int, sub: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    # A fixed mixing of (seed, tensor id, sub-index) into one 63-bit seed.
    g.manual_seed((seed * 1_000_003 + tid * 10_007 + sub * 101 + 12345) & ((1 << 63) - 1))
    return g


def normal(shape, std: float, seed: int, tid: int, sub: int = 0, *, dtype: str = "bf16",
           device="cpu", mean: float = 0.0) -> torch.Tensor:
    """N(mean, std^2) draws in fp32, then (for bf16) one RNE rounding."""
    g = _gen(seed, tid, sub, device)
    x = torch.randn(*shape, generator=g, device=device, dtype=torch.float32)
    if std != 1.0:
        x.mul_(std)
    if mean != 0.0:
        x.add_(mean)
    return x.to(torch.bfloat16) if dtype == "bf16" else x


def uniform_int(shape, lo: int, hi: int, seed: int, tid: int, sub: int = 0,
                device="cpu") -> torch.Tensor:
    """Uniform integers in [lo, hi] (inclusive), int32."""
    g = _gen(seed, tid, sub, device)
    return torch.randint(lo, hi + 1, tuple(shape), generator=g, device=device,
                         dtype=torch.int64).to(torch.int32)


def uniform(shape, lo: float, hi: float, seed: int, tid: int, sub: int = 0,
            device="cpu") -> torch.Tensor:
    g = _gen(seed, tid, sub, device)
    return torch.rand(*shape, generator=g, device=device, dtype=torch.float32) * (hi - lo) + lo


# ---------------------------------------------------------------------------
# Workload descriptions
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class DrafterShape:
    d: int
    n_layers: int
    n_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    eps: float = 1e-6
    rope_theta: float = 10000.0


@dataclasses.dataclass
class Workload:
    name: str
    dtype: str                 # "f32" or "bf16"
    seed: int
    m: int
    d: int
    n_seq: int = 0
    ctx_lens: Optional[List[int]] = None
    block: int = 0
    drafter: Optional[DrafterShape] = None
    match_p: Optional[List[float]] = None   # per-sequence copy probability for targets
    n_tok: int = 0                           # reducer-only workloads
    path_scale: Optional[tuple] = None       # (lo, hi) per-path scale of H
    bias_std: float = 0.0                    # gate bias std (0 -> zero bias)
    w_std: float = 0.02
    new_rows: int = 0                        # context rows reduced/projected per step (warm)
    cold: bool = False                       # every context row reduced/projected per step


def tiny_fp32() -> Workload:
    """Tiny fp32 check: T=64, m=4, d=256, 1 layer of 4x64 heads, F=1024, V=4096, B=8."""
    return Workload("tiny_fp32", "f32", 0, m=4, d=256, n_seq=1, ctx_lens=[64], block=8,
                    drafter=DrafterShape(d=256, n_layers=1, n_heads=4, head_dim=64,
                                         d_ff=1024, vocab=4096),
                    match_p=None, new_rows=64)


def small_bf16() -> Workload:
    """Small bf16 step: 4 sequences x 512 context, d=1024, 2 layers of 16x64, F=4096,
    V=32000, B=16, targets copy the draft with p=0.7."""
    return Workload("small_bf16", "bf16", 1, m=4, d=1024, n_seq=4, ctx_lens=[512] * 4,
                    block=16,
                    drafter=DrafterShape(d=1024, n_layers=2, n_heads=16, head_dim=64,
                                         d_ff=4096, vocab=32000),
                    match_p=[0.7] * 4, new_rows=16)


def reducer_stress() -> Workload:
    """Reducer bandwidth stress: one reduce over 65536 tokens x 4 paths x 7168."""
    return Workload("reducer_stress", "bf16", 2, m=4, d=7168, n_tok=65536,
                    path_scale=(0.5, 2.0), bias_std=0.1)


def drafter_full() -> Workload:
    """Full-size drafter step: 8 sequences x 2048 context, d=4096, 1 layer of 32x128,
    F=12288, V=129280, B=16, targets copy the draft with p=0.8."""
    return Workload("drafter_full", "bf16", 3, m=4, d=4096, n_seq=8, ctx_lens=[2048] * 8,
                    block=16,
                    drafter=DrafterShape(d=4096, n_layers=1, n_heads=32, head_dim=128,
                                         d_ff=12288, vocab=129280),
                    match_p=[0.8] * 8, new_rows=16)


def drafter_full_cold() -> Workload:
    """Cold step of the full-size drafter: the cache starts empty and every one of the
    2048 context rows of each of the 8 sequences is reduced and projected in the step."""
    wl = drafter_full()
    wl.name = "drafter_full_cold"
    wl.new_rows = 2048
    wl.cold = True
    return wl


def ragged_decode(n_seq: int = 64) -> Workload:
    """Batched ragged decode: 64 sequences, context lengths U[1024, 16384], same drafter
    as the full-size step, per-sequence copy probability U[0.3, 0.95]."""
    seed = 4
    lens = uniform_int([n_seq], 1024, 16384, seed, _TID["ctx_len"]).tolist()
    ps = uniform([n_seq], 0.3, 0.95, seed, _TID["match_p"]).tolist()
    return Workload("ragged_decode", "bf16", seed, m=4, d=4096, n_seq=n_seq, ctx_lens=lens,
                    block=16,
                    drafter=DrafterShape(d=4096, n_layers=1, n_heads=32, head_dim=128,
                                         d_ff=12288, vocab=129280),
                    match_p=ps, new_rows=16)


def ragged_decode_cold(n_seq: int = 64) -> Workload:
    """Cold step of the batched ragged workload: the cache starts empty and every context
    row of the 64 sequences (lengths U[1024, 16384]) is reduced and projected."""
    wl = ragged_decode(n_seq)
    wl.name = "ragged_decode_cold"
    wl.new_rows = 0
    wl.cold = True
    return wl


WORKLOADS = {
    "tiny_fp32": tiny_fp32,
    "small_bf16": small_bf16,
    "reducer_stress": reducer_stress,
    "drafter_full": drafter_full,
    "drafter_full_cold": drafter_full_cold,
    "ragged_decode": ragged_decode,
    "ragged_decode_cold": ragged_decode_cold,
}


# ---------------------------------------------------------------------------
# Tensor draws
# ---------------------------------------------------------------------------

def reducer_inputs(wl: Workload, n_tok: int, *, device="cpu", sub: int = 0,
                   zero_bias: Optional[bool] = None) -> Dict[str, torch.Tensor]:
    """H [n_tok, m, d], W_g [m, m*d], b_g [m] (fp32).

    H ~ N(0,1) (times a per-path scale s_j ~ U[lo,hi] where the workload asks for
    one, applied before the single rounding), W_g ~ N(0, w_std), b_g ~ N(0, bias_std)
    or zero."""
    m, d = wl.m, wl.d
    H = normal([n_tok, m, d], 1.0, wl.seed, _TID["H"], sub, dtype="f32", device=device)
    if wl.path_scale is not None:
        s = uniform([m], wl.path_scale[0], wl.path_scale[1], wl.seed, _TID["path_scale"],
                    device=device)
        H.mul_(s.view(1, m, 1))
    if wl.dtype == "bf16":
        H = H.to(torch.bfloat16)
    W_g = normal([m, m * d], wl.w_std, wl.seed, _TID["W_g"], dtype=wl.dtype, device=device)
    if wl.bias_std > 0 and not zero_bias:
        b_g = normal([m], wl.bias_std, wl.seed, _TID["b_g"], dtype="f32", device=device)
    else:
        b_g = torch.zeros(m, dtype=torch.float32, device=device)
    return {"H": H, "W_g": W_g, "b_g": b_g}


def drafter_weights(wl: Workload, *, device="cpu", random_norms: bool = False
                    ) -> Dict[str, object]:
    """Drafter weights: embeddings, per-layer projections, LM head (all N(0, w_std)),
    and fp32 RMSNorm weights (ones, or N(1, 0.1) when random_norms is set so that
    tests see every norm weight actually applied)."""
    dr = wl.drafter
    d, F, V, L = dr.d, dr.d_ff, dr.vocab, dr.n_layers
    s, dt, sd = wl.seed, wl.dtype, wl.w_std

    def nrm(name, sub=0):
        if random_norms:
            return normal([d], 0.1, s, _TID[name], sub, dtype="f32", device=device, mean=1.0)
        return torch.ones(d, dtype=torch.float32, device=device)

    return {
        "tok_emb": normal([V, d], sd, s, _TID["tok_emb"], dtype=dt, device=device),
        "w_qkv": [normal([3 * d, d], sd, s, _TID["w_qkv"], l, dtype=dt, device=device)
                  for l in range(L)],
        "w_o": [normal([d, d], sd, s, _TID["w_o"], l, dtype=dt, device=device)
                for l in range(L)],
        "w_gate_up": [normal([2 * F, d], sd, s, _TID["w_gate_up"], l, dtype=dt, device=device)
                      for l in range(L)],
        "w_down": [normal([d, F], sd, s, _TID["w_down"], l, dtype=dt, device=device)
                   for l in range(L)],
        "w_lm": normal([V, d], sd, s, _TID["w_lm"], dtype=dt, device=device),
        "ctx_norm": nrm("ctx_norm"),
        "attn_norm": [nrm("attn_norm", l) for l in range(L)],
        "mlp_norm": [nrm("mlp_norm", l) for l in range(L)],
        "final_norm": nrm("final_norm"),
    }


def block_tokens(wl: Workload, *, device="cpu", sub: int = 0) -> torch.Tensor:
    """[n_seq, B] int32: slot 0 is the accepted anchor (uniform over the vocabulary),
    slots 1..B-1 hold the mask token id, taken as V-1."""
    V = wl.drafter.vocab
    anchors = uniform_int([wl.n_seq], 0, V - 1, wl.seed, _TID["anchor"], sub, device=device)
    toks = torch.full((wl.n_seq, wl.block), V - 1, dtype=torch.int32, device=device)
    toks[:, 0] = anchors
    return toks


def kv_prefix(wl: Workload, n_rows: int, layer: int, *, device="cpu", sub: int = 0):
    """Synthetic already-cached context keys/values (rows of earlier rounds), [n_rows, d]
    each, at the scale a projection of a unit-RMS state by N(0, w_std) weights has:
    std = w_std * sqrt(d)."""
    d = wl.d
    std = wl.w_std * math.sqrt(d)
    k = normal([n_rows, d], std, wl.seed, _TID["kv_prefix"], 2 * (layer * 64 + sub),
               dtype=wl.dtype, device=device)
    v = normal([n_rows, d], std, wl.seed, _TID["kv_prefix"], 2 * (layer * 64 + sub) + 1,
               dtype=wl.dtype, device=device)
    return k, v


def reduced_states(wl: Workload, n_rows: int, *, device="cpu", sub: int = 0) -> torch.Tensor:
    """Stand-in reduced context states [n_rows, d] for drafter-only tests: N(0, 1), the
    scale of a gated sum of unit-variance paths with gates near 1/2."""
    return normal([n_rows, wl.d], 1.0, wl.seed, _TID["H_ctx"], sub, dtype=wl.dtype, device=device)


def make_targets(drafts: np.ndarray, match_p: Sequence[float], vocab: int, seed: int,
                 sub: int = 0) -> np.ndarray:
    """Synthetic target-model tokens for greedy verification.

    drafts: [n_seq, K] draft tokens.  Returns [n_seq, K+1] int32: position i copies
    the draft with probability p_s, otherwise it is a token guaranteed to differ,
    (draft + 1 + U{0..V-2}) mod V; the last position (the bonus token) is uniform."""
    drafts = np.asarray(drafts, dtype=np.int64)
    n, K = drafts.shape
    rng = np.random.default_rng([seed, _TID["targets"], sub])
    u = rng.random((n, K))
    off = rng.integers(0, vocab - 1, size=(n, K))
    other = (drafts + 1 + off) % vocab
    p = np.asarray(match_p, dtype=np.float64).reshape(n, 1)
    tgt = np.where(u < p, drafts, other)
    bonus = rng.integers(0, vocab, size=(n, 1))
    return np.concatenate([tgt, bonus], axis=1).astype(np.int32)


def offsets(lens: Sequence[int]) -> np.ndarray:
    o = np.zeros(len(lens) + 1, dtype=np.int32)
    o[1:] = np.cumsum(np.asarray(lens, dtype=np.int64))
    return o


def to_numpy_bits(t: torch.Tensor) -> np.ndarray:
    """Host copy of a tensor's exact bits: bf16 -> uint16 array, others -> numpy."""
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()
