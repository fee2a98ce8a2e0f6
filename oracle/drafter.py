"""Oracle of the one-pass DFlash block drafter.  Test infrastructure only.

The paper fixes what the drafter consumes and predicts, not its layers:
  * it drafts a whole block in one pass from the accepted anchor token plus the
    target-side context, in the anchor-plus-mask block input format (Sec. 1,
    Sec. 2.1);
  * the context is the target's pre-collapse residual reduced by the gated
    reducer and injected into the drafter (Sec. 2.1, Sec. 2.2, Fig. 2 caption);
  * slot k of a block whose anchor sits at index a targets token index a+k
    (Sec. 2.3).

Readings taken for the layer itself (listed in the design notes): pre-norm
transformer layers with multi-head attention (n_heads * head_dim = d) and a
SiLU-gated MLP, no biases; the reduced context row c_i = RMSNorm(y_i) * g_ctx is
projected by each layer's own key/value weights and its keys/values precede the
block's own; the B block queries attend to every context key and to every block
key with no mask (bidirectional within the block); rotate-half RoPE over the
whole head with base theta, context row i at position i, block slot k at
position T + k where T is the context length (the anchor sits at a = T).

Precision (the storage points of the GPU path): u, c, Q, K, V (after RoPE), the
attention output, v, SiLU(g)*up and the final-normed state are rounded to the
working dtype; the residual stream h is rounded to fp32 after every update;
everything else is float64.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from .numerics import as_f64, rmsnorm, round_f32, silu, store


def rope(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotate-half rotary embedding of x [n, hd] at integer positions pos [n]:
    pairs (i, i + hd/2) turn by angle pos * theta^(-2i/hd).  theta = 0 means no
    rotary embedding."""
    if theta == 0:
        return x
    n, hd = x.shape
    half = hd // 2
    inv_freq = theta ** (-(2.0 * np.arange(half, dtype=np.float64)) / hd)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv_freq[None, :]
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[:, :half], x[:, half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=1)


def rope_heads(x: np.ndarray, pos: np.ndarray, n_heads: int, theta: float) -> np.ndarray:
    """RoPE applied to every head of x [n, n_heads*hd] independently."""
    n, dd = x.shape
    hd = dd // n_heads
    out = np.empty_like(x)
    for h in range(n_heads):
        out[:, h * hd:(h + 1) * hd] = rope(x[:, h * hd:(h + 1) * hd], pos, theta)
    return out


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray) -> np.ndarray:
    """Unmasked scaled dot-product attention of one head: q [nq, hd] over keys
    k [nk, hd] and values v [nk, hd]; softmax over all keys (max-subtracted)."""
    hd = q.shape[1]
    s = (q @ k.T) / np.sqrt(hd)
    s = s - s.max(axis=1, keepdims=True)
    p = np.exp(s)
    p = p / p.sum(axis=1, keepdims=True)
    return p @ v


class Weights:
    """Plain container of the drafter weights as float64 arrays."""

    def __init__(self, w: Dict[str, object], *, d: int, n_layers: int, n_heads: int,
                 head_dim: int, d_ff: int, vocab: int, eps: float = 1e-6,
                 rope_theta: float = 10000.0, dtype: str = "bf16"):
        self.d, self.L, self.nh, self.hd = d, n_layers, n_heads, head_dim
        self.F, self.V, self.eps, self.theta, self.dtype = d_ff, vocab, eps, rope_theta, dtype
        assert n_heads * head_dim == d
        self.tok_emb = w["tok_emb"]          # decoded row by row on use
        self.w_qkv = [as_f64(x) for x in w["w_qkv"]]
        self.w_o = [as_f64(x) for x in w["w_o"]]
        self.w_gate_up = [as_f64(x) for x in w["w_gate_up"]]
        self.w_down = [as_f64(x) for x in w["w_down"]]
        self.w_lm = w.get("w_lm")            # decoded by the LM head

        def g(x):
            return None if x is None else np.asarray(x, dtype=np.float64)
        self.ctx_norm = g(w.get("ctx_norm"))
        self.attn_norm = [g(x) for x in w.get("attn_norm", [None] * n_layers)]
        self.mlp_norm = [g(x) for x in w.get("mlp_norm", [None] * n_layers)]
        self.final_norm = g(w.get("final_norm"))


def context_kv(W: Weights, y_rows: np.ndarray, positions: np.ndarray
               ) -> List[Tuple[np.ndarray, np.ndarray]]:
    """Keys and values of reduced context rows for every layer.

    y_rows: [n, d] reduced states (already stored values); positions: [n].
    Returns per layer (K [n, d] after RoPE, V [n, d]), both stored values."""
    dt, d = W.dtype, W.d
    c = store(rmsnorm(as_f64(y_rows), W.ctx_norm, W.eps), dt)
    out = []
    for l in range(W.L):
        wk = W.w_qkv[l][d:2 * d]
        wv = W.w_qkv[l][2 * d:3 * d]
        k = store(rope_heads(c @ wk.T, positions, W.nh, W.theta), dt)
        v = store(c @ wv.T, dt)
        out.append((k, v))
    return out


def block_forward(W: Weights, ctx_kv: Sequence[Tuple[np.ndarray, np.ndarray]],
                  tokens: np.ndarray, trace: Optional[dict] = None,
                  pos_shift: int = 0) -> np.ndarray:
    """One pass of the drafter over one block of one sequence.

    ctx_kv: per layer (K_c [T, d], V_c [T, d]) of the T context rows.
    tokens: [B] block tokens (anchor, then mask ids).
    pos_shift: added to every block position (tests of relative-position
        invariance shift the context keys by the same amount).
    Returns the final-normed hidden states [B, d] (stored values)."""
    dt, d, nh, hd = W.dtype, W.d, W.nh, W.hd
    T = ctx_kv[0][0].shape[0]
    B = len(tokens)
    pos = pos_shift + T + np.arange(B)
    h = round_f32(as_f64(np.asarray(W.tok_emb)[np.asarray(tokens, dtype=np.int64)]))  # fp32 residual
    for l in range(W.L):
        u = store(rmsnorm(h, W.attn_norm[l], W.eps), dt)
        qkv = u @ W.w_qkv[l].T
        q = store(rope_heads(qkv[:, :d], pos, nh, W.theta), dt)
        kb = store(rope_heads(qkv[:, d:2 * d], pos, nh, W.theta), dt)
        vb = store(qkv[:, 2 * d:], dt)
        kc, vc = ctx_kv[l]
        o = np.empty((B, d), dtype=np.float64)
        for hh in range(nh):
            sl = slice(hh * hd, (hh + 1) * hd)
            keys = np.concatenate([kc[:, sl], kb[:, sl]], axis=0)
            vals = np.concatenate([vc[:, sl], vb[:, sl]], axis=0)
            o[:, sl] = attention(q[:, sl], keys, vals)
        o = store(o, dt)
        h = round_f32(h + o @ W.w_o[l].T)
        v = store(rmsnorm(h, W.mlp_norm[l], W.eps), dt)
        gu = v @ W.w_gate_up[l].T
        act = store(silu(gu[:, :W.F]) * gu[:, W.F:], dt)
        h = round_f32(h + act @ W.w_down[l].T)
        if trace is not None:
            trace.setdefault("layers", []).append(
                {"u": u, "q": q, "k": kb, "v": vb, "o": o, "act": act, "h": h})
    return store(rmsnorm(h, W.final_norm, W.eps), dt)


def draft_block(W: Weights, y_ctx: Sequence[np.ndarray], tokens: np.ndarray,
                kv_prefix: Optional[Sequence[Sequence[Tuple[np.ndarray, np.ndarray]]]] = None,
                seqs: Optional[Sequence[int]] = None) -> np.ndarray:
    """Block drafter over a batch of sequences, one sequence at a time.

    y_ctx[s]: reduced states of the context rows of sequence s that this step
        projects (the last rows of its context).
    kv_prefix[s]: optional per-layer (K, V) of the rows before those, already
        cached by earlier rounds (stored values).  Without it, y_ctx[s] is the
        whole context.
    tokens: [n_seq, B].
    seqs: optional subset of sequence indices to evaluate.
    Returns hidden [len(seqs) * B, d]."""
    tokens = np.asarray(tokens)
    if seqs is None:
        seqs = range(tokens.shape[0])
    outs = []
    for s in seqs:
        pre = kv_prefix[s] if kv_prefix is not None else None
        t0 = pre[0][0].shape[0] if pre is not None else 0
        y = as_f64(y_ctx[s])
        new = context_kv(W, y, t0 + np.arange(y.shape[0]))
        if pre is not None:
            kv = [(np.concatenate([as_f64(pre[l][0]), new[l][0]]),
                   np.concatenate([as_f64(pre[l][1]), new[l][1]])) for l in range(W.L)]
        else:
            kv = new
        outs.append(block_forward(W, kv, tokens[s]))
    return np.concatenate(outs, axis=0)
