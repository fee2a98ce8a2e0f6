"""Oracle of the LM head and greedy draft.  Test infrastructure only.

Draft logits z_k = LMHead(f_k) of the final-normed drafter state (Sec. 2.3, where
z_k are the draft logits of block position k); the greedy draft token is the
argmax over the vocabulary.  Readings: logits are reported in fp32 (the GPU's
output precision) and the argmax is taken on those fp32 logits, the lowest index
winning a tie; the top-2 margin is taken on the float64 logits.
"""
from __future__ import annotations

import numpy as np

from .numerics import as_f64


_CHUNK = 8192   # vocabulary rows decoded at a time


def lm_head_logits(hidden, w_lm) -> np.ndarray:
    """[M, d] x [V, d]^T -> float64 logits [M, V].  bf16 weights (uint16 bits) are
    decoded to float64 a block of vocabulary rows at a time into one reused buffer, so
    the full-vocabulary matrix never exists in float64 (4.2 GB at V = 129280, d = 4096);
    every logit is the same float64 dot product either way."""
    h = as_f64(hidden)
    w = np.asarray(w_lm)
    if w.dtype != np.uint16:
        return h @ as_f64(w).T
    V, d = w.shape
    z = np.empty((h.shape[0], V), dtype=np.float64)
    bits = np.empty((min(_CHUNK, V), d), dtype=np.uint32)
    wf = np.empty((min(_CHUNK, V), d), dtype=np.float64)
    for c0 in range(0, V, _CHUNK):
        n = min(_CHUNK, V - c0)
        np.left_shift(w[c0:c0 + n], 16, out=bits[:n], dtype=np.uint32)   # bf16 -> fp32 bits
        wf[:n] = bits[:n].view(np.float32)
        z[:, c0:c0 + n] = h @ wf[:n].T
    return z


def lm_head_argmax(hidden, w_lm):
    """Returns (argmax int32 [M], fp32 logits [M, V], top-2 margin float64 [M])."""
    z = lm_head_logits(hidden, w_lm)
    z32 = z.astype(np.float32)
    am = np.argmax(z32, axis=1).astype(np.int32)      # first index of the maximum
    top2 = np.partition(z, -2, axis=1)[:, -2:]
    margin = top2[:, 1] - top2[:, 0]
    return am, z32, margin
