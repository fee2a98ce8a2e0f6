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


def lm_head_logits(hidden, w_lm) -> np.ndarray:
    """[M, d] x [V, d]^T -> float64 logits [M, V]."""
    return as_f64(hidden) @ as_f64(w_lm).T


def lm_head_argmax(hidden, w_lm):
    """Returns (argmax int32 [M], fp32 logits [M, V], top-2 margin float64 [M])."""
    z = lm_head_logits(hidden, w_lm)
    z32 = z.astype(np.float32)
    am = np.argmax(z32, axis=1).astype(np.int32)      # first index of the maximum
    top2 = np.partition(z, -2, axis=1)[:, -2:]
    margin = top2[:, 1] - top2[:, 0]
    return am, z32, margin
