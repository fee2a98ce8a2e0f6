"""Oracle of the generic fc reducer (the fallback path collapse).  Test
infrastructure only.

Sec. 2.2 (and Table 1) describe the generic DFlash reducer as a static dense
projection fc: R^{m d} -> R^d of the flattened multi-path residual, learned from
scratch (about 67M parameters at m = 4, d = 4096), and name it the fallback when
the gated reducer's assumptions fail.  Readings taken here: vec() is path-major
(index j*d + c, as for the gated reducer); no normalisation precedes the
projection; an optional bias b [d] is added (None = no bias).  The result is
stored in the working dtype.
"""
from __future__ import annotations

import numpy as np

from .numerics import as_f64, store


def fc_reduce(H, W_fc, b_fc=None, *, dtype: str = "bf16"):
    """y_t = W_fc vec(H_t) (+ b) for every token.

    H:    [n_tok, m, d]  (uint16 bf16 bits, float32 or float64)
    W_fc: [d, m*d]       one row per output feature
    b_fc: [d] or None
    Returns Y [n_tok, d] float64 holding values representable in ``dtype``."""
    H = as_f64(H)
    W = as_f64(W_fc)
    n, m, d = H.shape
    assert W.shape == (d, m * d)
    y = H.reshape(n, m * d) @ W.T
    if b_fc is not None:
        y = y + np.asarray(b_fc, dtype=np.float64).reshape(1, d)
    return store(y, dtype)


def fc_parameter_count(m: int, d: int, bias: bool = False) -> int:
    """Trainable parameters of the fc projection: m*d*d (+ d with a bias)."""
    return m * d * d + (d if bias else 0)
