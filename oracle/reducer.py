"""Oracle of the Inherited HC-Gate Reducer.  Test infrastructure only.

Eq. (1) of Sec. 2.2 defines the target's hc_head collapse for one token t with
an m-path residual H_t (m rows of width d):

    x~_t   = RMSNorm(vec(H_t))
    alpha_t = sigmoid(W_f x~_t + b)          (m independent sigmoid gates)
    y_t    = sum_j alpha_{t,j} H_{t,j}

Sec. 2.2 adds that the real module uses inverse-RMS scaling, a scale factor and
a small offset, and that the drafter-side reducer keeps the same form with an
extra per-path RMSNorm of its input.  Readings taken here (listed in the design
notes): vec() is path-major (index j*d + c); the RMSNorm inside the gate carries
no weight of its own; the gate logit is gate_scale * r * (W_f x) + b with
r = 1/sqrt(mean(x^2) + eps), which equals W_f RMSNorm(x) + b for gate_scale = 1;
gate_offset is added to the sigmoid; the per-path norm, when enabled,
normalises each path over d before the weighted sum and leaves the gates as they
are.  The scale and offset defaults (1 and 0) are parity unpinned against the
real target, whose weights are not available.
"""
from __future__ import annotations

import numpy as np

from .numerics import as_f64, rmsnorm, sigmoid, store


def hc_reduce(H, W_g, b_g, *, eps: float = 1e-6, gate_scale: float = 1.0,
              gate_offset: float = 0.0, per_path_norm: bool = False,
              dtype: str = "bf16"):
    """Gated path collapse of Eq. (1), for every token independently.

    H:   [n_tok, m, d]  (uint16 bf16 bits, float32 or float64)
    W_g: [m, m*d]       the paper's W_f, one row per gate
    b_g: [m]
    Returns (Y [n_tok, d] float64 holding values representable in ``dtype``,
             alpha [n_tok, m] float64 unrounded gates).
    """
    H = as_f64(H)
    W = as_f64(W_g)
    b = np.asarray(b_g, dtype=np.float64)
    n, m, d = H.shape
    assert W.shape == (m, m * d) and b.shape == (m,)
    x = H.reshape(n, m * d)                       # vec(H_t), path-major
    ms = np.mean(x * x, axis=1, keepdims=True)    # mean square over all m*d entries
    r = 1.0 / np.sqrt(ms + eps)                   # inverse RMS
    z = gate_scale * r * (x @ W.T) + b            # W_f RMSNorm(vec H_t) + b
    alpha = sigmoid(z) + gate_offset              # independent per-path gates
    paths = H
    if per_path_norm:
        paths = rmsnorm(H, None, eps)             # each path over its own d entries
    y = np.zeros((n, d), dtype=np.float64)
    for j in range(m):                            # ascending path order
        y += alpha[:, j:j + 1] * paths[:, j, :]
    return store(y, dtype), alpha
