"""Oracle of the LM-head KL distillation forward (Sec. 2.4).  Test infrastructure
only.

Index convention (Sec. 2.3): with a the anchor's position, slot k of the block targets
token index a+k, and its teacher is LMHead applied to the target's state at index
a+k-1.  Only slots k = 1..P enter the loss:
    L_KL = T^2 / P * sum_{k=1..P} E_blocks[ KL(p_k^T || q_k^T) ]
    L    = L_CE + alpha * L_KL
with p^T, q^T the softmax of teacher and draft logits divided by T (Hinton's T^2
factor), and L_CE the usual cross entropy of the draft logits against the ground-
truth tokens.  The teacher state mean-pools the m residual paths (the paper's current
implementation, Sec. 2.4).
Readings taken here: LMHead(h) = RMSNorm(h) * gamma followed by the LM-head weights
(the head the drafter shares); the pooled, normed teacher state is stored in the
working dtype before the projection, as every GEMM input of the drafter; E_blocks is
the mean over blocks; L_CE is the mean over the B-1 draft positions of every block of
-log softmax(z)[label] at temperature 1.
"""
from __future__ import annotations

import numpy as np

from .lm_head import lm_head_logits
from .numerics import as_f64, rmsnorm, store


def teacher_hidden(H_pos, gamma, eps: float, dtype: str):
    """H_pos [R, m, d]: target residual paths at positions a+k-1 -> stored normed mean."""
    h = as_f64(H_pos).mean(axis=1)
    return store(rmsnorm(h, gamma, eps), dtype)


def _log_softmax(z):
    m = z.max(axis=-1, keepdims=True)
    return z - (m + np.log(np.exp(z - m).sum(axis=-1, keepdims=True)))


def kl_rows(teacher_logits, student_logits, T: float) -> np.ndarray:
    """KL(softmax(t / T) || softmax(z / T)) per row, float64."""
    lp = _log_softmax(as_f64(teacher_logits) / T)
    lq = _log_softmax(as_f64(student_logits) / T)
    return (np.exp(lp) * (lp - lq)).sum(axis=-1)


def ce_rows(student_logits, labels) -> np.ndarray:
    """-log softmax(z)[label] per row (temperature 1)."""
    lq = _log_softmax(as_f64(student_logits))
    return -np.take_along_axis(lq, np.asarray(labels, dtype=np.int64)[:, None], axis=1)[:, 0]


def kl_forward(H_pos, gamma, eps, w_lm, student_logits, labels, *, P: int, T: float,
               alpha: float, dtype: str = "bf16"):
    """H_pos [n, P, m, d] (positions a .. a+P-1 of every block); student_logits
    [n, B, V] (slot k of block s); labels [n, B-1] (ground truth of slots 1..B-1) or None.
    Returns (kl [n, P], ce [n, B-1] or None, (L_KL, L_CE, L))."""
    H_pos = np.asarray(H_pos)
    n = H_pos.shape[0]
    h = teacher_hidden(H_pos.reshape((n * P,) + H_pos.shape[2:]), gamma, eps, dtype)
    t = lm_head_logits(h, w_lm)                                  # teacher logits, [n*P, V]
    z = as_f64(student_logits)
    B = z.shape[1]
    kl = kl_rows(t, z[:, 1:P + 1].reshape(n * P, -1), T).reshape(n, P)
    L_kl = T * T / P * kl.sum(axis=1).mean()
    ce = None
    L_ce = 0.0
    if labels is not None:
        ce = ce_rows(z[:, 1:].reshape(n * (B - 1), -1), np.asarray(labels).reshape(-1)).reshape(n, B - 1)
        L_ce = ce.mean()
    return kl, ce, (L_kl, L_ce, L_ce + alpha * L_kl)
