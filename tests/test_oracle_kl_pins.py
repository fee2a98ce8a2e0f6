"""Pins of the KL-distillation oracle (Sec. 2.4) against closed forms and special
cases.  CPU only."""
import math

import numpy as np

from oracle import numerics as nm
from oracle.kl import ce_rows, kl_forward, kl_rows, teacher_hidden


def test_kl_of_identical_distributions_is_zero_and_kl_is_nonnegative():
    rng = np.random.default_rng(0)
    z = rng.standard_normal((5, 40))
    assert np.allclose(kl_rows(z, z, 1.0), 0.0, atol=1e-12)
    assert np.allclose(kl_rows(z, z + 3.0, 0.5), 0.0, atol=1e-12)       # shift invariance
    t = rng.standard_normal((5, 40))
    assert np.all(kl_rows(t, z, 1.0) > 0)


def test_kl_two_point_closed_form():
    """p = (a, 1-a), q = (b, 1-b): KL = a log(a/b) + (1-a) log((1-a)/(1-b))."""
    a, b = 0.7, 0.2
    t = np.array([[math.log(a), math.log(1 - a)]])
    z = np.array([[math.log(b), math.log(1 - b)]])
    want = a * math.log(a / b) + (1 - a) * math.log((1 - a) / (1 - b))
    assert abs(kl_rows(t, z, 1.0)[0] - want) < 1e-12
    # temperature T: the distributions of logits / T
    T = 2.0
    pa = a ** (1 / T) / (a ** (1 / T) + (1 - a) ** (1 / T))
    pb = b ** (1 / T) / (b ** (1 / T) + (1 - b) ** (1 / T))
    want_t = pa * math.log(pa / pb) + (1 - pa) * math.log((1 - pa) / (1 - pb))
    assert abs(kl_rows(t, z, T)[0] - want_t) < 1e-12


def test_cross_entropy_of_uniform_logits_is_log_vocab():
    V = 64
    assert np.allclose(ce_rows(np.zeros((3, V)), [0, 5, 63]), math.log(V))


def test_teacher_mean_pools_the_paths():
    """Identical paths pool to that path; the pooled state is RMS-normalised."""
    rng = np.random.default_rng(1)
    x = rng.standard_normal((2, 1, 32))
    H = np.repeat(x, 4, axis=1)
    h = teacher_hidden(H, None, 1e-6, "f32")
    y = x[:, 0] / np.sqrt((x[:, 0] ** 2).mean(axis=1, keepdims=True) + 1e-6)
    np.testing.assert_allclose(h, nm.round_f32(y), rtol=1e-6)
    # opposite paths cancel: the mean is zero and so is its RMSNorm
    H2 = np.concatenate([x, -x], axis=1)
    assert np.allclose(teacher_hidden(H2, None, 1e-6, "f32"), 0.0)


def test_loss_assembly_and_alignment():
    """L_KL = T^2/P * mean over blocks of the sum over the first P positions; draft
    position k is paired with the teacher of position a+k-1 (row k-1 of H_pos) and the
    draft logits of slot k; L = L_CE + alpha L_KL."""
    rng = np.random.default_rng(2)
    n, P, m, d, V, B = 3, 2, 2, 16, 11, 5
    H = rng.standard_normal((n, P, m, d))
    w = rng.standard_normal((V, d)) * 0.3
    z = rng.standard_normal((n, B, V))
    labels = rng.integers(0, V, (n, B - 1))
    T, alpha = 1.5, 0.15
    kl, ce, (L_kl, L_ce, L) = kl_forward(H, None, 1e-6, w, z, labels, P=P, T=T, alpha=alpha,
                                         dtype="f32")
    for s in range(n):
        for k in range(1, P + 1):
            t = teacher_hidden(H[s, k - 1][None], None, 1e-6, "f32") @ w.T
            assert abs(kl[s, k - 1] - kl_rows(t, z[s, k][None], T)[0]) < 1e-12
    assert abs(L_kl - T * T / P * kl.sum(axis=1).mean()) < 1e-12
    assert abs(L_ce - ce.mean()) < 1e-12 and abs(L - (L_ce + alpha * L_kl)) < 1e-12
    # a student equal to the teacher has zero KL
    t_all = np.stack([teacher_hidden(H[s], None, 1e-6, "f32") @ w.T for s in range(n)])
    z2 = z.copy()
    z2[:, 1:P + 1] = t_all
    kl2, _, _ = kl_forward(H, None, 1e-6, w, z2, None, P=P, T=T, alpha=alpha, dtype="f32")
    assert np.allclose(kl2, 0.0, atol=1e-9)
