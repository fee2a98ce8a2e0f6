"""Pins of the sampling oracle (temperature sampling and speculative-sampling
verification) against the published generator, distributional facts and special
cases.  CPU only."""
import numpy as np
import pytest

from oracle.sampling import (PURPOSE_DRAFT, accept_sample, philox4x64_10, sample_tokens,
                             uniforms)


def _softmax(x):
    e = np.exp(x - x.max())
    return e / e.sum()


@pytest.mark.parametrize("key,ctr", [((1, 2), (1, 0, 0, 0)), ((0, 0), (5, 7, 9, 11)),
                                     ((2**64 - 1, 12345), (2**63 + 3, 1, 2**40, 7))])
def test_philox_matches_numpy_bit_generator(key, ctr):
    """numpy's Philox bit generator is Philox4x64-10 and increments its 256-bit counter
    before each block: its first block from counter c - 1 is the block of counter c."""
    c = list(ctr)
    c_prev = c[:]
    c_prev[0] = (c_prev[0] - 1) % 2**64       # no borrow in these cases (c[0] >= 1)
    bg = np.random.Philox(key=np.array(key, dtype=np.uint64),
                          counter=np.array(c_prev, dtype=np.uint64))
    want = bg.random_raw(4)
    got = philox4x64_10(np.array([c], dtype=np.uint64), np.array([key], dtype=np.uint64))[0]
    assert np.array_equal(got, want)


def test_uniforms_on_the_24_bit_grid():
    u = uniforms(11, 2, np.arange(64)[:, None], np.arange(64)[None, :], PURPOSE_DRAFT)
    k = u * 2**24 - 0.5
    assert np.array_equal(k, np.round(k)) and k.min() >= 0 and k.max() < 2**24
    assert 0.0 < u.min() and u.max() < 1.0
    # roughly uniform: mean 1/2, variance 1/12
    assert abs(u.mean() - 0.5) < 0.01 and abs(u.var() - 1 / 12) < 0.01
    # distinct streams and purposes draw different numbers
    assert not np.array_equal(u, uniforms(11, 3, np.arange(64)[:, None], np.arange(64)[None, :], 0))
    assert not np.array_equal(u, uniforms(11, 2, np.arange(64)[:, None], np.arange(64)[None, :], 1))


@pytest.mark.parametrize("T", [1.0, 0.5])
def test_gumbel_max_draws_follow_softmax(T):
    """Frequencies of Gumbel-max draws over 20000 rows match softmax(z / T) within 5 sigma."""
    z = np.array([1.0, 0.2, -0.5, 2.0, 0.0])
    R = 20000
    tok, lse, _ = sample_tokens(np.tile(z, (R, 1)), T, seed=3, stream=1)
    p = _softmax(z / T)
    f = np.bincount(tok, minlength=5) / R
    assert np.all(np.abs(f - p) < 5 * np.sqrt(p * (1 - p) / R) + 1e-12), (f, p)
    assert np.allclose(lse, np.log(np.exp(z / T).sum()))


def test_verification_preserves_the_target_distribution():
    """Speculative sampling is exact: whatever the draft distribution, the first committed
    token is distributed as the target's p_0 (here 20000 independent blocks, K = 2)."""
    V, K, n = 4, 2, 20000
    zq = np.array([[2.0, 0.0, -1.0, 0.5], [0.0, 1.0, 0.0, -2.0]])      # draft logits, slots 1, 2
    zp = np.array([[0.0, 1.5, 0.3, -0.2], [1.0, 0.0, 0.0, 0.0], [0.0, 0.0, 2.0, 0.0]])
    dl = np.broadcast_to(zq, (n, K, V))
    drafts = np.stack([sample_tokens(np.tile(zq[i], (n, 1)), 1.0, seed=8, stream=5 + i)[0]
                       for i in range(K)], axis=1)
    acc, nxt, offs, toks, _, _ = accept_sample(drafts, dl, np.broadcast_to(zp, (n, K + 1, V)),
                                               1.0, seed=9, stream=0)
    first = toks[offs[:-1]]
    p0 = _softmax(zp[0])
    f = np.bincount(first, minlength=V) / n
    assert np.all(np.abs(f - p0) < 5 * np.sqrt(p0 * (1 - p0) / n)), (f, p0)
    # acceptance of slot 1 happens with probability sum_x min(p0, q0)
    q0 = _softmax(zq[0])
    a1 = np.minimum(p0, q0).sum()
    assert abs((acc >= 1).mean() - a1) < 5 * np.sqrt(a1 * (1 - a1) / n)
    assert np.array_equal(np.diff(offs), acc + 1)


def test_identical_distributions_accept_every_draft():
    V, K, n = 6, 3, 50
    rng = np.random.default_rng(0)
    z = rng.standard_normal((K + 1, V))
    drafts = rng.integers(0, V, (n, K))
    acc, nxt, _, _, _, _ = accept_sample(drafts, np.broadcast_to(z[:K], (n, K, V)),
                                         np.broadcast_to(z, (n, K + 1, V)), 1.0, 1, 1)
    assert np.all(acc == K)


def test_draft_outside_the_target_support_is_rejected():
    V, K = 5, 3
    zd = np.zeros((1, K, V))
    zt = np.zeros((1, K + 1, V))
    zt[0, 1, 2] = -1e9                     # the target never produces token 2 at slot 2
    drafts = np.array([[0, 2, 1]])
    for seed in range(20):
        acc, nxt, _, _, _, _ = accept_sample(drafts, zd, zt, 1.0, seed, 0)
        assert acc[0] <= 1
        if acc[0] == 1:
            assert nxt[0] != 2             # the residual max(0, p - q) excludes it


def test_no_drafts_draws_the_bonus_from_the_target():
    V, n = 3, 12000
    zt = np.array([[0.5, -1.0, 1.0]])
    acc, nxt, offs, toks, _, _ = accept_sample(np.zeros((n, 0), dtype=np.int64), np.zeros((n, 0, V)),
                                               np.broadcast_to(zt, (n, 1, V)), 1.0, 4, 2)
    assert np.all(acc == 0) and np.array_equal(toks, nxt)
    p = _softmax(zt[0])
    f = np.bincount(nxt, minlength=V) / n
    assert np.all(np.abs(f - p) < 5 * np.sqrt(p * (1 - p) / n))
