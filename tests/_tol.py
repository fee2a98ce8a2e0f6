"""Parity tolerances, stated once.

fp32 outputs: per row, max|gpu - ref| <= 1e-4 * max|ref| (relative to the row's
scale; elementwise relative error is meaningless near zero).
bf16 outputs: |gpu - ref| <= max(2e-2, one bf16 ulp of ref) elementwise.  Both
sides round the same exact quantity to bf16; a float32-vs-float64 difference far
below one ulp can still land on opposite sides of a rounding boundary, which
moves the stored value by exactly one ulp, so one ulp is allowed even where it
exceeds 2e-2 (|ref| >= 4).
"""
import numpy as np

# End-to-end bounds for the drafter's bf16 chain, set from the measured spread of the
# oracle itself when every pre-rounding value is perturbed by a relative 1e-7 (small
# configuration) or 1e-6 (the full-size shape, d=4096, V=129280; the size of an fp32
# dot product's rounding error over K = 4096), tests/test_bf16_chain_sensitivity.py.
# Measured at full size: block-state row RMS up to 4e-3 (6e-3 at 4e-6), logits up to
# 2.5e-2 (3.4e-2 at 4e-6), argmax flips only on rows whose top-2 margin is below 3.2e-3.
STATE_RMS_REL = 1e-2      # block states / cached K,V: per-row RMS difference / RMS
STATE_ABS = 4e-2          # ... and elementwise max(STATE_ABS, STATE_ULPS ulp)
STATE_ULPS = 4
E2E_LOGIT_ABS = 5e-2      # logits of a whole step (the LM head alone meets 2e-2)
E2E_MARGIN = 2e-2         # end-to-end argmax compared where the oracle's top-2 margin
                          # clears this; below it the GPU's pick must be a near-tie
STAGE_MARGIN = 1e-2       # the LM-head stage on identical inputs (the stated bound)


def bf16_ulp(x):
    a = np.abs(np.asarray(x, dtype=np.float64))
    a = np.maximum(a, 2.0 ** -126)
    return 2.0 ** (np.floor(np.log2(a)) - 7)


def assert_bf16_close(got, ref, what=""):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    tol = np.maximum(2e-2, bf16_ulp(ref))
    err = np.abs(got - ref)
    bad = err > tol
    if bad.any():
        i = np.argwhere(bad)[0]
        raise AssertionError(f"{what}: {int(bad.sum())} of {bad.size} outside tolerance; first at "
                             f"{tuple(i)}: got {got[tuple(i)]!r} ref {ref[tuple(i)]!r}")
    return int(np.count_nonzero(got != ref))


def assert_bf16_state_close(got, ref, what="", ulps=STATE_ULPS, rms_rel=STATE_RMS_REL,
                            abs_tol=STATE_ABS):
    """Drafter-internal bf16 states (block states, cached K/V) after a chain of bf16
    storage points.  Both sides round the same quantities, but one rounding that lands
    on the other side of a boundary (1 ulp) perturbs every later GEMM output slightly,
    which moves further roundings: the chain leaves isolated elements a few ulps apart
    with neither side more exact.  Bound: |gpu - ref| <= max(abs_tol, ulps * ulp(ref))
    elementwise, and per row the RMS difference <= rms_rel * RMS(ref)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    tol = np.maximum(abs_tol, ulps * bf16_ulp(ref))
    err = np.abs(got - ref)
    bad = err > tol
    if bad.any():
        i = np.argwhere(bad)[0]
        raise AssertionError(f"{what}: {int(bad.sum())} of {bad.size} outside bound; first at "
                             f"{tuple(i)}: got {got[tuple(i)]!r} ref {ref[tuple(i)]!r}")
    g2 = got.reshape(got.shape[0], -1)
    r2 = ref.reshape(ref.shape[0], -1)
    rms_err = np.sqrt(np.mean((g2 - r2) ** 2, axis=1))
    rms_ref = np.maximum(np.sqrt(np.mean(r2 ** 2, axis=1)), 1e-30)
    worst = float((rms_err / rms_ref).max())
    assert worst <= rms_rel, f"{what}: row RMS difference {worst:.2e} > {rms_rel}"
    return int(np.count_nonzero(got != ref)), worst


def assert_f32_rows_close(got, ref, what="", rel=1e-4):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    g2 = got.reshape(got.shape[0], -1) if got.ndim > 1 else got[:, None]
    r2 = ref.reshape(ref.shape[0], -1) if ref.ndim > 1 else ref[:, None]
    scale = np.maximum(np.abs(r2).max(axis=1), 1e-30)
    err = np.abs(g2 - r2).max(axis=1)
    bad = err > rel * scale
    if bad.any():
        i = int(np.argmax(bad))
        raise AssertionError(f"{what}: {int(bad.sum())} rows outside {rel} relative; row {i}: "
                             f"max err {err[i]!r} vs scale {scale[i]!r}")


def assert_abs_close(got, ref, atol, what=""):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    err = np.abs(got - ref)
    if (err > atol).any():
        i = np.unravel_index(int(np.argmax(err)), err.shape)
        raise AssertionError(f"{what}: max abs err {err[i]!r} at {i} > {atol}")
