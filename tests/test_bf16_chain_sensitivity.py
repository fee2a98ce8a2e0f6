"""How far apart two correct bf16 drafter pipelines can land.

Every stored intermediate of the drafter (normed states, Q/K/V, attention output,
SiLU*up) is rounded to bf16.  Two implementations that both compute each rounded
quantity from exact-enough arithmetic (the GPU in fp32, the oracle in fp64) still
disagree wherever a pre-rounding value lies within their tiny arithmetic difference
of a bf16 rounding boundary, and every such one-ulp disagreement perturbs all later
GEMM outputs a little, moving more roundings.  This test measures that spread on the
oracle itself: it perturbs every pre-rounding value by 1e-7 relative (below fp32
precision) and records how far the final block states and logits move.  The
end-to-end tolerances of the GPU parity tests (tests/_tol.py) are set from these
figures; the test fails if the chain ever becomes much less sensitive (which would
mean the tolerances are looser than they need to be) or much more.  It runs at the
small configuration with a 1e-7 perturbation and at the full-size shape (d=4096,
V=129280, four sequences of 2048 positions) with 1e-6, about the relative rounding
error of an fp32 dot product over K = 4096 terms.
"""
import numpy as np

import synth
import oracle.drafter as od
import oracle.numerics as nm
from oracle.drafter import Weights, draft_block
from oracle.lm_head import lm_head_argmax
from tests._tol import E2E_LOGIT_ABS, E2E_MARGIN, STATE_RMS_REL


def test_bf16_chain_spread_sets_the_end_to_end_tolerances(monkeypatch):
    wl = synth.small_bf16()
    w = synth.drafter_weights(wl, device="cpu")
    b = synth.to_numpy_bits
    wb = {k: ([b(x) for x in v] if isinstance(v, list) else b(v)) for k, v in w.items()}
    dr = wl.drafter
    W = Weights(wb, d=dr.d, n_layers=dr.n_layers, n_heads=dr.n_heads, head_dim=dr.head_dim,
                d_ff=dr.d_ff, vocab=dr.vocab, dtype="bf16")
    wl.n_seq = 2
    ys = [b(synth.reduced_states(wl, 512, sub=s)) for s in range(2)]
    toks = b(synth.block_tokens(wl))
    ref = draft_block(W, ys, toks)
    rng = np.random.default_rng(0)
    orig = nm.store

    def noisy(x, dtype):
        x = np.asarray(x, dtype=np.float64)
        return orig(x * (1 + 1e-7 * rng.standard_normal(x.shape)), dtype)

    monkeypatch.setattr(od, "store", noisy)
    pert = draft_block(W, ys, toks)
    monkeypatch.setattr(od, "store", orig)
    d = pert - ref
    changed = np.mean(d != 0)
    rms = np.sqrt((d ** 2).mean(1)) / np.sqrt((ref ** 2).mean(1))
    _, lg0, _ = lm_head_argmax(ref, wb["w_lm"])
    _, lg1, _ = lm_head_argmax(pert, wb["w_lm"])
    dl = np.abs(lg1.astype(np.float64) - lg0).max()
    print(f"changed {changed:.1%}, row RMS rel max {rms.max():.2e}, logits max {dl:.4f}")
    assert changed > 0.3                      # most elements move
    assert 1e-3 < rms.max() < STATE_RMS_REL   # the state tolerance sits above the spread
    assert 5e-3 < dl < E2E_LOGIT_ABS          # and so does the end-to-end logit tolerance


def test_bf16_chain_spread_at_full_size(monkeypatch):
    """The full-size shape: 4 sequences x 2048 positions (16 new rows projected, the rest
    a cached prefix), d=4096, 32 x 128 heads, F=12288, V=129280."""
    wl = synth.drafter_full()
    wl.n_seq = n_seq = 4
    w = synth.drafter_weights(wl, device="cpu")
    b = synth.to_numpy_bits
    wb = {k: ([b(x) for x in v] if isinstance(v, list) else b(v)) for k, v in w.items()}
    del w
    dr = wl.drafter
    W = Weights(wb, d=dr.d, n_layers=dr.n_layers, n_heads=dr.n_heads, head_dim=dr.head_dim,
                d_ff=dr.d_ff, vocab=dr.vocab, dtype="bf16")
    T, n = wl.ctx_lens[0], wl.new_rows
    pre = []
    for s in range(n_seq):
        k, v = synth.kv_prefix(wl, T - n, 0, sub=s)
        pre.append([(b(k), b(v))])
    ys = [b(synth.reduced_states(wl, n, sub=s)) for s in range(n_seq)]
    toks = b(synth.block_tokens(wl))
    ref = draft_block(W, ys, toks, kv_prefix=pre)
    w_lm = wb["w_lm"]                  # bf16 bits: the oracle decodes them a block at a time
    am0, lg0, mg0 = lm_head_argmax(ref, w_lm)
    rng = np.random.default_rng(0)
    orig = nm.store

    def noisy(x, dtype):
        x = np.asarray(x, dtype=np.float64)
        return orig(x * (1 + 1e-6 * rng.standard_normal(x.shape)), dtype)

    monkeypatch.setattr(od, "store", noisy)
    pert = draft_block(W, ys, toks, kv_prefix=pre)
    monkeypatch.setattr(od, "store", orig)
    am1, lg1, _ = lm_head_argmax(pert, w_lm)
    d = pert - ref
    changed = np.mean(d != 0)
    rms = np.sqrt((d ** 2).mean(1)) / np.sqrt((ref ** 2).mean(1))
    dl = np.abs(lg1.astype(np.float64) - lg0).max()
    flips = np.nonzero(am1 != am0)[0]
    print(f"full size: changed {changed:.1%}, row RMS rel max {rms.max():.2e}, logits max "
          f"{dl:.4f}, argmax flips at margins {mg0[flips].round(4).tolist()}; rows with margin "
          f"< 1e-2: {int((mg0 < 1e-2).sum())}, < 2e-2: {int((mg0 < 2e-2).sum())}, < 5e-2: "
          f"{int((mg0 < 5e-2).sum())} of {mg0.size}")
    assert changed > 0.3
    assert 1e-3 < rms.max() < STATE_RMS_REL
    assert 5e-3 < dl < E2E_LOGIT_ABS
    assert np.all(mg0[flips] < E2E_MARGIN)   # a flip only where the argmax is a near-tie
