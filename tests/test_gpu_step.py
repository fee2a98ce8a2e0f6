"""End-to-end parity of one drafter step (reduce -> draft block -> LM head argmax ->
accept) on the GPU against the oracle chain on the CPU, over every sequence of the
batch.

Three comparisons per step:
  1. Stage parity of the LM head on identical inputs: the oracle's LM head applied to
     the GPU's own block states.  Logits within 2e-2 (bf16) / 1e-4 relative (fp32) and
     argmax bit-exact wherever that oracle's top-2 margin is >= 1e-2 (the stated bound),
     on at least 80% of the rows.
  2. The whole chain against the oracle run from scratch on the same inputs.  Reduced
     rows at the reducer's bounds, block states at the bf16-chain bounds, logits within
     E2E_LOGIT_ABS, argmax bit-exact wherever the oracle's margin is >= E2E_MARGIN (at
     least 80% of the rows).  On every other row the GPU's pick must be a near-tie: its
     oracle logit within E2E_MARGIN of the oracle's maximum.
  3. Acceptance: the GPU's accept_len, next_anchor and commits equal oracle.accept on
     the GPU's own drafts for every sequence (integer stage, bit-exact), and equal the
     from-scratch oracle's for every sequence.  The synthetic targets copy the oracle's
     drafts with the workload's probability; at a slot whose oracle margin is below
     E2E_MARGIN the target is the oracle's lowest-logit token instead, outside the
     slot's near-tie set, so both sides reject there whatever near-tie they pick and
     every acceptance length is comparable (the same holds for uniform targets).
The bounds and their derivation are in tests/_tol.py."""
import numpy as np
import pytest
import torch

import synth
from oracle.accept import accept as ref_accept
from oracle.lm_head import lm_head_argmax as ref_lm
from oracle.drafter import draft_block as ref_draft
from oracle.reducer import hc_reduce as ref_reduce
from oracle.numerics import as_f64
from paper_2606_26744_amd import hdf
from paper_2606_26744_amd.step import StepBuffers, drafter_step
from tests._case import DraftCase, bits
from tests._tol import (E2E_LOGIT_ABS, E2E_MARGIN, STAGE_MARGIN, assert_abs_close,
                        assert_bf16_close, assert_bf16_state_close, assert_f32_rows_close)

pytestmark = pytest.mark.gpu


def _step_case(wl, ctx, new, *, sub=0, uniform_targets=False):
    n_seq = len(ctx)
    seqs = list(range(n_seq))
    print(f"[step] {wl.name} n_seq={n_seq} ctx={ctx[:8]} new={new[:8]}", flush=True)
    n_new = sum(new)
    red = synth.reducer_inputs(wl, n_new, device="cuda", sub=sub)
    case = DraftCase(wl, ctx, new, random_norms=False, sub=sub,
                     y_from=torch.empty((n_new, wl.d), dtype=red["H"].dtype, device="cuda"))
    B = case.B
    bf = wl.dtype == "bf16"
    W = case.oracle_weights()
    wlm = bits(case.w["w_lm"])
    no = case.new_offsets.tolist()
    Hn = bits(red["H"])
    Wg, bg = bits(red["W_g"]), bits(red["b_g"])
    # Oracle chain from scratch: reduce -> draft block -> LM head.
    ys = [ref_reduce(Hn[no[s]:no[s + 1]], Wg, bg, dtype=wl.dtype)[0] for s in seqs]
    toks = bits(case.tokens)
    hid_ref = ref_draft(W, ys, toks, kv_prefix=case.prefix)
    am_ref, lg_ref, margin = ref_lm(hid_ref, wlm)
    drafts_ref = am_ref.reshape(n_seq, B)[:, 1:]
    MARGIN = E2E_MARGIN if bf else STAGE_MARGIN
    V = wl.drafter.vocab
    if uniform_targets:
        rng = np.random.default_rng([wl.seed, 99, sub])
        targets = rng.integers(0, V, (n_seq, B)).astype(np.int32)
    else:
        targets = synth.make_targets(drafts_ref, (wl.match_p or [0.8] * n_seq)[:n_seq], V, seed=wl.seed,
                                     sub=sub)
    near = margin.reshape(n_seq, B)[:, 1:] < MARGIN
    low = np.argmin(lg_ref.reshape(n_seq, B, V)[:, 1:], axis=2).astype(np.int32)
    targets[:, :B - 1] = np.where(near, low, targets[:, :B - 1])
    tg = torch.as_tensor(targets).cuda()
    bufs = StepBuffers(case.h, n_seq, B, n_new, case.max_ctx, wl.m)
    out = drafter_step(case.h, bufs, H_new=red["H"], W_g=red["W_g"], b_g=red["b_g"],
                       new_offsets=case.new_offsets, ctx_len=case.ctx_len, max_ctx=case.max_ctx,
                       kv_offsets=case.kv_offsets, kv_k=case.kv_k, kv_vt=case.kv_vt,
                       tokens=case.tokens, targets=tg, logits=True)
    torch.cuda.synchronize()
    M = n_seq * B
    # Reduced rows
    for s in seqs:
        y = bits(out["Y"][no[s]:no[s + 1]])
        if bf:
            assert_bf16_close(as_f64(y), ys[s], "Y")
        else:
            assert_f32_rows_close(y, ys[s], "Y")
    hid = bits(out["hidden"])
    lg = out["logits"][:M].cpu().numpy()
    am = out["argmax"].cpu().numpy()[:M]
    # 1. The LM-head stage on the GPU's own block states.
    am_st, lg_st, mg_st = ref_lm(hid, wlm)
    if bf:
        assert_abs_close(lg, lg_st, 2e-2, "logits (LM-head stage)")
    else:
        assert_f32_rows_close(lg, lg_st, "logits (LM-head stage)")
    ok_st = mg_st >= STAGE_MARGIN
    assert np.array_equal(am[ok_st], am_st[ok_st]), np.nonzero(am[ok_st] != am_st[ok_st])
    # 2. The whole chain against the oracle from scratch.
    if bf:
        _, worst = assert_bf16_state_close(as_f64(hid), hid_ref, "hidden")
        assert_abs_close(lg, lg_ref, E2E_LOGIT_ABS, "logits")
    else:
        assert_f32_rows_close(hid, hid_ref, "hidden")
        assert_f32_rows_close(lg, lg_ref, "logits")
        worst = 0.0
    ok = margin >= MARGIN
    assert np.array_equal(am[ok], am_ref[ok]), np.nonzero(am[ok] != am_ref[ok])
    # rows left out: the GPU's pick is one of the oracle's near-ties
    z = lg_ref.astype(np.float64)
    picked = z[np.arange(M), am]
    near_ok = picked >= z.max(axis=1) - MARGIN
    assert near_ok.all(), np.nonzero(~near_ok)
    # 3. Acceptance: on the GPU's own drafts (always exact) and against the oracle chain.
    acc = out["accept_len"].cpu().numpy()
    anc = out["next_anchor"].cpu().numpy()
    offs = out["commit_offsets"].cpu().numpy()
    ctoks = out["commit_tokens"].cpu().numpy()
    g_acc, g_anc, g_offs, g_toks = ref_accept(am.reshape(n_seq, B)[:, 1:], targets)
    assert np.array_equal(acc, g_acc) and np.array_equal(anc, g_anc)
    assert np.array_equal(offs, g_offs) and np.array_equal(ctoks[:g_offs[-1]], g_toks)
    r_acc, r_anc, _, _ = ref_accept(drafts_ref, targets)
    assert np.array_equal(acc, r_acc) and np.array_equal(anc, r_anc), (acc, r_acc)
    compared = n_seq
    n_ok, n_st = int(ok.sum()), int(ok_st.sum())
    dlog = float(np.abs(lg.astype(np.float64) - lg_ref).max())
    print(f"  argmax: stage compared {n_st}/{M} (margin >= {STAGE_MARGIN}), end-to-end "
          f"compared {n_ok}/{M} (margin >= {MARGIN}), near-ties validated {M - n_ok}; "
          f"rows under 1e-2: {int((margin < 1e-2).sum())}, under 5e-2: "
          f"{int((margin < 5e-2).sum())}; max |dlogit| end-to-end {dlog:.4f}, block-state "
          f"row RMS {worst:.2e}; acceptance compared {compared}/{n_seq}, accept lens "
          f"{acc.tolist()}", flush=True)
    assert n_st >= 0.8 * M and n_ok >= 0.8 * M
    assert compared >= 0.5 * n_seq
    return out


def test_tiny_fp32_step():
    wl = synth.tiny_fp32()
    _step_case(wl, [64], [64], uniform_targets=True)


def test_small_bf16_step_cold():
    wl = synth.small_bf16()
    _step_case(wl, [512] * 4, [512] * 4)


def test_small_bf16_step_warm():
    wl = synth.small_bf16()
    _step_case(wl, [512] * 4, [16] * 4, sub=1)


def test_full_size_step():
    """The benchmark's configuration: 8 x 2048 context, 16 new rows per sequence, all
    eight sequences."""
    wl = synth.drafter_full()
    _step_case(wl, [2048] * 8, [16] * 8)
    torch.cuda.empty_cache()


def test_ragged_step():
    """Six sequences of the ragged workload (contexts from its U[1024, 16384] draw), every
    one checked."""
    wl = synth.ragged_decode()
    ctx = wl.ctx_lens[:6]
    _step_case(wl, ctx, [16] * 6, sub=2)
    torch.cuda.empty_cache()


def test_sampled_step_wiring():
    """The temperature-sampled step (drafter_step_sampled): its draws come from its own
    logits and its verification equals the oracle's on the same logits, tokens and
    target logits (checks the slot offsets and strides of the sampled path)."""
    from oracle.sampling import accept_sample as ref_accept_sample, sample_tokens as ref_sample
    from paper_2606_26744_amd.step import SampledStepBuffers, drafter_step_sampled
    wl = synth.small_bf16()
    ctx, new = [512] * 4, [16] * 4
    n_new = sum(new)
    red = synth.reducer_inputs(wl, n_new, device="cuda", sub=5)
    case = DraftCase(wl, ctx, new, random_norms=False, sub=5,
                     y_from=torch.empty((n_new, wl.d), dtype=red["H"].dtype, device="cuda"))
    n_seq, B, V = len(ctx), case.B, wl.drafter.vocab
    bufs = StepBuffers(case.h, n_seq, B, n_new, case.max_ctx, wl.m)
    sb = SampledStepBuffers(case.h, n_seq, B)
    g = torch.Generator(device="cuda").manual_seed(1)
    tgt = 2.0 * torch.randn((n_seq, B, V), generator=g, device="cuda")
    kw = dict(H_new=red["H"], W_g=red["W_g"], b_g=red["b_g"], new_offsets=case.new_offsets,
              ctx_len=case.ctx_len, max_ctx=case.max_ctx, kv_offsets=case.kv_offsets,
              kv_k=case.kv_k, kv_vt=case.kv_vt, tokens=case.tokens)
    out = drafter_step_sampled(case.h, bufs, sb, target_logits=tgt, temperature=1.0, seed=7,
                               round_id=3, **kw)
    torch.cuda.synchronize()
    lg = out["logits"].cpu().numpy()
    tok = out["tokens"].cpu().numpy()
    r_tok, _, margin = ref_sample(lg, 1.0, 7, 6)                  # stream 2 * round_id
    ok = margin >= 1e-3
    assert ok.mean() > 0.9 and np.array_equal(tok[ok], r_tok[ok])
    drafts = tok.reshape(n_seq, B)[:, 1:]
    dl = lg.reshape(n_seq, B, V)[:, 1:]
    r_acc, r_anc, _, _, dmarg, smarg = ref_accept_sample(drafts, dl, tgt.cpu().numpy(), 1.0, 7, 7)
    acc = out["accept_len"].cpu().numpy()
    anc = out["next_anchor"].cpu().numpy()
    good = dmarg >= 1e-4
    assert good.mean() > 0.5
    assert np.array_equal(acc[good], r_acc[good])
    good &= smarg >= 1e-3
    assert np.array_equal(anc[good], r_anc[good])
