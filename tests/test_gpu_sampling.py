"""GPU parity of temperature sampling (hdf_sample_tokens) and speculative-sampling
verification (hdf_accept_sample) against the oracle, which draws the same Philox
numbers.  Log-sum-exp within 1e-5 relative; a draw is compared where the oracle's
top-2 perturbed-score gap is at least 1e-3 (fp32 against fp64 scores); an acceptance
length where every decision it took has |u q - p| / max(p, q) >= 1e-4."""
import numpy as np
import pytest
import torch

import synth
from oracle.lm_head import lm_head_logits
from oracle.sampling import accept_sample as ref_accept_sample, sample_tokens as ref_sample
from paper_2606_26744_amd import hdf

pytestmark = pytest.mark.gpu
SMARGIN, DMARGIN = 1e-3, 1e-4


def _logits(R, V, seed, scale=2.0):
    g = torch.Generator(device="cuda").manual_seed(seed)
    return (torch.randn((R, V), generator=g, device="cuda") * scale).contiguous()


def _check_sample(lg, T, seed, stream, rows=None):
    R, V = lg.shape
    tok, lse = hdf.sample_tokens(lg, temperature=T, seed=seed, stream_id=stream)
    torch.cuda.synchronize()
    sel = np.arange(R) if rows is None else np.asarray(rows)
    r_tok, r_lse, margin = ref_sample(lg.cpu().numpy()[sel], T, seed, stream, rows=sel)
    np.testing.assert_allclose(lse.cpu().numpy()[sel], r_lse, rtol=1e-5, atol=1e-5)
    ok = margin >= SMARGIN
    assert ok.mean() > 0.9
    assert np.array_equal(tok.cpu().numpy()[sel][ok], r_tok[ok])
    return tok, lse


@pytest.mark.parametrize("R,V,T", [(64, 5000, 1.0), (7, 1001, 0.7), (300, 257, 1.5)])
def test_sample_tokens_vs_oracle(R, V, T):
    print(f"[sample] R={R} V={V} T={T}", flush=True)
    _check_sample(_logits(R, V, R + V), T, seed=11, stream=3)


def test_sample_tokens_row_stride():
    """Rows with a stride larger than the vocabulary (a view into wider logits)."""
    full = _logits(20, 1024, 5)
    _check_sample(full[:, :1000], 1.0, seed=2, stream=0)


def test_sample_full_vocabulary_lm_head_logits():
    """Draws from the full-size LM head's logits (128 rows x 129280), sampled rows."""
    d, V, M = 4096, 129280, 128
    hid = synth.normal([M, d], 1.0, 7, 50, dtype="bf16", device="cuda")
    w = synth.normal([V, d], 0.02, 7, 51, dtype="bf16", device="cuda")
    _, _, lg = hdf.lm_head_argmax(hid, hdf.pack_weight(w), want_logits=True)
    _check_sample(lg, 1.0, seed=21, stream=1, rows=[0, 1, 17, 64, 127])
    torch.cuda.empty_cache()


def _accept_case(n_seq, K, V, T, seed, noise=0.5, forbid=None):
    print(f"[accept_sample] n_seq={n_seq} K={K} V={V} T={T}", flush=True)
    B = K + 1
    draft_lg = _logits(n_seq * B, V, seed)                       # slot rows s*B + k
    g = torch.Generator(device="cuda").manual_seed(seed + 1)
    tgt_lg = torch.empty((n_seq, K + 1, V), device="cuda")
    for s in range(n_seq):
        # the target's logits for draft i resemble the draft's (slot i+1) plus noise
        base = draft_lg[s * B + 1:s * B + B] if K > 0 else draft_lg[s * B:s * B]
        tgt_lg[s, :K] = base + noise * torch.randn((K, V), generator=g, device="cuda")
        tgt_lg[s, K] = 2.0 * torch.randn((V,), generator=g, device="cuda")
    tok, lse = hdf.sample_tokens(draft_lg, temperature=T, seed=seed, stream_id=0)
    if forbid is not None:
        s, i = forbid                                              # draft i of s outside the target
        x = int(tok[s * B + 1 + i])
        tgt_lg[s, i, x] = -1e4
    acc, anc, offs, toks = hdf.accept_sample(tok[1:], draft_lg[1:], lse[1:], tgt_lg, K=K,
                                             draft_stride=B, ld=V, temperature=T, seed=seed,
                                             stream_id=9)
    torch.cuda.synchronize()
    drafts = tok.cpu().numpy().reshape(n_seq, B)[:, 1:]
    dl = draft_lg.cpu().numpy().reshape(n_seq, B, V)[:, 1:]
    r_acc, r_anc, r_offs, r_toks, dmarg, smarg = ref_accept_sample(
        drafts, dl, tgt_lg.cpu().numpy(), T, seed, 9)
    acc, anc = acc.cpu().numpy(), anc.cpu().numpy()
    ok = dmarg >= DMARGIN
    assert ok.mean() > 0.7
    assert np.array_equal(acc[ok], r_acc[ok])
    ok2 = ok & (smarg >= SMARGIN)
    assert np.array_equal(anc[ok2], r_anc[ok2])
    o = offs.cpu().numpy()
    assert np.array_equal(np.diff(o), acc + 1)
    t = toks.cpu().numpy()
    for s in range(n_seq):
        seg = t[o[s]:o[s + 1]]
        assert np.array_equal(seg[:-1], drafts[s, :acc[s]]) and seg[-1] == anc[s]
        if acc[s] < K:
            assert anc[s] != drafts[s, acc[s]]     # a rejected draft is never redrawn
    return acc


def test_accept_sample_vs_oracle():
    acc = _accept_case(24, 15, 3000, 1.0, seed=31)
    print("accept lengths", acc.tolist(), flush=True)


def test_accept_sample_temperature_and_wide_vocab():
    _accept_case(8, 7, 20000, 0.8, seed=32, noise=0.3)


def test_accept_sample_rejects_a_draft_outside_the_target():
    acc = _accept_case(4, 5, 500, 1.0, seed=33, noise=0.05, forbid=(2, 0))
    assert acc[2] == 0


def test_accept_sample_without_drafts_draws_the_bonus():
    _accept_case(16, 0, 700, 1.0, seed=34)
