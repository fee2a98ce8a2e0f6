"""GPU parity of hdf_lm_head_argmax (draft logits and greedy tokens, Sec. 2.3) against
the CPU oracle.  Argmax is bit-exact except on rows whose oracle top-2 margin is
below 1e-2; logits within 1e-4 relative (fp32) or 2e-2 absolute (bf16)."""
import numpy as np
import pytest
import torch

import synth
from oracle.lm_head import lm_head_argmax as ref_lm
from paper_2606_26744_amd import hdf
from tests._tol import assert_abs_close, assert_f32_rows_close

pytestmark = pytest.mark.gpu
MARGIN = 1e-2


def _inputs(M, d, V, dtype, seed):
    wl = synth.Workload("lm", dtype, seed, m=4, d=d)
    hid = synth.normal([M, d], 1.0, seed, 50, dtype=dtype, device="cuda")   # unit-RMS states
    w = synth.normal([V, d], 0.02, seed, 51, dtype=dtype, device="cuda")
    return hid, w


def _check(hid, w, rows=None, want_logits=True, dtype="bf16"):
    M, V = hid.shape[0], w.shape[0]
    print(f"[lm_head] M={M} d={hid.shape[1]} V={V} dtype={dtype}", flush=True)
    am, mx, lg = hdf.lm_head_argmax(hid, hdf.pack_weight(w), want_logits=want_logits)
    torch.cuda.synchronize()
    sel = np.arange(M) if rows is None else np.asarray(rows)
    r_am, r_lg, r_margin = ref_lm(synth.to_numpy_bits(hid)[sel], synth.to_numpy_bits(w))
    g_am = am.cpu().numpy()[sel]
    ok = r_margin >= MARGIN
    print(f"  argmax compared on {int(ok.sum())} of {ok.size} rows (margin >= {MARGIN})",
          flush=True)
    assert ok.mean() > 0.8
    assert np.array_equal(g_am[ok], r_am[ok]), np.nonzero(g_am[ok] != r_am[ok])
    # rows left out: the GPU's pick is one of the oracle's near-ties
    z = r_lg.astype(np.float64)
    assert np.all(z[np.arange(len(sel)), g_am] >= z.max(axis=1) - MARGIN)
    # the GPU's own max logit equals the logit at its argmax, and is the row max
    g_mx = mx.cpu().numpy()[sel]
    if want_logits:
        g_lg = lg[torch.as_tensor(sel, device=lg.device)].cpu().numpy()
        if dtype == "bf16":
            assert_abs_close(g_lg, r_lg, 2e-2, "logits")
        else:
            assert_f32_rows_close(g_lg, r_lg, "logits")
        assert np.array_equal(g_mx, g_lg.max(axis=1))
        assert np.array_equal(g_am, np.argmax(g_lg, axis=1))   # fused argmax = argmax of its logits
    assert_abs_close(g_mx, r_lg.max(axis=1), 2e-2 if dtype == "bf16" else 1e-4, "max logit")
    return am, mx


def test_tiny_fp32():
    hid, w = _inputs(8, 256, 4096, "f32", 60)
    _check(hid, w, dtype="f32")


@pytest.mark.parametrize("M,d,V", [(64, 1024, 32000), (1, 1024, 1000), (130, 512, 1000),
                                   (16, 64, 129), (200, 1024, 32000), (256, 512, 5000),
                                   (300, 256, 3000)])
def test_bf16_shapes(M, d, V):
    hid, w = _inputs(M, d, V, "bf16", M + V)
    _check(hid, w)


def test_full_vocab_block_rows():
    """The full-size step's LM head: 8 sequences x 16 slots, d=4096, V=129280; every row,
    logits included."""
    hid, w = _inputs(128, 4096, 129280, "bf16", 61)
    _check(hid, w, want_logits=True)
    torch.cuda.empty_cache()


def test_ragged_batch_rows():
    """64 sequences x 16 slots (M=1024, eight 128-row tiles): 256 rows, 32 from every row
    tile (first and last rows of each tile among them), logits included."""
    hid, w = _inputs(1024, 4096, 129280, "bf16", 62)
    rng = np.random.default_rng(62)
    rows = sorted({r for t in range(8) for r in
                   [128 * t, 128 * t + 127] + rng.choice(np.arange(128 * t + 1, 128 * t + 127),
                                                         30, replace=False).tolist()})
    assert len(rows) == 256
    _check(hid, w, rows=rows, want_logits=True)
    torch.cuda.empty_cache()


def test_rows_past_one_launch():
    """More rows than one launch takes (2^20; the row offsets of a launch stay in int32
    tile arithmetic): 2^20 + 300 rows of d = 64, V = 129, no logits; the rows around the
    boundary, the first and last rows and 500 others against the oracle, and the keys
    handed back zeroed for the next call."""
    M = (1 << 20) + 300
    hid, w = _inputs(M, 64, 129, "bf16", 65)
    rng = np.random.default_rng(65)
    edge = [0, 1, M - 2, M - 1] + list(range((1 << 20) - 3, (1 << 20) + 3))
    rows = sorted(set(edge) | set(rng.choice(M, 500, replace=False).tolist()))
    _check(hid, w, rows=rows, want_logits=False)
    ws = torch.zeros(hdf.lm_head_workspace(M, 129), dtype=torch.uint8, device="cuda")
    hdf.lm_head_argmax(hid, hdf.pack_weight(w), ws=ws)
    torch.cuda.synchronize()
    assert int(torch.count_nonzero(ws)) == 0
    del hid, ws
    torch.cuda.empty_cache()


def test_ties_take_lowest_index():
    d, V = 128, 3000
    hid, w = _inputs(4, d, V, "bf16", 63)
    w[2999] = w[17]
    w[1200] = w[17]
    hid[0] = (w[17].float() * 40).to(torch.bfloat16)   # row 0's maximum is the tied row
    am, _, lg = hdf.lm_head_argmax(hid, hdf.pack_weight(w), want_logits=True)
    assert am[0].item() == 17
    assert lg[0, 17].item() == lg[0, 1200].item() == lg[0, 2999].item()


@pytest.mark.parametrize("M", [4, 100, 136, 250])
def test_ties_inside_one_tile_take_lowest_index(M):
    """Tied columns inside one 512-column tile, one pair per row, placed so that each
    level of the tile's (max, lowest index) combine decides one pair: the same lane
    (33 vs 40), the two lane halves (4 vs 8), the two 32-column blocks of a wave (20 vs
    36) and different waves (70 vs 200).  M = 4 runs 64-row tiles, M = 100 one 128-row
    tile, M = 136 and 250 one 192- and one 256-row tile (the tie rows repeat from row
    130)."""
    d, V = 128, 3000
    pairs = [(4, 8), (33, 40), (20, 36), (70, 200)]      # (expected, tied higher column)
    hid, w = _inputs(M, d, V, "bf16", 65)
    for lo, hi in pairs:
        w[hi] = w[lo]
    rows = list(range(len(pairs))) + ([130 + i for i in range(len(pairs))] if M > 128 else [])
    for r in rows:
        lo = pairs[r % 130][0]
        hid[r] = (w[lo].float() * 40).to(torch.bfloat16)
    print(f"[lm_head ties] M={M}", flush=True)
    am, _, lg = hdf.lm_head_argmax(hid, hdf.pack_weight(w), want_logits=True)
    torch.cuda.synchronize()
    for r in rows:
        lo, hi = pairs[r % 130]
        assert lg[r, lo].item() == lg[r, hi].item() == lg[r].max().item(), (r, lo, hi)
        assert am[r].item() == lo, (r, am[r].item(), lo)


def test_pack_weight_layout():
    """The packed layout puts (n, k) at (((n/128)(K/16) + k/16)*4 + (n%128)/32)*512
    + ((n%32) + 32((k%16)/8))*8 + k%8 and pads rows to a multiple of 128 with zeros."""
    for dt in (torch.bfloat16, torch.float32):
        N, K = 170, 48
        w = torch.randn(N, K, generator=torch.Generator().manual_seed(5)).to(dt).cuda()
        p = hdf.pack_weight(w).data.cpu()
        R = 256
        assert p.numel() == R * K
        n = torch.arange(R).view(-1, 1)
        k = torch.arange(K).view(1, -1)
        idx = (((n // 128) * (K // 16) + k // 16) * 4 + (n % 128) // 32) * 512 + \
            ((n % 32) + 32 * ((k % 16) // 8)) * 8 + k % 8
        got = p[idx.reshape(-1)].view(R, K)
        assert torch.equal(got[:N], w.cpu())
        assert torch.all(got[N:] == 0)


def test_empty():
    hid = torch.empty((0, 128), dtype=torch.bfloat16, device="cuda")
    w = torch.zeros((10, 128), dtype=torch.bfloat16, device="cuda")
    am, _, _ = hdf.lm_head_argmax(hid, hdf.pack_weight(w))
    assert am.numel() == 0


def test_determinism():
    hid, w = _inputs(128, 1024, 32000, "bf16", 64)
    wp = hdf.pack_weight(w)
    a1, m1, l1 = hdf.lm_head_argmax(hid, wp, want_logits=True)
    a2, m2, l2 = hdf.lm_head_argmax(hid, wp, want_logits=True)
    assert torch.equal(a1, a2) and torch.equal(m1, m2) and torch.equal(l1, l2)
