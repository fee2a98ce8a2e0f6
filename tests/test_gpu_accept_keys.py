"""GPU tests of hdf_lm_head_argmax_keys + hdf_accept_keys, called through the C ABI: the
same argmax, max logit, acceptance lengths, anchors and committed tokens, bit for bit, as
hdf_lm_head_argmax followed by hdf_accept on its drafts (slots 1..B-1 of every block), and
the workspace handed back zeroed.  The acceptance itself is pinned to the oracle in
test_gpu_accept.py and the LM head in test_gpu_lm_head.py; the greedy step through this
path is compared with the oracle in test_gpu_step.py."""
import numpy as np
import pytest
import torch

import synth
from paper_2606_26744_amd import hdf

pytestmark = pytest.mark.gpu


def _reference(hid, w_lm, tg, B):
    am, mx, _ = hdf.lm_head_argmax(hid, w_lm)
    acc, anc, offs, toks = hdf.accept(am[1:], tg, K=B - 1, draft_stride=B)
    return [t.cpu().numpy() for t in (am, mx, acc, anc, offs, toks)]


@pytest.mark.parametrize("n_seq,B,d,V,p", [(8, 16, 4096, 129280, 0.8), (3, 1, 256, 3000, 0.5),
                                           (64, 16, 1024, 32000, 0.7), (100, 16, 512, 5000, 0.9),
                                           (2, 40, 256, 1000, 1.0), (1, 2, 64, 129, 0.0)])
def test_keys_path_equals_the_two_calls(n_seq, B, d, V, p):
    print(f"[accept_keys] n_seq={n_seq} B={B} d={d} V={V}", flush=True)
    M = n_seq * B
    hid = synth.normal([M, d], 1.0, 70 + B, 50, dtype="bf16", device="cuda")
    w = hdf.pack_weight(synth.normal([V, d], 0.02, 70 + B, 51, dtype="bf16", device="cuda"))
    # targets: the reference path's drafts kept with probability p (geometric acceptance)
    am0, _, _ = hdf.lm_head_argmax(hid, w)
    drafts = am0.cpu().numpy().reshape(n_seq, B)[:, 1:]
    tg = torch.as_tensor(synth.make_targets(drafts, [p] * n_seq, V, seed=B)).cuda()
    ref = _reference(hid, w, tg, B)
    ws = torch.zeros(hdf.lm_head_workspace(M, V), dtype=torch.uint8, device="cuda")
    am = torch.full((M,), -5, dtype=torch.int32, device="cuda")
    mx = torch.full((M,), -5.0, dtype=torch.float32, device="cuda")
    for call in range(2):   # the second call reuses the workspace the first handed back
        hdf.lm_head_argmax_keys(hid, w, ws)
        got = hdf.accept_keys(ws, tg, B, argmax=am, max_logit=mx)
        torch.cuda.synchronize()
        g_acc, g_anc, g_offs, g_toks = [t.cpu().numpy() for t in got]
        r_am, r_mx, r_acc, r_anc, r_offs, r_toks = ref
        assert np.array_equal(am.cpu().numpy(), r_am)
        assert np.array_equal(mx.cpu().numpy(), r_mx)
        assert np.array_equal(g_acc, r_acc) and np.array_equal(g_anc, r_anc)
        assert np.array_equal(g_offs, r_offs)
        assert np.array_equal(g_toks[:g_offs[-1]], r_toks[:r_offs[-1]])
        assert int(torch.count_nonzero(ws)) == 0
    print(f"  mean accepted {g_acc.mean():.2f}", flush=True)


def test_keys_path_without_max_logit_or_commits():
    n_seq, B, d, V = 4, 16, 256, 2000
    M = n_seq * B
    hid = synth.normal([M, d], 1.0, 90, 50, dtype="bf16", device="cuda")
    w = hdf.pack_weight(synth.normal([V, d], 0.02, 90, 51, dtype="bf16", device="cuda"))
    tg = torch.randint(0, V, (n_seq, B), dtype=torch.int32, device="cuda")
    r_am, _, r_acc, r_anc, _, _ = _reference(hid, w, tg, B)
    ws = torch.zeros(hdf.lm_head_workspace(M, V), dtype=torch.uint8, device="cuda")
    am = torch.empty(M, dtype=torch.int32, device="cuda")
    hdf.lm_head_argmax_keys(hid, w, ws)
    acc, anc, offs, toks = hdf.accept_keys(ws, tg, B, argmax=am, commits=False)
    torch.cuda.synchronize()
    assert offs is None and toks is None
    assert np.array_equal(am.cpu().numpy(), r_am)
    assert np.array_equal(acc.cpu().numpy(), r_acc) and np.array_equal(anc.cpu().numpy(), r_anc)
    assert int(torch.count_nonzero(ws)) == 0
