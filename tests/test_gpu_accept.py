"""GPU parity of hdf_accept (greedy verification) against the CPU oracle: bit-exact."""
import numpy as np
import pytest
import torch

import synth
from oracle.accept import accept as ref_accept
from paper_2606_26744_amd import hdf

pytestmark = pytest.mark.gpu


def _run(draft, target, **kw):
    d = torch.as_tensor(np.asarray(draft, dtype=np.int32)).cuda()
    t = torch.as_tensor(np.asarray(target, dtype=np.int32)).cuda()
    acc, anc, offs, toks = hdf.accept(d, t, **kw)
    torch.cuda.synchronize()
    return acc.cpu().numpy(), anc.cpu().numpy(), offs.cpu().numpy(), toks.cpu().numpy()


def _compare(draft, target):
    print(f"[accept] n_seq={len(target)} K={np.asarray(target).shape[1] - 1}", flush=True)
    acc, anc, offs, toks = _run(draft, target)
    r_acc, r_anc, r_offs, r_toks = ref_accept(np.asarray(draft), np.asarray(target))
    assert np.array_equal(acc, r_acc)
    assert np.array_equal(anc, r_anc)
    assert np.array_equal(offs, r_offs)
    assert np.array_equal(toks[:offs[-1]], r_toks)


def test_hand_built():
    acc, anc, offs, toks = _run([[5, 7, 9]], [[5, 7, 2, 4]])
    assert acc[0] == 2 and anc[0] == 2 and list(toks[:3]) == [5, 7, 2] and list(offs) == [0, 3]
    acc, anc, _, _ = _run([[5, 7, 9]], [[5, 7, 9, 4]])
    assert acc[0] == 3 and anc[0] == 4
    acc, anc, _, _ = _run([[1, 7, 9]], [[5, 7, 9, 4]])
    assert acc[0] == 0 and anc[0] == 5


def test_k_zero():
    d = torch.zeros((3, 1), dtype=torch.int32, device="cuda")
    t = torch.tensor([[4], [5], [6]], dtype=torch.int32, device="cuda")
    acc, anc, offs, toks = hdf.accept(d, t, K=0, draft_stride=1)
    assert acc.tolist() == [0, 0, 0] and anc.tolist() == [4, 5, 6] and offs.tolist() == [0, 1, 2, 3]


@pytest.mark.parametrize("n_seq,K,p", [(8, 15, 0.8), (64, 15, 0.5), (3000, 15, 0.9), (5, 200, 0.99),
                                        (4, 63, 1.0), (4, 64, 1.0), (3, 128, 1.0), (2, 1024, 1.0),
                                        (1025, 64, 0.95)])
def test_random_geometric(n_seq, K, p):
    rng = np.random.default_rng(n_seq + K)
    drafts = rng.integers(0, 129280, (n_seq, K))
    tgt = synth.make_targets(drafts, [p] * n_seq, 129280, seed=3)
    _compare(drafts, tgt)


def test_drafts_read_from_argmax_layout():
    """Drafts are slots 1..B-1 of the LM head's argmax array (row s*B + k)."""
    n_seq, B = 6, 16
    rng = np.random.default_rng(7)
    am = rng.integers(0, 1000, (n_seq * B,)).astype(np.int32)
    drafts = am.reshape(n_seq, B)[:, 1:]
    tgt = synth.make_targets(drafts, [0.7] * n_seq, 1000, seed=4)
    am_d = torch.as_tensor(am).cuda()
    t = torch.as_tensor(tgt).cuda()
    acc, anc, offs, toks = hdf.accept(am_d[1:], t, K=B - 1, draft_stride=B)
    r = ref_accept(drafts, tgt)
    assert np.array_equal(acc.cpu().numpy(), r[0]) and np.array_equal(anc.cpu().numpy(), r[1])
    assert np.array_equal(offs.cpu().numpy(), r[2])
