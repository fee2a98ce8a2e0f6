"""hdf_lm_head_argmax_noalloc, the LM head for callers that cannot allocate, against the
workspace entry point hdf_lm_head_argmax on the same inputs (and both against the
oracle), through the C ABI: two calls in a row, the second with a smaller input, so the
shared key array must come back cleared by the first."""
import ctypes

import numpy as np
import pytest
import torch

import synth
from oracle.lm_head import lm_head_argmax as ref_lm
from paper_2606_26744_amd import hdf
from tests._tol import assert_abs_close

pytestmark = pytest.mark.gpu


def _p(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _run(fn_name, hid, wp, V, with_ws):
    M, d = hid.shape
    am = torch.full((M,), -5, dtype=torch.int32, device="cuda")
    mx = torch.empty(M, dtype=torch.float32, device="cuda")
    lg = torch.empty((M, V), dtype=torch.float32, device="cuda")
    L = hdf.lib()
    s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if with_ws:
        ws = torch.zeros(int(L.hdf_lm_head_workspace(M, V)), dtype=torch.uint8, device="cuda")
        st = L.hdf_lm_head_argmax(_p(hid), ctypes.c_void_p(wp.data_ptr()), M, d, V, hdf.HDF_BF16,
                                  _p(am), _p(mx), _p(lg), _p(ws), ws.numel(), s)
    else:
        st = L.hdf_lm_head_argmax_noalloc(_p(hid), ctypes.c_void_p(wp.data_ptr()), M, d, V,
                                          hdf.HDF_BF16, _p(am), _p(mx), _p(lg), s)
    assert st == 0, L.hdf_last_error()
    torch.cuda.synchronize()
    return am.cpu().numpy(), mx.cpu().numpy(), lg.cpu().numpy()


@pytest.mark.parametrize("M,d,V,seed", [(200, 256, 3000, 71), (16, 128, 1000, 72)])
def test_no_alloc_matches_workspace_entry_point(M, d, V, seed):
    """Run in this order: 200 rows (two row tiles), then 16 rows."""
    print(f"[no_alloc] M={M} d={d} V={V}", flush=True)
    hid = synth.normal([M, d], 1.0, seed, 50, device="cuda")
    w = synth.normal([V, d], 0.02, seed, 51, device="cuda")
    wp = hdf.pack_weight(w)
    a0, m0, l0 = _run("ws", hid, wp, V, True)
    a1, m1, l1 = _run("noalloc", hid, wp, V, False)
    assert np.array_equal(a1, a0) and np.array_equal(m1, m0) and np.array_equal(l1, l0)
    # and both meet the oracle's bounds
    r_am, r_lg, r_mg = ref_lm(synth.to_numpy_bits(hid), synth.to_numpy_bits(w))
    ok = r_mg >= 1e-2
    assert ok.mean() > 0.8 and np.array_equal(a1[ok], r_am[ok])
    assert_abs_close(l1, r_lg, 2e-2, "logits")
    # a second no-alloc call on the same inputs gives the same bits (keys came back zeroed)
    a2, m2, l2 = _run("noalloc", hid, wp, V, False)
    assert np.array_equal(a2, a1) and np.array_equal(m2, m1)


def test_no_alloc_rejects_oversized_calls_before_launching():
    L = hdf.lib()
    f = ctypes.c_void_p(4096)
    st = L.hdf_lm_head_argmax_noalloc(f, f, 65537, 128, 1000, hdf.HDF_BF16, f, None, None, None)
    assert hdf.STATUS[st] == "HDF_E_UNSUPPORTED"
    st = L.hdf_lm_head_argmax_noalloc(f, f, 10, 100, 1000, hdf.HDF_BF16, f, None, None, None)
    assert hdf.STATUS[st] == "HDF_E_INVALID"
    st = L.hdf_lm_head_argmax_noalloc(None, None, 0, 128, 1000, hdf.HDF_BF16, None, None, None, None)
    assert hdf.STATUS[st] == "HDF_OK"
