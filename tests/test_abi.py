"""Host-side checks of the C ABI (no GPU needed): the library loads, exports every
symbol include/hdf.h declares, and rejects bad arguments before touching a device."""
import ctypes
import os
import re

import pytest

from paper_2606_26744_amd import hdf

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_symbols():
    src = open(os.path.join(ROOT, "include", "hdf.h")).read()
    return sorted(set(re.findall(r"\b(hdf_[a-z0-9_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    L = hdf.lib()
    declared = _declared_symbols()
    assert declared, "no declarations found"
    for name in declared:
        assert hasattr(L, name), name
    assert sorted(hdf.EXPORTS) == declared
    assert L.hdf_version() >= 100


def _status(st):
    return hdf.STATUS[st]


def test_reduce_validation():
    L = hdf.lib()
    P = ctypes.c_void_p
    fake = P(4096)   # never dereferenced: every call below fails validation first
    bad = [
        dict(n=-1, m=4, d=64, dt=1),
        dict(n=1, m=0, d=64, dt=1),
        dict(n=1, m=9, d=64, dt=1),
        dict(n=1, m=4, d=60, dt=1),       # bf16 needs d % 8 == 0
        dict(n=1, m=4, d=6, dt=0),        # fp32 needs d % 4 == 0
        dict(n=1, m=4, d=64, dt=7),
    ]
    for b in bad:
        st = L.hdf_hc_reduce(fake, fake, fake, b["n"], b["m"], b["d"], b["dt"], None, fake, None, None)
        assert _status(st) == "HDF_E_INVALID", b
    st = L.hdf_hc_reduce(fake, fake, fake, 1, 4, 8200, 1, None, fake, None, None)
    assert _status(st) == "HDF_E_UNSUPPORTED"
    st = L.hdf_hc_reduce(None, fake, fake, 1, 4, 64, 1, None, fake, None, None)
    assert _status(st) == "HDF_E_INVALID"
    assert b"null" in L.hdf_last_error()
    p = hdf.ReduceParams(0.0, 1.0, 0.0, 0)
    st = L.hdf_hc_reduce(fake, fake, fake, 1, 4, 64, 1, ctypes.byref(p), fake, None, None)
    assert _status(st) == "HDF_E_INVALID"
    # misaligned pointers
    st = L.hdf_hc_reduce(P(4098), fake, fake, 1, 4, 64, 1, None, fake, None, None)
    assert _status(st) == "HDF_E_INVALID"
    # n_tok = 0 is a no-op that succeeds without touching anything
    st = L.hdf_hc_reduce(None, None, None, 0, 4, 64, 1, None, None, None, None)
    assert _status(st) == "HDF_OK" and L.hdf_last_error() == b""


def test_accept_validation():
    L = hdf.lib()
    fake = ctypes.c_void_p(4096)
    assert _status(L.hdf_accept(fake, 15, fake, -1, 15, fake, fake, None, None, None)) == "HDF_E_INVALID"
    assert _status(L.hdf_accept(fake, 15, fake, 1, 1025, fake, fake, None, None, None)) == "HDF_E_INVALID"
    assert _status(L.hdf_accept(fake, 3, fake, 1, 15, fake, fake, None, None, None)) == "HDF_E_INVALID"
    assert _status(L.hdf_accept(fake, 15, None, 1, 15, fake, fake, None, None, None)) == "HDF_E_INVALID"
    assert _status(L.hdf_accept(None, 15, None, 0, 15, None, None, None, None, None)) == "HDF_OK"


def test_keys_path_validation():
    L = hdf.lib()
    fake = ctypes.c_void_p(4096)
    odd = ctypes.c_void_p(4100)
    # hdf_lm_head_argmax_keys: width, vocabulary, pointers, workspace size and alignment
    assert _status(L.hdf_lm_head_argmax_keys(fake, fake, 16, 100, 1000, 1, fake, 1 << 20, None)) == "HDF_E_INVALID"
    assert _status(L.hdf_lm_head_argmax_keys(fake, fake, 16, 128, 0, 1, fake, 1 << 20, None)) == "HDF_E_INVALID"
    assert _status(L.hdf_lm_head_argmax_keys(None, fake, 16, 128, 1000, 1, fake, 1 << 20, None)) == "HDF_E_INVALID"
    assert _status(L.hdf_lm_head_argmax_keys(fake, fake, 16, 128, 1000, 1, fake, 8, None)) == "HDF_E_WORKSPACE"
    assert _status(L.hdf_lm_head_argmax_keys(fake, fake, 16, 128, 1000, 1, odd, 1 << 20, None)) == "HDF_E_INVALID"
    assert _status(L.hdf_lm_head_argmax_keys(None, None, 0, 128, 1000, 1, None, 0, None)) == "HDF_OK"
    # hdf_accept_keys: sizes, pointers, workspace alignment
    assert _status(L.hdf_accept_keys(fake, -1, 16, fake, None, fake, fake, fake, None, None, None)) == "HDF_E_INVALID"
    assert _status(L.hdf_accept_keys(fake, 2, 0, fake, None, fake, fake, fake, None, None, None)) == "HDF_E_INVALID"
    assert _status(L.hdf_accept_keys(fake, 2, 1026, fake, None, fake, fake, fake, None, None, None)) == "HDF_E_INVALID"
    assert _status(L.hdf_accept_keys(fake, 2, 16, None, None, fake, fake, fake, None, None, None)) == "HDF_E_INVALID"
    assert _status(L.hdf_accept_keys(odd, 2, 16, fake, None, fake, fake, fake, None, None, None)) == "HDF_E_INVALID"
    assert _status(L.hdf_accept_keys(fake, 1 << 30, 16, fake, None, fake, fake, fake, None, None, None)) == "HDF_E_UNSUPPORTED"
    assert _status(L.hdf_accept_keys(None, 0, 16, None, None, None, None, None, None, None, None)) == "HDF_OK"


def test_rope_table_host_values():
    import math
    t = hdf.rope_table(5, 8, 10000.0)
    for p in range(5):
        for i in range(4):
            a = p * 10000.0 ** (-2.0 * i / 8)
            assert t[p, i, 0].item() == pytest.approx(math.cos(a), abs=1e-7)
            assert t[p, i, 1].item() == pytest.approx(math.sin(a), abs=1e-7)
    L = hdf.lib()
    assert _status(L.hdf_rope_table(None, 4, 8, 1e4)) == "HDF_E_INVALID"
    buf = (ctypes.c_float * 64)()
    assert _status(L.hdf_rope_table(buf, 4, 7, 1e4)) == "HDF_E_INVALID"
    assert _status(L.hdf_rope_table(buf, 4, 8, 0.0)) == "HDF_E_INVALID"


def test_pack_weight_validation():
    L = hdf.lib()
    fake = ctypes.c_void_p(4096)
    assert L.hdf_packed_weight_bytes(70, 48, 1) == 128 * 48 * 2
    assert L.hdf_packed_weight_bytes(70, 40, 1) == 0          # K % 16 != 0
    assert L.hdf_packed_weight_bytes(0, 48, 0) == 0
    assert _status(L.hdf_pack_weight(fake, None, 70, 48, 1, None)) == "HDF_E_INVALID"
    assert _status(L.hdf_pack_weight(fake, fake, 70, 48, 1, None)) == "HDF_E_INVALID"   # in place
    assert _status(L.hdf_pack_weight(fake, ctypes.c_void_p(8192), 70, 40, 1, None)) == "HDF_E_INVALID"
    assert _status(L.hdf_pack_weight(fake, ctypes.c_void_p(8192), 70, 48, 5, None)) == "HDF_E_INVALID"


def test_kv_rows_validation():
    """hdf_kv_write_rows / hdf_kv_read_rows reject bad sizes, layouts and pointers on the
    host; n_rows = 0 is a no-op."""
    L = hdf.lib()
    f = ctypes.c_void_p(4096)

    def w(n=10, rows=None, row0=0, layer=0, nh=2, hd=64, dt=1, kc=f, vc=f, cap=128, k=f, v=f):
        return _status(L.hdf_kv_write_rows(k, v, n, rows, row0, layer, nh, hd, dt, kc, vc, cap,
                                           None))

    def r(n=10, rows=None, row0=0, layer=0, nh=2, hd=64, dt=1, kc=f, vc=f, cap=128, k=f, v=f):
        return _status(L.hdf_kv_read_rows(kc, vc, cap, layer, nh, hd, dt, rows, row0, n, k, v,
                                          None))
    for call in (w, r):
        assert call(n=-1) == "HDF_E_INVALID"
        assert call(layer=-1) == "HDF_E_INVALID"
        assert call(hd=96) == "HDF_E_UNSUPPORTED"
        assert call(cap=100) == "HDF_E_INVALID"              # not a multiple of 64
        assert call(cap=0) == "HDF_E_INVALID"
        assert call(dt=3) == "HDF_E_INVALID"
        assert call(row0=120) == "HDF_E_INVALID"             # rows 120..129 leave a 128-row cache
        assert call(kc=None, vc=None) == "HDF_E_INVALID"     # nothing to copy
        assert call(k=None) == "HDF_E_INVALID"               # a cache array without rows
        assert call(kc=ctypes.c_void_p(4100)) == "HDF_E_INVALID"   # misaligned
        assert call(n=0, kc=None, vc=None, k=None, v=None) == "HDF_OK"


def _fake_drafter(L_layers=1, d=256, nh=4, hd=64):
    fake = ctypes.c_void_p(4096)
    arr = (ctypes.c_void_p * L_layers)(*([4096] * L_layers))
    w = hdf.Drafter()
    w.n_layers, w.d, w.n_heads, w.head_dim, w.d_ff, w.vocab = L_layers, d, nh, hd, 512, 1000
    w.dtype, w.eps = hdf.HDF_BF16, 1e-6
    w.tok_emb = fake
    w.ctx_norm = None
    for f in ("attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down"):
        setattr(w, f, ctypes.cast(arr, ctypes.POINTER(ctypes.c_void_p)))
    w.final_norm = None
    w.rope_cs = None
    w.rope_max_pos = 0
    return w, arr


def test_draft_block_paged_validation():
    """The paged entry point rejects a missing page table, a table too narrow for
    max_ctx and an out-of-range page count before any launch; n_seq = 0 is a no-op."""
    L = hdf.lib()
    w, keep = _fake_drafter()
    fake = ctypes.c_void_p(4096)
    ws = 1 << 30

    def call(page_table, max_pages, kv_pages, n_seq=2, max_ctx=100):
        return _status(L.hdf_draft_block_paged(ctypes.byref(w), n_seq, 16, fake, max_ctx, fake,
                                               fake, None, 8, page_table, max_pages, fake, fake,
                                               kv_pages, fake, fake, fake, ws, None))
    assert call(None, 4, 8) == "HDF_E_INVALID"                 # no page table
    assert call(fake, 1, 8) == "HDF_E_INVALID"                 # 64 rows < max_ctx = 100
    assert call(fake, -1, 8) == "HDF_E_INVALID"
    assert call(fake, 4, 1 << 25) == "HDF_E_INVALID"           # kv_pages * 64 >= 2^31
    assert call(fake, 4, -1) == "HDF_E_INVALID"
    assert call(None, 0, 0, n_seq=0, max_ctx=0) == "HDF_OK"
    # the contiguous entry point still requires its offsets
    st = L.hdf_draft_block(ctypes.byref(w), 2, 16, fake, 100, fake, fake, 8, None, fake, fake,
                           128, fake, fake, fake, ws, None)
    assert _status(st) == "HDF_E_INVALID"


def test_advance_context_validation():
    """Null inputs, a negative count, block tokens without anchors and a block size outside
    [1, 1025] are rejected on the host; n_seq = 0 is a no-op."""
    L = hdf.lib()
    fake = ctypes.c_void_p(4096)

    def call(n, acc, ctx, anchor=None, toks=None, B=0):
        return _status(L.hdf_advance_context(n, acc, ctx, fake, anchor, toks, B, None))
    assert call(-1, fake, fake) == "HDF_E_INVALID"
    assert call(2, None, fake) == "HDF_E_INVALID"
    assert call(2, fake, None) == "HDF_E_INVALID"
    assert call(2, fake, fake, None, fake, 16) == "HDF_E_INVALID"     # tokens need anchors
    assert call(2, fake, fake, fake, fake, 0) == "HDF_E_INVALID"
    assert call(2, fake, fake, fake, fake, 1026) == "HDF_E_INVALID"
    assert call(1 << 22, fake, fake, fake, fake, 1024) == "HDF_E_UNSUPPORTED"
    assert call(0, None, None) == "HDF_OK"


def test_fc_reduce_validation():
    L = hdf.lib()
    fake = ctypes.c_void_p(4096)
    ws = 1 << 30
    call = lambda n, m, d, dt=1, H=fake: _status(L.hdf_fc_reduce(H, fake, None, n, m, d, dt, fake,
                                                                 fake, ws, None))
    assert call(-1, 4, 256) == "HDF_E_INVALID"
    assert call(1, 0, 256) == "HDF_E_INVALID"
    assert call(1, 9, 256) == "HDF_E_INVALID"
    assert call(1, 1, 36) == "HDF_E_INVALID"          # m*d = 36: not a multiple of 64
    assert call(1, 4, 256, H=None) == "HDF_E_INVALID"
    assert call(0, 4, 256, H=None) == "HDF_OK"
    assert L.hdf_fc_reduce_workspace(10, 4, 256, 1) > 0
    assert L.hdf_fc_reduce_workspace(10, 4, 30, 1) == 0
    # too small a workspace
    st = L.hdf_fc_reduce(fake, fake, None, 10, 4, 256, 1, fake, fake, 16, None)
    assert _status(st) == "HDF_E_WORKSPACE"


def test_binding_rejects_wrong_dtypes_and_sizes():
    """The C ABI takes bare pointers, so the binding checks the dtype and size of the index
    and output tensors before any call (here with host tensors: the check comes first)."""
    import torch
    i32 = torch.zeros(64, dtype=torch.int32)
    with pytest.raises(ValueError, match="argmax"):
        hdf.accept_keys(torch.zeros(64 * 8, dtype=torch.uint8), i32.view(4, 16), 16,
                        argmax=torch.zeros(64, dtype=torch.int64))
    with pytest.raises(ValueError, match="max_logit"):
        hdf.accept_keys(torch.zeros(64 * 8, dtype=torch.uint8), i32.view(4, 16), 16,
                        argmax=i32, max_logit=torch.zeros(64, dtype=torch.float64))
    with pytest.raises(ValueError, match="target"):
        hdf.accept_keys(torch.zeros(64 * 8, dtype=torch.uint8), i32.view(4, 16).long(), 16,
                        argmax=i32)
    with pytest.raises(ValueError, match="accept_len"):
        hdf.accept(i32.view(4, 16), i32.view(4, 16),
                   out=(torch.zeros(3, dtype=torch.int32), i32[:4], i32[:5], i32))
    with pytest.raises(ValueError, match="draft"):
        hdf.accept(i32.view(4, 16).float(), i32.view(4, 16))
    H = torch.zeros((2, 4, 64), dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="b_g"):
        hdf.hc_reduce(H, torch.zeros((4, 256), dtype=torch.bfloat16), torch.zeros(4, dtype=torch.bfloat16))
    with pytest.raises(ValueError, match="W_g"):
        hdf.hc_reduce(H, torch.zeros((4, 256), dtype=torch.float32), torch.zeros(4))
    with pytest.raises(ValueError, match="Y"):
        hdf.hc_reduce(H, torch.zeros((4, 256), dtype=torch.bfloat16), torch.zeros(4),
                      Y=torch.zeros((1, 64), dtype=torch.bfloat16))
