"""Python binding of libhdf (ctypes).  Argument marshalling only.

Every computation runs in the HIP kernels of libhdf.so; this module turns torch
tensors into device pointers, picks the current HIP stream, allocates output
tensors with torch (device memory only) and raises on a non-OK status.  There is
no fallback: if the library is missing, loading fails loudly.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libhdf.so")

HDF_F32, HDF_BF16 = 0, 1
STATUS = {0: "HDF_OK", 1: "HDF_E_INVALID", 2: "HDF_E_UNSUPPORTED", 3: "HDF_E_WORKSPACE",
          4: "HDF_E_HIP"}

# Every symbol include/hdf.h declares.
EXPORTS = ("hdf_last_error", "hdf_version", "hdf_hc_reduce", "hdf_rope_table",
           "hdf_packed_weight_bytes", "hdf_pack_weight",
           "hdf_kv_cache_bytes", "hdf_draft_block_workspace", "hdf_draft_block",
           "hdf_draft_block_paged", "hdf_fc_reduce_workspace", "hdf_fc_reduce",
           "hdf_lm_head_workspace", "hdf_lm_head_argmax", "hdf_accept",
           "hdf_sample_workspace", "hdf_sample_tokens", "hdf_accept_sample_workspace",
           "hdf_accept_sample", "hdf_kl_forward_workspace", "hdf_kl_forward",
           "hdf_advance_context", "hdf_kv_write_rows", "hdf_kv_read_rows",
           "hdf_lm_head_argmax_noalloc", "hdf_lm_head_argmax_keys", "hdf_accept_keys")


class HdfError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


class ReduceParams(ctypes.Structure):
    _fields_ = [("eps", ctypes.c_float), ("gate_scale", ctypes.c_float),
                ("gate_offset", ctypes.c_float), ("per_path_norm", ctypes.c_int)]


class Drafter(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int), ("d", ctypes.c_int), ("n_heads", ctypes.c_int),
                ("head_dim", ctypes.c_int), ("d_ff", ctypes.c_int), ("vocab", ctypes.c_int),
                ("dtype", ctypes.c_int), ("eps", ctypes.c_float),
                ("tok_emb", ctypes.c_void_p), ("ctx_norm", ctypes.c_void_p),
                ("attn_norm", ctypes.POINTER(ctypes.c_void_p)),
                ("w_qkv", ctypes.POINTER(ctypes.c_void_p)),
                ("w_o", ctypes.POINTER(ctypes.c_void_p)),
                ("mlp_norm", ctypes.POINTER(ctypes.c_void_p)),
                ("w_gate_up", ctypes.POINTER(ctypes.c_void_p)),
                ("w_down", ctypes.POINTER(ctypes.c_void_p)),
                ("final_norm", ctypes.c_void_p), ("rope_cs", ctypes.c_void_p),
                ("rope_max_pos", ctypes.c_int)]


_lib = None
_P, _I, _I64, _SZ, _F = (ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_size_t,
                         ctypes.c_float)


def lib() -> ctypes.CDLL:
    """Load libhdf.so (built in-tree by paper_2606_26744_amd.build)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with "
                          "`python -m paper_2606_26744_amd.build` (no fallback exists)")
    L = ctypes.CDLL(LIB_PATH)
    L.hdf_last_error.restype = ctypes.c_char_p
    L.hdf_last_error.argtypes = []
    L.hdf_version.restype = _I
    L.hdf_hc_reduce.restype = _I
    L.hdf_hc_reduce.argtypes = [_P, _P, _P, _I64, _I, _I, _I, ctypes.POINTER(ReduceParams), _P, _P, _P]
    L.hdf_rope_table.restype = _I
    L.hdf_rope_table.argtypes = [_P, _I, _I, ctypes.c_double]
    L.hdf_packed_weight_bytes.restype = _SZ
    L.hdf_packed_weight_bytes.argtypes = [_I, _I, _I]
    L.hdf_pack_weight.restype = _I
    L.hdf_pack_weight.argtypes = [_P, _P, _I, _I, _I, _P]
    L.hdf_kv_cache_bytes.restype = _SZ
    L.hdf_kv_cache_bytes.argtypes = [ctypes.POINTER(Drafter), _I64]
    L.hdf_draft_block_workspace.restype = _SZ
    L.hdf_draft_block_workspace.argtypes = [ctypes.POINTER(Drafter), _I, _I, _I64, _I]
    L.hdf_draft_block.restype = _I
    L.hdf_draft_block.argtypes = [ctypes.POINTER(Drafter), _I, _I, _P, _I, _P, _P, _I64, _P, _P, _P,
                                  _I64, _P, _P, _P, _SZ, _P]
    L.hdf_draft_block_paged.restype = _I
    L.hdf_draft_block_paged.argtypes = [ctypes.POINTER(Drafter), _I, _I, _P, _I, _P, _P, _P, _I64,
                                        _P, _I, _P, _P, _I64, _P, _P, _P, _SZ, _P]
    L.hdf_kv_write_rows.restype = _I
    L.hdf_kv_write_rows.argtypes = [_P, _P, _I64, _P, _I64, _I, _I, _I, _I, _P, _P, _I64, _P]
    L.hdf_kv_read_rows.restype = _I
    L.hdf_kv_read_rows.argtypes = [_P, _P, _I64, _I, _I, _I, _I, _P, _I64, _I64, _P, _P, _P]
    L.hdf_advance_context.restype = _I
    L.hdf_advance_context.argtypes = [_I, _P, _P, _P, _P, _P, _I, _P]
    L.hdf_fc_reduce_workspace.restype = _SZ
    L.hdf_fc_reduce_workspace.argtypes = [_I64, _I, _I, _I]
    L.hdf_fc_reduce.restype = _I
    L.hdf_fc_reduce.argtypes = [_P, _P, _P, _I64, _I, _I, _I, _P, _P, _SZ, _P]
    L.hdf_lm_head_workspace.restype = _SZ
    L.hdf_lm_head_workspace.argtypes = [_I64, _I]
    L.hdf_lm_head_argmax.restype = _I
    L.hdf_lm_head_argmax.argtypes = [_P, _P, _I64, _I, _I, _I, _P, _P, _P, _P, _SZ, _P]
    L.hdf_lm_head_argmax_noalloc.restype = _I
    L.hdf_lm_head_argmax_noalloc.argtypes = [_P, _P, _I64, _I, _I, _I, _P, _P, _P, _P]
    L.hdf_accept.restype = _I
    L.hdf_accept.argtypes = [_P, _I, _P, _I, _I, _P, _P, _P, _P, _P]
    L.hdf_lm_head_argmax_keys.restype = _I
    L.hdf_lm_head_argmax_keys.argtypes = [_P, _P, _I64, _I, _I, _I, _P, _SZ, _P]
    L.hdf_accept_keys.restype = _I
    L.hdf_accept_keys.argtypes = [_P, _I, _I, _P, _P, _P, _P, _P, _P, _P, _P]
    _U64 = ctypes.c_uint64
    L.hdf_sample_workspace.restype = _SZ
    L.hdf_sample_workspace.argtypes = [_I64, _I]
    L.hdf_sample_tokens.restype = _I
    L.hdf_sample_tokens.argtypes = [_P, _I64, _I, _I64, _F, _U64, _U64, _P, _P, _P, _SZ, _P]
    L.hdf_accept_sample_workspace.restype = _SZ
    L.hdf_accept_sample_workspace.argtypes = [_I, _I, _I]
    L.hdf_accept_sample.restype = _I
    L.hdf_accept_sample.argtypes = [_P, _I, _P, _P, _I64, _P, _I, _I, _I, _F, _U64, _U64, _P, _P,
                                    _P, _P, _P, _SZ, _P]
    L.hdf_kl_forward_workspace.restype = _SZ
    L.hdf_kl_forward_workspace.argtypes = [_I, _I, _I, _I, _I, _I]
    L.hdf_kl_forward.restype = _I
    L.hdf_kl_forward.argtypes = [_P, _I, _P, _F, _P, _I, _I, _I, _P, _I64, _I, _P, _I, _I, _F, _F,
                                 _P, _P, _P, _P, _SZ, _P]
    _lib = L
    return L


def _check(st: int):
    if st != 0:
        raise HdfError(st, lib().hdf_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return HDF_BF16
    if t.dtype == torch.float32:
        return HDF_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _dev(*ts):
    for t in ts:
        if t is not None:
            if not t.is_cuda:
                raise ValueError("libhdf takes device tensors")
            if not t.is_contiguous():
                raise ValueError("libhdf takes contiguous tensors")


def _typed(t: Optional[torch.Tensor], dtype, numel: int, what: str):
    """The C ABI takes bare pointers, so a tensor of another dtype or too few elements
    would be read or written past its meaning; checked here instead."""
    if t is not None and (t.dtype != dtype or t.numel() < numel):
        raise ValueError(f"{what} must be a {dtype} tensor of at least {numel} elements "
                         f"(got {t.dtype}, {t.numel()})")


# ----------------------------------------------------------------------------- reducer

def hc_reduce(H: torch.Tensor, W_g: torch.Tensor, b_g: torch.Tensor, *, eps: float = 1e-6,
              gate_scale: float = 1.0, gate_offset: float = 0.0, per_path_norm: bool = False,
              Y: Optional[torch.Tensor] = None, alpha: Optional[torch.Tensor] = None,
              want_alpha: bool = False, stream=None):
    """hdf_hc_reduce: H [n_tok, m, d], W_g [m, m*d], b_g [m] fp32 -> (Y [n_tok, d], alpha)."""
    n, m, d = H.shape
    if Y is None:
        Y = torch.empty((n, d), dtype=H.dtype, device=H.device)
    if alpha is None and want_alpha:
        alpha = torch.empty((n, m), dtype=torch.float32, device=H.device)
    _typed(W_g, H.dtype, m * m * d, "W_g")
    _typed(b_g, torch.float32, m, "b_g")
    _typed(Y, H.dtype, n * d, "Y")
    _typed(alpha, torch.float32, n * m, "alpha")
    _dev(H, W_g, b_g, Y, alpha)
    p = ReduceParams(eps, gate_scale, gate_offset, int(per_path_norm))
    _check(lib().hdf_hc_reduce(_ptr(H), _ptr(W_g), _ptr(b_g), n, m, d, _dt(H), ctypes.byref(p),
                               _ptr(Y), _ptr(alpha), _stream(stream)))
    return Y, alpha


def fc_reduce(H: torch.Tensor, W_fc: "PackedWeight", b_fc: Optional[torch.Tensor] = None, *,
              Y: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None, stream=None):
    """hdf_fc_reduce: H [n_tok, m, d], W_fc packed [d][m*d], b_fc [d] fp32 or None ->
    Y [n_tok, d]."""
    n, m, d = H.shape
    if W_fc.N != d or W_fc.K != m * d:
        raise ValueError("W_fc must be a packed [d][m*d] weight")
    if Y is None:
        Y = torch.empty((n, d), dtype=H.dtype, device=H.device)
    need = int(lib().hdf_fc_reduce_workspace(n, m, d, _dt(H)))
    if ws is None or ws.numel() < need:
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=H.device)
    _dev(H, W_fc.data, b_fc, Y, ws)
    _check(lib().hdf_fc_reduce(_ptr(H), W_fc.data_ptr(), _ptr(b_fc), n, m, d, _dt(H), _ptr(Y),
                               _ptr(ws), ws.numel(), _stream(stream)))
    return Y


# ----------------------------------------------------------------------------- accept

def accept(draft: torch.Tensor, target: torch.Tensor, *, K: Optional[int] = None,
           draft_stride: Optional[int] = None, commits: bool = True, out=None, stream=None):
    """hdf_accept.  draft: int32 with row s at s*draft_stride (a [n_seq, >=K] tensor or a
    view into a bigger array), target [n_seq, K+1] int32.  out: optional preallocated
    (accept_len, next_anchor, commit_offsets, commit_tokens)."""
    n_seq = target.shape[0]
    K = target.shape[1] - 1 if K is None else K
    if draft_stride is None:
        draft_stride = draft.stride(0) if draft.dim() == 2 else K
    dev = target.device
    if out is not None:
        acc, anc, offs, toks = out
    else:
        acc = torch.empty(n_seq, dtype=torch.int32, device=dev)
        anc = torch.empty(n_seq, dtype=torch.int32, device=dev)
        offs = torch.empty(n_seq + 1, dtype=torch.int32, device=dev) if commits else None
        toks = (torch.empty(max(1, n_seq * (K + 1)), dtype=torch.int32, device=dev)
                if commits else None)
    _typed(target, torch.int32, n_seq * (K + 1), "target")
    if draft.dtype != torch.int32:
        raise ValueError("draft must be int32")
    for t, k, what in ((acc, n_seq, "accept_len"), (anc, n_seq, "next_anchor"),
                       (offs, n_seq + 1, "commit_offsets"), (toks, n_seq * (K + 1), "commit_tokens")):
        _typed(t, torch.int32, k, what)
    _dev(target, acc, anc, offs, toks)
    if not draft.is_cuda:
        raise ValueError("libhdf takes device tensors")
    _check(lib().hdf_accept(_ptr(draft), draft_stride, _ptr(target), n_seq, K, _ptr(acc),
                            _ptr(anc), _ptr(offs), _ptr(toks), _stream(stream)))
    return acc, anc, offs, toks


def advance_context(accept_len: torch.Tensor, ctx_len: torch.Tensor,
                    new_counts: Optional[torch.Tensor] = None, stream=None,
                    next_anchor: Optional[torch.Tensor] = None,
                    block_tokens: Optional[torch.Tensor] = None):
    """hdf_advance_context: ctx_len += accept_len + 1 and new_counts = accept_len + 1, on
    the device (int32 [n_seq] tensors; ctx_len in place); with block_tokens (int32
    [n_seq, B], contiguous) also block_tokens[s, 0] = next_anchor[s]."""
    n_seq = ctx_len.shape[0]
    for t in (accept_len, ctx_len, new_counts, next_anchor):
        if t is not None and (t.dtype != torch.int32 or t.numel() != n_seq):
            raise ValueError("advance_context takes int32 [n_seq] tensors")
    B = 0
    if block_tokens is not None:
        if next_anchor is None:
            raise ValueError("advance_context: block_tokens needs next_anchor")
        if (block_tokens.dtype != torch.int32 or block_tokens.dim() != 2
                or block_tokens.shape[0] != n_seq or not block_tokens.is_contiguous()):
            raise ValueError("advance_context: block_tokens must be contiguous int32 [n_seq, B]")
        B = block_tokens.shape[1]
    _dev(accept_len, ctx_len, new_counts, next_anchor, block_tokens)
    _check(lib().hdf_advance_context(n_seq, _ptr(accept_len), _ptr(ctx_len), _ptr(new_counts),
                                     _ptr(next_anchor), _ptr(block_tokens), B,
                                     _stream(stream)))


# ----------------------------------------------------------------------------- sampling

def sample_tokens(logits: torch.Tensor, *, temperature: float = 1.0, seed: int = 0,
                  stream_id: int = 0, want_tokens: bool = True, ws=None, out=None, stream=None):
    """hdf_sample_tokens: logits [rows, vocab] fp32 -> (tokens [rows] int32 or None,
    lse [rows] fp32)."""
    rows, V = logits.shape
    dev = logits.device
    if out is None:
        tok = torch.empty(rows, dtype=torch.int32, device=dev) if want_tokens else None
        lse = torch.empty(rows, dtype=torch.float32, device=dev)
    else:
        tok, lse = out
    need = int(lib().hdf_sample_workspace(rows, V))
    if ws is None or ws.numel() < need:
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    if logits.dtype != torch.float32 or logits.stride(1) != 1:
        raise ValueError("logits must be fp32 with unit column stride")
    _check(lib().hdf_sample_tokens(_ptr(logits), rows, V, logits.stride(0), float(temperature),
                                   int(seed), int(stream_id), _ptr(tok), _ptr(lse), _ptr(ws),
                                   ws.numel(), _stream(stream)))
    return tok, lse


def accept_sample(draft: torch.Tensor, draft_logits: torch.Tensor, draft_lse: torch.Tensor,
                  target_logits: torch.Tensor, *, K: int, draft_stride: int, ld: int,
                  temperature: float = 1.0, seed: int = 0, stream_id: int = 0, ws=None,
                  stream=None):
    """hdf_accept_sample.  draft / draft_logits / draft_lse are base pointers (tensors
    or views) addressed as in hdf.h; target_logits [n_seq, K+1, vocab] fp32."""
    n_seq, _, V = target_logits.shape
    dev = target_logits.device
    acc = torch.empty(n_seq, dtype=torch.int32, device=dev)
    anc = torch.empty(n_seq, dtype=torch.int32, device=dev)
    offs = torch.empty(n_seq + 1, dtype=torch.int32, device=dev)
    toks = torch.empty(max(1, n_seq * (K + 1)), dtype=torch.int32, device=dev)
    need = int(lib().hdf_accept_sample_workspace(n_seq, K, V))
    if ws is None or ws.numel() < need:
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    _dev(target_logits, acc, ws)
    _check(lib().hdf_accept_sample(_ptr(draft), draft_stride, _ptr(draft_logits), _ptr(draft_lse),
                                   ld, _ptr(target_logits), n_seq, K, V, float(temperature),
                                   int(seed), int(stream_id), _ptr(acc), _ptr(anc), _ptr(offs),
                                   _ptr(toks), _ptr(ws), ws.numel(), _stream(stream)))
    return acc, anc, offs, toks


def kl_forward(H_pos: torch.Tensor, w_lm: "PackedWeight", student_logits: torch.Tensor, *,
               B: int, P: int, gamma: Optional[torch.Tensor] = None, eps: float = 1e-6,
               labels: Optional[torch.Tensor] = None, temperature: float = 1.0,
               alpha: float = 0.1, ws=None, stream=None):
    """hdf_kl_forward: H_pos [n_seq, P, m, d], student_logits [n_seq*B, V] fp32 ->
    (kl [n_seq, P], ce [n_seq, B-1] or None, loss [3] = L_KL, L_CE, L)."""
    n_seq, P_, m, d = H_pos.shape
    if P_ != P:
        raise ValueError("H_pos must hold P positions per block")
    V = w_lm.N
    dev = H_pos.device
    kl = torch.empty((n_seq, P), dtype=torch.float32, device=dev)
    ce = torch.empty((n_seq, B - 1), dtype=torch.float32, device=dev) if labels is not None else None
    loss = torch.empty(3, dtype=torch.float32, device=dev)
    need = int(lib().hdf_kl_forward_workspace(n_seq, B, P, d, V, _dt(H_pos)))
    if ws is None or ws.numel() < need:
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    if student_logits.dtype != torch.float32 or student_logits.stride(1) != 1:
        raise ValueError("student_logits must be fp32 with unit column stride")
    _dev(H_pos, w_lm.data, gamma, labels, kl, ws)
    _check(lib().hdf_kl_forward(_ptr(H_pos), m, _ptr(gamma), float(eps), w_lm.data_ptr(), d, V,
                                _dt(H_pos), _ptr(student_logits), student_logits.stride(0), B,
                                _ptr(labels), n_seq, P, float(temperature), float(alpha),
                                _ptr(kl), _ptr(ce), _ptr(loss), _ptr(ws), ws.numel(),
                                _stream(stream)))
    return kl, ce, loss


# ----------------------------------------------------------------------------- weights

class PackedWeight:
    """A weight W[N][K] in the library's packed layout (hdf_pack_weight)."""

    def __init__(self, data: torch.Tensor, N: int, K: int):
        self.data, self.N, self.K = data, N, K

    @property
    def dtype(self):
        return self.data.dtype

    def data_ptr(self):
        return self.data.data_ptr()


def pack_weight(w: torch.Tensor, stream=None) -> PackedWeight:
    """Packs a row-major [N][K] device weight with hdf_pack_weight."""
    N, K = w.shape
    _dev(w)
    nbytes = int(lib().hdf_packed_weight_bytes(N, K, _dt(w)))
    if nbytes == 0:
        raise ValueError(f"cannot pack a {N} x {K} weight (K must be a multiple of 16)")
    out = torch.empty(nbytes // w.element_size(), dtype=w.dtype, device=w.device)
    _check(lib().hdf_pack_weight(_ptr(w), _ptr(out), N, K, _dt(w), _stream(stream)))
    return PackedWeight(out, N, K)


# ----------------------------------------------------------------------------- LM head

def lm_head_workspace(M: int, vocab: int) -> int:
    return int(lib().hdf_lm_head_workspace(M, vocab))


def lm_head_argmax(hidden: torch.Tensor, w_lm: PackedWeight, *, want_logits: bool = False,
                   want_max: bool = True, ws: Optional[torch.Tensor] = None, out=None,
                   logits_out: Optional[torch.Tensor] = None, stream=None):
    """hdf_lm_head_argmax: hidden [M, d], packed w_lm [V, d] -> (argmax int32 [M], max fp32
    [M], logits fp32 [M, V] or None).  logits_out: a preallocated [M, V] fp32 tensor for
    the logits (implies want_logits)."""
    if not isinstance(w_lm, PackedWeight):
        raise TypeError("w_lm must be packed with pack_weight()")
    M, d = hidden.shape
    V = w_lm.N
    if w_lm.K != d or w_lm.dtype != hidden.dtype:
        raise ValueError("hidden and w_lm disagree in width or dtype")
    dev = hidden.device
    if out is None:
        am = torch.empty(M, dtype=torch.int32, device=dev)
        mx = torch.empty(M, dtype=torch.float32, device=dev) if want_max else None
    else:
        am, mx = out
    _typed(am, torch.int32, M, "argmax")
    _typed(mx, torch.float32, M, "max_logit")
    if logits_out is not None:
        if logits_out.shape != (M, V) or logits_out.dtype != torch.float32:
            raise ValueError("logits_out must be a [M, V] fp32 tensor")
        lg = logits_out
    else:
        lg = torch.empty((M, V), dtype=torch.float32, device=dev) if want_logits else None
    need = lm_head_workspace(M, V)
    if ws is None or ws.numel() < need:
        ws = torch.zeros(max(need, 1), dtype=torch.uint8, device=dev)   # zero before first use
    _dev(hidden, w_lm.data, am, mx, lg, ws)
    _check(lib().hdf_lm_head_argmax(_ptr(hidden), _ptr(w_lm), M, d, V, _dt(hidden), _ptr(am),
                                    _ptr(mx), _ptr(lg), _ptr(ws), ws.numel(), _stream(stream)))
    return am, mx, lg


def lm_head_argmax_keys(hidden: torch.Tensor, w_lm: PackedWeight, ws: torch.Tensor,
                        stream=None):
    """hdf_lm_head_argmax_keys: the LM-head GEMM alone; the packed argmax keys of the M
    rows stay in `ws` (a zeroed workspace of lm_head_workspace(M, V) bytes) for
    accept_keys."""
    if not isinstance(w_lm, PackedWeight):
        raise TypeError("w_lm must be packed with pack_weight()")
    M, d = hidden.shape
    V = w_lm.N
    if w_lm.K != d or w_lm.dtype != hidden.dtype:
        raise ValueError("hidden and w_lm disagree in width or dtype")
    if ws is None or ws.numel() < lm_head_workspace(M, V):
        raise ValueError("lm_head_argmax_keys needs a workspace of lm_head_workspace(M, V) bytes")
    _dev(hidden, w_lm.data, ws)
    _check(lib().hdf_lm_head_argmax_keys(_ptr(hidden), _ptr(w_lm), M, d, V, _dt(hidden),
                                         _ptr(ws), ws.numel(), _stream(stream)))


def accept_keys(ws: torch.Tensor, target: torch.Tensor, B: int, *, argmax: torch.Tensor,
                max_logit: Optional[torch.Tensor] = None, commits: bool = True, out=None,
                stream=None):
    """hdf_accept_keys: argmax (and max_logit) of the n_seq*B block rows from the keys in
    `ws`, the keys cleared, then the acceptance of the drafts (slots 1..B-1) against
    target [n_seq, B] int32.  Returns (accept_len, next_anchor, commit_offsets,
    commit_tokens); out: optional preallocated tuple of those."""
    n_seq = target.shape[0]
    if target.shape[1] != B:
        raise ValueError("target must be [n_seq, B] (K + 1 = B tokens per sequence)")
    M = n_seq * B
    _typed(argmax, torch.int32, M, "argmax")
    _typed(max_logit, torch.float32, M, "max_logit")
    _typed(target, torch.int32, M, "target")
    dev = target.device
    if out is not None:
        acc, anc, offs, toks = out
    else:
        acc = torch.empty(n_seq, dtype=torch.int32, device=dev)
        anc = torch.empty(n_seq, dtype=torch.int32, device=dev)
        offs = torch.empty(n_seq + 1, dtype=torch.int32, device=dev) if commits else None
        toks = torch.empty(max(1, n_seq * B), dtype=torch.int32, device=dev) if commits else None
    for t, k, what in ((acc, n_seq, "accept_len"), (anc, n_seq, "next_anchor"),
                       (offs, n_seq + 1, "commit_offsets"), (toks, M, "commit_tokens")):
        _typed(t, torch.int32, k, what)
    _dev(ws, target, argmax, max_logit, acc, anc, offs, toks)
    _check(lib().hdf_accept_keys(_ptr(ws), n_seq, B, _ptr(argmax), _ptr(max_logit), _ptr(target),
                                 _ptr(acc), _ptr(anc), _ptr(offs), _ptr(toks), _stream(stream)))
    return acc, anc, offs, toks


# ----------------------------------------------------------------------------- drafter

def rope_table(n_pos: int, head_dim: int, theta: float) -> torch.Tensor:
    """Host-computed (fp64 -> fp32) cos/sin table [n_pos, head_dim/2, 2] on the CPU."""
    t = torch.empty((n_pos, head_dim // 2, 2), dtype=torch.float32)
    _check(lib().hdf_rope_table(ctypes.c_void_p(t.data_ptr()), n_pos, head_dim, theta))
    return t


class DrafterHandle:
    """Keeps the device weights (projections packed once, here) and the ctypes
    hdf_drafter struct alive together."""

    def __init__(self, weights: dict, *, n_layers: int, d: int, n_heads: int, head_dim: int,
                 d_ff: int, vocab: int, eps: float = 1e-6, rope_theta: float = 10000.0,
                 rope_max_pos: int = 0, device="cuda"):
        self.w = weights
        self.L = n_layers
        dt = weights["tok_emb"].dtype
        self.packed = {k: [pack_weight(x).data for x in weights[k]]
                       for k in ("w_qkv", "w_o", "w_gate_up", "w_down")}
        self.w_lm = pack_weight(weights["w_lm"]) if weights.get("w_lm") is not None else None
        self.torch_dtype = dt
        keep = []

        def arr(ts):
            a = (ctypes.c_void_p * n_layers)(*[None if t is None else t.data_ptr() for t in ts])
            keep.append(a)
            return ctypes.cast(a, ctypes.POINTER(ctypes.c_void_p))

        self.rope = None
        if rope_theta and rope_theta > 0:
            self.rope = rope_table(rope_max_pos, head_dim, rope_theta).to(device)
        self.s = Drafter(
            n_layers, d, n_heads, head_dim, d_ff, vocab, _dt(weights["tok_emb"]), eps,
            weights["tok_emb"].data_ptr(),
            None if weights.get("ctx_norm") is None else weights["ctx_norm"].data_ptr(),
            arr(weights.get("attn_norm", [None] * n_layers)), arr(self.packed["w_qkv"]),
            arr(self.packed["w_o"]), arr(weights.get("mlp_norm", [None] * n_layers)),
            arr(self.packed["w_gate_up"]), arr(self.packed["w_down"]),
            None if weights.get("final_norm") is None else weights["final_norm"].data_ptr(),
            None if self.rope is None else self.rope.data_ptr(),
            rope_max_pos if self.rope is not None else 0)
        self._keep = keep
        self.d, self.nh, self.hd, self.F, self.V = d, n_heads, head_dim, d_ff, vocab
        self.eps = eps

    def kv_cache_bytes(self, kv_cap: int) -> int:
        return int(lib().hdf_kv_cache_bytes(ctypes.byref(self.s), kv_cap))

    def workspace_bytes(self, n_seq: int, B: int, n_new: int, max_ctx: int) -> int:
        return int(lib().hdf_draft_block_workspace(ctypes.byref(self.s), n_seq, B, n_new, max_ctx))

    def alloc_kv(self, kv_cap: int, device="cuda"):
        """KV cache tensors in the library's layout: keys and values each
        [L][nh][cap/64][64*hd], 64-position tiles in matrix-core operand order."""
        if kv_cap % 64:
            raise ValueError("kv_cap must be a multiple of 64")
        shape = (self.L, self.nh, kv_cap // 64, 64 * self.hd)
        return (torch.zeros(shape, dtype=self.torch_dtype, device=device),
                torch.zeros(shape, dtype=self.torch_dtype, device=device))

    def draft_block(self, *, ctx_len: torch.Tensor, max_ctx: int, y_new: torch.Tensor,
                    new_offsets: torch.Tensor, kv_k: torch.Tensor, kv_vt: torch.Tensor,
                    tokens: torch.Tensor, kv_offsets: Optional[torch.Tensor] = None,
                    page_table: Optional[torch.Tensor] = None,
                    new_counts: Optional[torch.Tensor] = None,
                    hidden: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                    stream=None):
        """hdf_draft_block over a contiguous cache (kv_offsets [n_seq+1]) or
        hdf_draft_block_paged over a paged one (page_table [n_seq][max_pages], optionally
        with device new_counts [n_seq]: only the first new_counts[s] rows of each
        sequence's rows in y_new are new)."""
        if (kv_offsets is None) == (page_table is None):
            raise ValueError("give exactly one of kv_offsets and page_table")
        if new_counts is not None and page_table is None:
            raise ValueError("new_counts goes with a paged cache")
        n_seq, B = tokens.shape
        n_new = y_new.shape[0]
        dev = tokens.device
        if hidden is None:
            hidden = torch.empty((n_seq * B, self.d), dtype=self.torch_dtype, device=dev)
        need = self.workspace_bytes(n_seq, B, n_new, max_ctx)
        if ws is None or ws.numel() < need:
            ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
        if page_table is not None:
            if page_table.dtype != torch.int32 or page_table.dim() != 2 or \
                    page_table.shape[0] != n_seq or not page_table.is_contiguous():
                raise ValueError("page_table must be a contiguous int32 [n_seq][max_pages] tensor")
            if new_counts is not None and (new_counts.dtype != torch.int32 or
                                           new_counts.numel() != n_seq):
                raise ValueError("new_counts must be an int32 [n_seq] tensor")
            _dev(ctx_len, y_new, new_offsets, new_counts, page_table, kv_k, kv_vt, tokens, hidden,
                 ws)
            _check(lib().hdf_draft_block_paged(
                ctypes.byref(self.s), n_seq, B, _ptr(ctx_len), max_ctx, _ptr(y_new),
                _ptr(new_offsets), _ptr(new_counts), n_new, _ptr(page_table), page_table.shape[1],
                _ptr(kv_k),
                _ptr(kv_vt), kv_k.shape[2], _ptr(tokens), _ptr(hidden), _ptr(ws), ws.numel(),
                _stream(stream)))
            return hidden
        kv_cap = kv_k.shape[2] * 64
        _dev(ctx_len, y_new, new_offsets, kv_offsets, kv_k, kv_vt, tokens, hidden, ws)
        _check(lib().hdf_draft_block(ctypes.byref(self.s), n_seq, B, _ptr(ctx_len), max_ctx,
                                     _ptr(y_new), _ptr(new_offsets), n_new, _ptr(kv_offsets),
                                     _ptr(kv_k), _ptr(kv_vt), kv_cap, _ptr(tokens), _ptr(hidden),
                                     _ptr(ws), ws.numel(), _stream(stream)))
        return hidden


def _kv_dims(kv_k: torch.Tensor):
    """(n_layers, n_heads, head_dim, kv_cap) of a cache tensor [L][nh][cap/64][64*hd]."""
    L, nh, tiles, tsz = kv_k.shape
    return L, nh, tsz // 64, tiles * 64


def kv_write_rows(kv_k: torch.Tensor, kv_vt: torch.Tensor, layer: int, k_rows: torch.Tensor,
                  v_rows: torch.Tensor, *, row0: int = 0, rows: Optional[torch.Tensor] = None,
                  stream=None):
    """hdf_kv_write_rows: row i of k_rows / v_rows [n, nh*hd] into cache row rows[i] (int32
    device tensor) or row0 + i of one layer.  Either k_rows or v_rows may be None."""
    L, nh, hd, cap = _kv_dims(kv_k)
    src = k_rows if k_rows is not None else v_rows
    n = src.shape[0]
    if not 0 <= layer < L:
        raise ValueError(f"layer {layer} outside [0, {L})")
    if rows is not None and (rows.dtype != torch.int32 or rows.numel() != n):
        raise ValueError("rows must be an int32 tensor with one entry per row")
    _dev(kv_k, kv_vt, k_rows, v_rows, rows)
    _check(lib().hdf_kv_write_rows(_ptr(k_rows), _ptr(v_rows), n, _ptr(rows), row0, layer, nh, hd,
                                   _dt(kv_k), _ptr(kv_k) if k_rows is not None else None,
                                   _ptr(kv_vt) if v_rows is not None else None, cap,
                                   _stream(stream)))


def kv_read_rows(kv_k: torch.Tensor, kv_vt: torch.Tensor, layer: int, n: int, *, row0: int = 0,
                 rows: Optional[torch.Tensor] = None, stream=None):
    """hdf_kv_read_rows: cache rows rows[i] (or row0 + i), i < n, of one layer as row-major
    (keys [n, nh*hd], values [n, nh*hd])."""
    L, nh, hd, cap = _kv_dims(kv_k)
    if not 0 <= layer < L:
        raise ValueError(f"layer {layer} outside [0, {L})")
    if rows is not None and (rows.dtype != torch.int32 or rows.numel() != n):
        raise ValueError("rows must be an int32 tensor with one entry per row")
    k = torch.empty((n, nh * hd), dtype=kv_k.dtype, device=kv_k.device)
    v = torch.empty_like(k)
    _dev(kv_k, kv_vt, rows)
    _check(lib().hdf_kv_read_rows(_ptr(kv_k), _ptr(kv_vt), cap, layer, nh, hd, _dt(kv_k),
                                  _ptr(rows), row0, n, _ptr(k), _ptr(v), _stream(stream)))
    return k, v


def write_kv_rows(kv_k: torch.Tensor, kv_vt: torch.Tensor, layer: int, row0: int,
                  k_rows: torch.Tensor, v_rows: torch.Tensor):
    """Keys/values of consecutive positions [n, nh*hd] into cache rows row0..row0+n-1 of
    one layer (hdf_kv_write_rows)."""
    if k_rows.shape[0] == 0:
        return
    kv_write_rows(kv_k, kv_vt, layer, k_rows.contiguous(), v_rows.contiguous(), row0=row0)


def read_kv_rows(kv_k: torch.Tensor, kv_vt: torch.Tensor, layer: int, row0: int, n: int):
    """Keys/values of cache rows row0..row0+n-1 of one layer as [n, nh*hd] tensors."""
    return kv_read_rows(kv_k, kv_vt, layer, n, row0=row0)


def paged_rows(pages: Sequence[int], n: int, device) -> torch.Tensor:
    """Cache rows of positions 0..n-1 of a sequence stored in `pages` (position p is row
    p % 64 of page pages[p // 64]), as an int32 device tensor."""
    pg = torch.as_tensor(list(pages)[:(n + 63) // 64], dtype=torch.int64)
    p = torch.arange(n, dtype=torch.int64)
    return (pg[p // 64] * 64 + p % 64).to(torch.int32).to(device)


def write_kv_rows_paged(kv_k: torch.Tensor, kv_vt: torch.Tensor, layer: int, pages: Sequence[int],
                        k_rows: torch.Tensor, v_rows: torch.Tensor):
    """Keys/values of positions 0..n-1 of one sequence into its pages (position i goes to
    row i%64 of page pages[i//64]) of one layer (hdf_kv_write_rows with a row list)."""
    n = k_rows.shape[0]
    if n == 0:
        return
    kv_write_rows(kv_k, kv_vt, layer, k_rows.contiguous(), v_rows.contiguous(),
                  rows=paged_rows(pages, n, kv_k.device))


def read_kv_rows_paged(kv_k: torch.Tensor, kv_vt: torch.Tensor, layer: int, pages: Sequence[int],
                       n: int):
    """Keys/values of positions 0..n-1 of one sequence, stored in `pages`, as [n, nh*hd]."""
    if n == 0:
        d = kv_k.shape[1] * (kv_k.shape[3] // 64)
        e = torch.empty((0, d), dtype=kv_k.dtype, device=kv_k.device)
        return e, e.clone()
    return kv_read_rows(kv_k, kv_vt, layer, n, rows=paged_rows(pages, n, kv_k.device))


def kv_slot_offsets(ctx_lens: Sequence[int]) -> list:
    """Cache slot offsets: each sequence's slot starts at a multiple of 64 rows and holds
    its context length rounded up to 64."""
    offs = [0]
    for t in ctx_lens:
        offs.append(offs[-1] + ((int(t) + 63) // 64) * 64)
    return offs
