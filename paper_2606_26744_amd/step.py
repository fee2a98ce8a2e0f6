"""One HyperDFlash drafter step on the device, through the C ABI.

The four stages run in order on the current HIP stream, every one of them in
libhdf's kernels:
    hdf_hc_reduce        H rows of the newest context positions -> Y
    hdf_draft_block      Y -> KV cache rows; block [anchor, mask...] -> hidden
    hdf_lm_head_argmax   hidden -> argmax per slot
    hdf_accept           drafts (slots 1..B-1) vs the target's tokens
With targets and no logits asked for, the last two are hdf_lm_head_argmax_keys (the
LM-head GEMM) and hdf_accept_keys (the argmax finalisation and the acceptance in one
launch), with the same outputs.
This module only allocates device buffers (once) and passes pointers.
"""
from __future__ import annotations

from typing import Optional

import torch

from . import hdf


class SampledStepBuffers:
    """Extra device buffers of a temperature-sampled step: fp32 logits [n_seq*B][V],
    drawn tokens, log-sum-exps and the two sampling workspaces."""

    def __init__(self, handle: hdf.DrafterHandle, n_seq: int, B: int, device="cuda"):
        M, V = n_seq * B, handle.V
        self.logits = torch.empty((M, V), dtype=torch.float32, device=device)
        self.tokens = torch.empty(M, dtype=torch.int32, device=device)
        self.lse = torch.empty(M, dtype=torch.float32, device=device)
        self.sample_ws = torch.empty(max(int(hdf.lib().hdf_sample_workspace(M, V)), 1),
                                     dtype=torch.uint8, device=device)
        self.accept_ws = torch.empty(
            max(int(hdf.lib().hdf_accept_sample_workspace(n_seq, B - 1, V)), 1),
            dtype=torch.uint8, device=device)


class StepBuffers:
    """Device buffers of one step, reused across steps (nothing is allocated per call)."""

    def __init__(self, handle: hdf.DrafterHandle, n_seq: int, B: int, n_new: int, max_ctx: int,
                 m: int, device="cuda"):
        dt = handle.torch_dtype
        d = handle.d
        self.Y = torch.empty((n_new, d), dtype=dt, device=device)
        self.hidden = torch.empty((n_seq * B, d), dtype=dt, device=device)
        self.ws = torch.empty(max(handle.workspace_bytes(n_seq, B, n_new, max_ctx), 1),
                              dtype=torch.uint8, device=device)
        self.lm_ws = torch.zeros(max(hdf.lm_head_workspace(n_seq * B, handle.V), 1),
                                 dtype=torch.uint8, device=device)   # zero before first use
        self.argmax = torch.empty(n_seq * B, dtype=torch.int32, device=device)
        self.max_logit = torch.empty(n_seq * B, dtype=torch.float32, device=device)


def drafter_step(handle: hdf.DrafterHandle, bufs: StepBuffers, *, H_new: torch.Tensor,
                 W_g: torch.Tensor, b_g: torch.Tensor, new_offsets: torch.Tensor,
                 ctx_len: torch.Tensor, max_ctx: int, kv_offsets: torch.Tensor,
                 kv_k: torch.Tensor, kv_vt: torch.Tensor, tokens: torch.Tensor,
                 targets: Optional[torch.Tensor], reduce_kw: Optional[dict] = None,
                 stream=None, logits: bool = False, marks: Optional[list] = None):
    """Runs reduce -> draft block -> LM head argmax -> accept.  Returns a dict of device
    tensors (Y, hidden, argmax, max_logit, and accept outputs when targets are given).
    marks: optional list of five timing events (entries may be None) recorded on the stream
    around the stages."""
    kw = dict(reduce_kw or {})
    kw.setdefault("eps", handle.eps)

    def mark(i):
        if marks is not None and marks[i] is not None:
            marks[i].record(stream if stream is not None else torch.cuda.current_stream())

    mark(0)
    hdf.hc_reduce(H_new, W_g, b_g, Y=bufs.Y, stream=stream, **kw)
    mark(1)
    handle.draft_block(ctx_len=ctx_len, max_ctx=max_ctx, y_new=bufs.Y, new_offsets=new_offsets,
                       kv_offsets=kv_offsets, kv_k=kv_k, kv_vt=kv_vt, tokens=tokens,
                       hidden=bufs.hidden, ws=bufs.ws, stream=stream)
    mark(2)
    if targets is not None and not logits:
        n_seq, B = tokens.shape
        hdf.lm_head_argmax_keys(bufs.hidden, handle.w_lm, bufs.lm_ws, stream=stream)
        mark(3)
        acc, anc, offs, toks = hdf.accept_keys(bufs.lm_ws, targets, B, argmax=bufs.argmax,
                                               max_logit=bufs.max_logit, stream=stream)
        mark(4)
        return {"Y": bufs.Y, "hidden": bufs.hidden, "argmax": bufs.argmax,
                "max_logit": bufs.max_logit, "logits": None, "accept_len": acc,
                "next_anchor": anc, "commit_offsets": offs, "commit_tokens": toks}
    am, mx, lg = hdf.lm_head_argmax(bufs.hidden, handle.w_lm, want_logits=logits,
                                    ws=bufs.lm_ws, out=(bufs.argmax, bufs.max_logit),
                                    stream=stream)
    mark(3)
    out = {"Y": bufs.Y, "hidden": bufs.hidden, "argmax": am, "max_logit": mx, "logits": lg}
    if targets is not None:
        n_seq, B = tokens.shape
        acc, anc, offs, toks = hdf.accept(am[1:], targets, K=B - 1, draft_stride=B,
                                          stream=stream)
        out.update(accept_len=acc, next_anchor=anc, commit_offsets=offs, commit_tokens=toks)
    mark(4)
    return out


def drafter_step_sampled(handle: hdf.DrafterHandle, bufs: StepBuffers, sbufs: SampledStepBuffers,
                         *, H_new: torch.Tensor, W_g: torch.Tensor, b_g: torch.Tensor,
                         new_offsets: torch.Tensor, ctx_len: torch.Tensor, max_ctx: int,
                         kv_offsets: torch.Tensor, kv_k: torch.Tensor, kv_vt: torch.Tensor,
                         tokens: torch.Tensor, target_logits: torch.Tensor,
                         temperature: float = 1.0, seed: int = 0, round_id: int = 0,
                         reduce_kw: Optional[dict] = None, stream=None):
    """The step at temperature T: reduce -> draft block -> LM head (logits kept) ->
    draws of every slot from softmax(logits / T) -> speculative-sampling verification
    against target_logits [n_seq, B, V] (row i: the target's logits for draft slot i+1;
    the last row for the token after the drafts).  round_id selects the Philox stream,
    so that every round draws fresh numbers."""
    kw = dict(reduce_kw or {})
    kw.setdefault("eps", handle.eps)
    hdf.hc_reduce(H_new, W_g, b_g, Y=bufs.Y, stream=stream, **kw)
    handle.draft_block(ctx_len=ctx_len, max_ctx=max_ctx, y_new=bufs.Y, new_offsets=new_offsets,
                       kv_offsets=kv_offsets, kv_k=kv_k, kv_vt=kv_vt, tokens=tokens,
                       hidden=bufs.hidden, ws=bufs.ws, stream=stream)
    hdf.lm_head_argmax(bufs.hidden, handle.w_lm, ws=bufs.lm_ws, out=(bufs.argmax, bufs.max_logit),
                       logits_out=sbufs.logits, stream=stream)
    hdf.sample_tokens(sbufs.logits, temperature=temperature, seed=seed, stream_id=2 * round_id,
                      ws=sbufs.sample_ws, out=(sbufs.tokens, sbufs.lse), stream=stream)
    n_seq, B = tokens.shape
    V = handle.V
    acc, anc, offs, toks = hdf.accept_sample(
        sbufs.tokens[1:], sbufs.logits[1:], sbufs.lse[1:], target_logits, K=B - 1,
        draft_stride=B, ld=V, temperature=temperature, seed=seed, stream_id=2 * round_id + 1,
        ws=sbufs.accept_ws, stream=stream)
    return {"hidden": bufs.hidden, "logits": sbufs.logits, "tokens": sbufs.tokens,
            "accept_len": acc, "next_anchor": anc, "commit_offsets": offs, "commit_tokens": toks}
