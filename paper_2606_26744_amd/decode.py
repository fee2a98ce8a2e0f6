"""Chained drafting rounds over a persistent paged KV cache.

Every round runs the four stages in libhdf's kernels, on the current stream:
    hdf_hc_reduce          target states of the newly committed positions -> Y
    hdf_draft_block_paged  Y -> cache pages; anchor + mask block -> hidden
    hdf_lm_head_argmax     hidden -> greedy drafts
    hdf_accept             drafts vs the target's tokens -> n_s, next anchor, commits
Between rounds the n_s + 1 positions a sequence committed (its accepted drafts and
the target's token after them) become its next context rows: their target states are
reduced and projected into the cache by the next round, the context grows by n_s + 1
and the target's token at the first rejected slot is the next anchor (Sec. 1; tau
= n_s + 1, Sec. 3.4).  The cache is a pool of 64-row pages, so a sequence grows by
taking any free page.  This module keeps only the host bookkeeping (page allocator,
page table, lengths), one small host-to-device copy and one device-to-host read of
the accepted lengths per round; it computes nothing itself.
"""
from __future__ import annotations

from typing import Callable, List, Optional, Sequence

import numpy as np
import torch

from . import hdf


class PagePool:
    """Free list of the cache's 64-row pages (handed out in `order`, default 0, 1, ...)."""

    def __init__(self, n_pages: int, order: Optional[Sequence[int]] = None):
        self.n_pages = n_pages
        order = list(range(n_pages)) if order is None else [int(p) for p in order]
        if sorted(order) != list(range(n_pages)):
            raise ValueError("order must be a permutation of the pages")
        self._free = order[::-1]

    def take(self) -> int:
        if not self._free:
            raise MemoryError("KV page pool exhausted")
        return self._free.pop()

    def release(self, pages: Sequence[int]):
        self._free.extend(reversed(list(pages)))

    @property
    def free(self) -> int:
        return len(self._free)


class PagedDecoder:
    """Decoding state of n_seq sequences: a paged KV cache, each sequence's pages and
    context length, the block tokens (anchor + masks) and the step buffers."""

    def __init__(self, handle: hdf.DrafterHandle, n_seq: int, B: int, max_ctx: int,
                 n_pages: int, max_new_rows: int, device="cuda",
                 page_order: Optional[Sequence[int]] = None):
        if handle.w_lm is None:
            raise ValueError("the drafter handle carries no LM head")
        self.h, self.n_seq, self.B, self.max_ctx = handle, n_seq, B, max_ctx
        self.max_pages = (max_ctx + 63) // 64
        self.pool = PagePool(n_pages, page_order)
        self.pages: List[List[int]] = [[] for _ in range(n_seq)]
        self.ctx = np.zeros(n_seq, dtype=np.int64)          # T_s on the host
        self.kv_k, self.kv_vt = handle.alloc_kv(n_pages * 64, device=device)
        dt, d = handle.torch_dtype, handle.d
        self.max_new_rows = max_new_rows
        self.Y = torch.empty((max(max_new_rows, 1), d), dtype=dt, device=device)
        self.hidden = torch.empty((n_seq * B, d), dtype=dt, device=device)
        self.ws = torch.empty(max(handle.workspace_bytes(n_seq, B, max_new_rows, max_ctx), 1),
                              dtype=torch.uint8, device=device)
        self.lm_ws = torch.zeros(max(hdf.lm_head_workspace(n_seq * B, handle.V), 1),
                                 dtype=torch.uint8, device=device)
        self.argmax = torch.empty(n_seq * B, dtype=torch.int32, device=device)
        self.max_logit = torch.empty(n_seq * B, dtype=torch.float32, device=device)
        self.tokens = torch.full((n_seq, B), handle.V - 1, dtype=torch.int32, device=device)
        # One staging copy per round: ctx_len [n_seq] | new_offsets [n_seq+1] | page table.
        n_meta = n_seq + (n_seq + 1) + n_seq * self.max_pages
        self._meta_host = torch.zeros(n_meta, dtype=torch.int32).pin_memory()
        self._meta = torch.zeros(n_meta, dtype=torch.int32, device=device)
        self._pt_host = self._meta_host[2 * n_seq + 1:].view(n_seq, self.max_pages).numpy()
        self._pt_host[:] = -1
        self.ctx_len = self._meta[:n_seq]
        self.new_offsets = self._meta[n_seq:2 * n_seq + 1]
        self.page_table = self._meta[2 * n_seq + 1:].view(n_seq, self.max_pages)
        self._copied = torch.cuda.Event()   # the last staging copy has been read

    def set_anchors(self, anchors: torch.Tensor):
        self.tokens[:, 0] = anchors

    def preload(self, counts: Sequence[int]):
        """Takes pages for counts[s] more context positions of every sequence and counts
        them as cached: for rows the caller writes into the pages itself (a prompt whose
        keys and values were computed elsewhere)."""
        self._grow(np.asarray(counts, dtype=np.int64))

    def _grow(self, new_counts: np.ndarray):
        self._copied.synchronize()          # the staging buffer is free again
        for s in range(self.n_seq):
            need = (int(self.ctx[s]) + int(new_counts[s]) + 63) // 64
            if need > self.max_pages:
                raise ValueError(f"sequence {s} outgrows max_ctx={self.max_ctx}")
            while len(self.pages[s]) < need:
                p = self.pool.take()
                self._pt_host[s, len(self.pages[s])] = p
                self.pages[s].append(p)
        self.ctx += new_counts
        m = self._meta_host.numpy()
        m[:self.n_seq] = self.ctx
        m[self.n_seq] = 0
        m[self.n_seq + 1:2 * self.n_seq + 1] = np.cumsum(new_counts)
        self._meta.copy_(self._meta_host, non_blocking=True)
        self._copied.record()

    def round(self, H_new: torch.Tensor, new_counts: Sequence[int], W_g: torch.Tensor,
              b_g: torch.Tensor, targets: Callable[[torch.Tensor], torch.Tensor],
              reduce_kw: Optional[dict] = None):
        """One round.  H_new [n_new, m, d]: target states of the new_counts[s] newest
        positions of every sequence, packed by sequence.  `targets(drafts)` stands in
        for the target model's verification: drafts [n_seq, B-1] int32 (device) ->
        target tokens [n_seq, B] int32 (device).  Returns a dict of device tensors."""
        new_counts = np.asarray(new_counts, dtype=np.int64)
        n_new = int(new_counts.sum())
        if n_new > self.max_new_rows or H_new.shape[0] != n_new:
            raise ValueError("H_new rows do not match new_counts / max_new_rows")
        self._grow(new_counts)
        kw = dict(reduce_kw or {})
        kw.setdefault("eps", self.h.eps)
        Y = self.Y[:n_new]
        hdf.hc_reduce(H_new, W_g, b_g, Y=Y, **kw)
        self.h.draft_block(ctx_len=self.ctx_len, max_ctx=self.max_ctx, y_new=Y,
                           new_offsets=self.new_offsets, page_table=self.page_table,
                           kv_k=self.kv_k, kv_vt=self.kv_vt, tokens=self.tokens,
                           hidden=self.hidden, ws=self.ws)
        am, mx, _ = hdf.lm_head_argmax(self.hidden, self.h.w_lm, ws=self.lm_ws,
                                       out=(self.argmax, self.max_logit))
        drafts = am.view(self.n_seq, self.B)[:, 1:]
        tg = targets(drafts)
        acc, anc, offs, toks = hdf.accept(am[1:], tg, K=self.B - 1, draft_stride=self.B)
        out = {"Y": Y, "hidden": self.hidden, "argmax": am, "drafts": drafts, "targets": tg,
               "accept_len": acc, "next_anchor": anc, "commit_offsets": offs,
               "commit_tokens": toks, "tokens": self.tokens.clone()}
        self.tokens[:, 0] = anc
        return out

    def next_counts(self, accept_len: torch.Tensor) -> np.ndarray:
        """n_s + 1 committed positions per sequence: the next round's new rows (reads
        the accepted lengths back to the host)."""
        return accept_len.cpu().numpy().astype(np.int64) + 1
