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
page table, lengths) and computes nothing itself.

Two ways to chain rounds:
  round()          the host reads the accepted lengths back after every round and sizes
                   the next one exactly (one small copy each way per round);
  chained_round()  the lengths stay on the device: hdf_advance_context turns the
                   accepted lengths into the next round's context lengths and row counts,
                   and the next hdf_draft_block_paged takes them through new_counts with
                   the launch sized for B rows per sequence.  The host only keeps an upper
                   bound on every length (+B a round, tightened from lengths it reads
                   back a round or two late without waiting) to take pages ahead of the
                   growth, so it never waits for a round to finish.
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


def pages_for(lengths, max_ctx: int) -> np.ndarray:
    """Pages of 64 rows that context lengths `lengths` occupy.  Raises ValueError when a
    length exceeds max_ctx: the drafter call is made with max_ctx, which also bounds the
    RoPE table (max_ctx + B rows), so a longer context would read past that table even
    where its last page still has room."""
    lengths = np.asarray(lengths, dtype=np.int64)
    over = np.nonzero(lengths > max_ctx)[0]
    if over.size:
        s = int(over[0])
        raise ValueError(f"sequence {s} outgrows max_ctx={max_ctx} (length {int(lengths[s])})")
    return (lengths + 63) // 64


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
        # Chained rounds (chained_round): device-owned lengths and counts, fixed row
        # offsets s*B, double-buffered page-table staging, lagged length read-backs.
        self.chain_ctx = torch.zeros(n_seq, dtype=torch.int32, device=device)
        self.chain_counts = torch.zeros(n_seq, dtype=torch.int32, device=device)
        self.chain_offsets = (torch.arange(n_seq + 1, dtype=torch.int32) * B).to(device)
        self._pt_stage = [torch.zeros(n_seq * self.max_pages, dtype=torch.int32).pin_memory()
                          for _ in range(2)]
        self._pt_events = [None, None]
        self._pt_slot = 0
        self._rb_host = [torch.zeros(n_seq, dtype=torch.int32).pin_memory() for _ in range(3)]
        self._rb_pending = []               # (event, slot, round index) of lagged read-backs
        self._rb_slot = 0
        self._rounds = 0                    # chained rounds launched
        self._ctx_hi = None                 # host upper bound on every device length
        self.acc = torch.empty(n_seq, dtype=torch.int32, device=device)
        self.anc = torch.empty(n_seq, dtype=torch.int32, device=device)
        self.offs = torch.empty(n_seq + 1, dtype=torch.int32, device=device)
        self.toks = torch.empty(n_seq * B, dtype=torch.int32, device=device)

    def set_anchors(self, anchors: torch.Tensor):
        self.tokens[:, 0] = anchors

    def preload(self, counts: Sequence[int]):
        """Takes pages for counts[s] more context positions of every sequence and counts
        them as cached: for rows the caller writes into the pages itself (a prompt whose
        keys and values were computed elsewhere)."""
        self._grow(np.asarray(counts, dtype=np.int64))

    def _grow(self, new_counts: np.ndarray):
        self._copied.synchronize()          # the staging buffer is free again
        need_all = pages_for(self.ctx + new_counts, self.max_ctx)
        for s in range(self.n_seq):
            need = int(need_all[s])
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

    # ------------------------------------------------------------------ chained rounds
    def start_chain(self, counts: Sequence[int]):
        """Switches to chained rounds: the first chained_round projects the counts[s] (<= B)
        newest positions of every sequence (rows s*B .. s*B + counts[s] - 1 of its
        H_block).  Takes their pages and writes the device lengths and counts once."""
        counts = np.asarray(counts, dtype=np.int64)
        if counts.shape != (self.n_seq,) or (counts < 0).any() or (counts > self.B).any():
            raise ValueError("start_chain: counts must be n_seq values in [0, B]")
        self._grow(counts)
        self._copied.synchronize()
        self.chain_ctx.copy_(torch.as_tensor(self.ctx, dtype=torch.int32))
        self.chain_counts.copy_(torch.as_tensor(counts, dtype=torch.int32))
        self._ctx_hi = self.ctx.copy()
        self._rb_pending.clear()
        self._rounds = 0

    def _tighten(self, wait: bool = False):
        """Folds read-backs that have landed into the upper bound: the device length
        after round j is exact, and every later round adds at most B."""
        while self._rb_pending:
            ev, slot, j = self._rb_pending[0]
            if not wait and not ev.query():
                break
            ev.synchronize()
            self._rb_pending.pop(0)
            exact = self._rb_host[slot].numpy().astype(np.int64)
            self.ctx = exact.copy()
            self._ctx_hi = np.minimum(self._ctx_hi, exact + self.B * (self._rounds - 1 - j))

    def _reserve(self):
        """Pages for every position below the upper bound; the page table goes to the
        device through a staging buffer no pending copy still reads."""
        if (self._ctx_hi > self.max_ctx).any():
            self._tighten(wait=True)
        need = pages_for(self._ctx_hi, self.max_ctx)
        changed = False
        for s in range(self.n_seq):
            while len(self.pages[s]) < need[s]:
                p = self.pool.take()
                self._pt_host[s, len(self.pages[s])] = p
                self.pages[s].append(p)
                changed = True
        if changed:
            k = self._pt_slot
            if self._pt_events[k] is not None:
                self._pt_events[k].synchronize()
            self._pt_stage[k].numpy()[:] = self._pt_host.reshape(-1)
            self.page_table.view(-1).copy_(self._pt_stage[k], non_blocking=True)
            ev = torch.cuda.Event()
            ev.record()
            self._pt_events[k] = ev
            self._pt_slot = 1 - k

    def chained_round(self, H_block: torch.Tensor, W_g: torch.Tensor, b_g: torch.Tensor,
                      targets: Callable[[torch.Tensor], torch.Tensor],
                      reduce_kw: Optional[dict] = None, record: bool = False):
        """One round without any host wait.  H_block [n_seq*B, m, d]: the target's states
        at the B slots of every sequence's previous block (row s*B + j); the first
        new_counts[s] of them are the positions sequence s committed and are projected
        into the cache, the others are ignored.  Returns a dict of device tensors
        (accept_len, next_anchor, commits, hidden, argmax: overwritten by the next round;
        with record=True also copies of the block tokens, lengths and counts the round
        started from)."""
        if self._ctx_hi is None:
            raise RuntimeError("start_chain() first")
        n, B = self.n_seq, self.B
        if H_block.shape[0] != n * B or n * B > self.max_new_rows:
            raise ValueError("H_block must hold n_seq*B rows (and max_new_rows >= n_seq*B)")
        self._tighten()
        self._reserve()
        kw = dict(reduce_kw or {})
        kw.setdefault("eps", self.h.eps)
        Y = self.Y[:n * B]
        hdf.hc_reduce(H_block, W_g, b_g, Y=Y, **kw)
        self.h.draft_block(ctx_len=self.chain_ctx, max_ctx=self.max_ctx, y_new=Y,
                           new_offsets=self.chain_offsets, new_counts=self.chain_counts,
                           page_table=self.page_table, kv_k=self.kv_k, kv_vt=self.kv_vt,
                           tokens=self.tokens, hidden=self.hidden, ws=self.ws)
        am, mx, _ = hdf.lm_head_argmax(self.hidden, self.h.w_lm, ws=self.lm_ws,
                                       out=(self.argmax, self.max_logit))
        drafts = am.view(n, B)[:, 1:]
        tg = targets(drafts)
        out = {"Y": Y, "hidden": self.hidden, "argmax": am, "drafts": drafts, "targets": tg}
        if record:
            out.update({"tokens": self.tokens.clone(), "new_counts": self.chain_counts.clone(),
                        "ctx_len": self.chain_ctx.clone()})
        acc, anc, offs, toks = hdf.accept(am[1:], tg, K=B - 1, draft_stride=B,
                                          out=(self.acc, self.anc, self.offs, self.toks))
        hdf.advance_context(acc, self.chain_ctx, self.chain_counts, next_anchor=anc,
                            block_tokens=self.tokens)
        # the lengths after this round, read back without waiting
        k = self._rb_slot
        if any(slot == k for _, slot, _ in self._rb_pending):
            self._tighten(wait=True)
        self._rb_host[k].copy_(self.chain_ctx, non_blocking=True)
        ev = torch.cuda.Event()
        ev.record()
        self._rb_pending.append((ev, k, self._rounds))
        self._rb_slot = (k + 1) % len(self._rb_host)
        self._rounds += 1
        self._ctx_hi = self._ctx_hi + B
        out.update({"accept_len": acc, "next_anchor": anc, "commit_offsets": offs,
                    "commit_tokens": toks})
        return out

    def sync_lengths(self) -> np.ndarray:
        """Waits for every read-back: the exact device lengths (host copy)."""
        self._tighten(wait=True)
        return self.ctx.copy()

    def next_counts(self, accept_len: torch.Tensor) -> np.ndarray:
        """n_s + 1 committed positions per sequence: the next round's new rows (reads
        the accepted lengths back to the host)."""
        return accept_len.cpu().numpy().astype(np.int64) + 1
