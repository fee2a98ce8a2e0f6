"""Builds drafter test cases on the GPU and the matching oracle inputs (host copies of
the very same bits)."""
import dataclasses

import numpy as np
import torch

import synth
from oracle.drafter import Weights
from paper_2606_26744_amd import hdf


def bits(t):
    return synth.to_numpy_bits(t)


class DraftCase:
    """ctx[s] context length of sequence s; new[s] rows of it projected by this call (the
    last ones); the rows before come from a synthetic already-filled cache.  With
    `stride` (paged cache only) every sequence has `stride` rows in y_new of which the
    first new[s] are new, given to the call as device row counts."""

    def __init__(self, wl, ctx, new, *, B=None, random_norms=True, rope=True, sub=0,
                 max_ctx=None, y_from=None, paged=False, spare_pages=0, stride=None):
        self.wl = wl = dataclasses.replace(wl, n_seq=len(ctx), ctx_lens=list(ctx),
                                           block=B or wl.block)
        dr = wl.drafter
        self.B = wl.block
        self.ctx = list(ctx)
        self.new = list(new)
        self.max_ctx = max_ctx if max_ctx is not None else max(self.ctx)
        dev = "cuda"
        self.w = synth.drafter_weights(wl, device=dev, random_norms=random_norms)
        theta = dr.rope_theta if rope else 0.0
        self.h = hdf.DrafterHandle(self.w, n_layers=dr.n_layers, d=dr.d, n_heads=dr.n_heads,
                                   head_dim=dr.head_dim, d_ff=dr.d_ff, vocab=dr.vocab, eps=dr.eps,
                                   rope_theta=theta, rope_max_pos=self.max_ctx + self.B)
        self.theta = theta
        offs = hdf.kv_slot_offsets(self.ctx)
        self.paged = paged
        if paged:
            # A pool with spare pages; every sequence gets pages at random places of it
            # (seeded), so no sequence's rows are contiguous.
            need = [(t + 63) // 64 for t in self.ctx]
            n_pages = sum(need) + spare_pages
            perm = np.random.default_rng(1000 + sub).permutation(n_pages).tolist()
            self.pages, k = [], 0
            for n in need:
                self.pages.append(perm[k:k + n])
                k += n
            self.max_pages = max(max(need), (self.max_ctx + 63) // 64)
            pt = np.full((len(self.ctx), self.max_pages), -1, dtype=np.int32)
            for s_, pg in enumerate(self.pages):
                pt[s_, :len(pg)] = pg
            self.page_table = torch.as_tensor(pt).to(dev)
            self.kv_offsets = None
            self.kv_k, self.kv_vt = self.h.alloc_kv(max(n_pages, 1) * 64)
        else:
            self.page_table = None
            self.kv_offsets = torch.tensor(offs, dtype=torch.int32, device=dev)
            self.cap = offs[-1]
            self.kv_k, self.kv_vt = self.h.alloc_kv(max(self.cap, 64))
        self.ctx_len = torch.tensor(self.ctx, dtype=torch.int32, device=dev)
        nh, hd, L = dr.n_heads, dr.head_dim, dr.n_layers
        self.prefix = []
        for s, (T, n) in enumerate(zip(self.ctx, self.new)):
            t0 = T - n
            per_layer = []
            for l in range(L):
                if t0 > 0:
                    k, v = synth.kv_prefix(wl, t0, l, device=dev, sub=sub * 1000 + s)
                    if paged:
                        hdf.write_kv_rows_paged(self.kv_k, self.kv_vt, l, self.pages[s], k, v)
                    else:
                        hdf.write_kv_rows(self.kv_k, self.kv_vt, l, offs[s], k, v)
                    per_layer.append((bits(k), bits(v)))
                else:
                    per_layer.append((np.zeros((0, dr.d)), np.zeros((0, dr.d))))
            self.prefix.append(per_layer)
        self.stride = stride
        self.new_counts = None
        if stride is not None:
            if not paged or max(self.new) > stride:
                raise ValueError("stride goes with a paged cache and new[s] <= stride")
            no = [s_ * stride for s_ in range(len(self.ctx) + 1)]
            self.new_counts = torch.tensor(self.new, dtype=torch.int32, device=dev)
        else:
            no = [0]
            for n in self.new:
                no.append(no[-1] + n)
        self.new_offsets = torch.tensor(no, dtype=torch.int32, device=dev)
        self.n_new = no[-1]
        self.y_new = (synth.reduced_states(wl, self.n_new, device=dev, sub=sub) if y_from is None
                      else y_from)
        self.tokens = synth.block_tokens(wl, device=dev, sub=sub)

    def run(self, hidden=None, ws=None):
        return self.h.draft_block(ctx_len=self.ctx_len, max_ctx=self.max_ctx, y_new=self.y_new,
                                  new_offsets=self.new_offsets, kv_offsets=self.kv_offsets,
                                  page_table=self.page_table, new_counts=self.new_counts,
                                  kv_k=self.kv_k, kv_vt=self.kv_vt,
                                  tokens=self.tokens, hidden=hidden, ws=ws)

    def read_cache(self, s, layer):
        """Keys and values of positions 0..T_s-1 of sequence s, as [T_s, d] tensors."""
        T = self.ctx[s]
        if self.paged:
            return hdf.read_kv_rows_paged(self.kv_k, self.kv_vt, layer, self.pages[s], T)
        return hdf.read_kv_rows(self.kv_k, self.kv_vt, layer, int(self.kv_offsets[s]), T)

    def oracle_weights(self):
        dr = self.wl.drafter
        wb = {k: ([bits(x) for x in v] if isinstance(v, list) else bits(v))
              for k, v in self.w.items()}
        return Weights(wb, d=dr.d, n_layers=dr.n_layers, n_heads=dr.n_heads, head_dim=dr.head_dim,
                       d_ff=dr.d_ff, vocab=dr.vocab, eps=dr.eps, rope_theta=self.theta,
                       dtype=self.wl.dtype)

    def y_rows(self, s):
        no = self.new_offsets.tolist()
        return bits(self.y_new[no[s]:no[s] + self.new[s]])

    def oracle_inputs(self):
        ys = [self.y_rows(s) for s in range(len(self.ctx))]
        return ys, bits(self.tokens)
