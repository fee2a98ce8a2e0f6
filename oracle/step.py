"""Oracle of one whole drafter step.  Test infrastructure only.

One decode round of the method (Sec. 1, Sec. 2.1, Fig. 2 caption): the target's
pre-collapse residual rows of the newest context positions are reduced by the
gated reducer (Eq. (1)), projected into the drafter's context, the block
[anchor, mask, ..., mask] is drafted in one pass, the LM head gives the draft
tokens of slots 1..B-1 (slot k predicts position a+k, Sec. 2.3), and greedy
verification against the target's tokens gives the accepted length.
"""
from __future__ import annotations

from typing import Optional, Sequence

import numpy as np

from .accept import accept
from .drafter import Weights, draft_block
from .lm_head import lm_head_argmax
from .reducer import hc_reduce


def drafter_step(W: Weights, H_new: Sequence[np.ndarray], W_g, b_g, tokens, *,
                 kv_prefix=None, targets: Optional[np.ndarray] = None,
                 reduce_kw: Optional[dict] = None, seqs=None, reduce_dtype=None):
    """H_new[s]: [n_s, m, d] residual rows of sequence s reduced this step.
    Returns a dict with Y (per sequence), hidden, argmax, logits, margin, draft,
    and, when targets are given, the acceptance outputs."""
    reduce_kw = dict(reduce_kw or {})
    reduce_kw.setdefault("eps", W.eps)
    tokens = np.asarray(tokens)
    if seqs is None:
        seqs = list(range(tokens.shape[0]))
    ys = {}
    for s in seqs:
        y, _ = hc_reduce(H_new[s], W_g, b_g, dtype=reduce_dtype or W.dtype, **reduce_kw)
        ys[s] = y
    y_list = [ys.get(s) for s in range(tokens.shape[0])]
    hidden = draft_block(W, y_list, tokens, kv_prefix=kv_prefix, seqs=seqs)
    am, logits, margin = lm_head_argmax(hidden, W.w_lm)
    B = tokens.shape[1]
    draft = am.reshape(len(seqs), B)[:, 1:]
    out = {"Y": ys, "hidden": hidden, "argmax": am, "logits": logits,
           "margin": margin, "draft": draft}
    if targets is not None:
        tg = np.asarray(targets)[list(seqs)]
        acc, anchor, offs, toks = accept(draft, tg)
        out.update(accept_len=acc, next_anchor=anchor, commit_offsets=offs,
                   commit_tokens=toks)
    return out
