"""Oracle of greedy acceptance.  Test infrastructure only.

The target verifies the drafted tokens in parallel and keeps the longest prefix
that agrees with its own tokens (Sec. 1); the accepted length tau is the mean
number of tokens committed per verification round (Sec. 3.4).  Reading: tau
counts the target's own token after the agreed prefix (the bonus token), since
Table 2 prints tau above the number of drafted steps for MTP (3).  So for one
round with K drafts d_1..d_K and target tokens t_1..t_{K+1}:
    n = max { j <= K : d_i = t_i for all i <= j }
    committed tokens = t_1..t_{n+1},   next anchor = t_{n+1},   tau = n + 1.
"""
from __future__ import annotations

import numpy as np


def accept(draft, target):
    """draft [n_seq, K], target [n_seq, K+1] ->
    (accept_len [n_seq], next_anchor [n_seq], commit_offsets [n_seq+1],
     commit_tokens [sum(n+1)])  -- all int32."""
    draft = np.asarray(draft)
    target = np.asarray(target)
    n_seq, K = draft.shape
    assert target.shape == (n_seq, K + 1)
    acc = np.zeros(n_seq, dtype=np.int32)
    anchor = np.zeros(n_seq, dtype=np.int32)
    commits = []
    for s in range(n_seq):
        n = 0
        while n < K and draft[s, n] == target[s, n]:
            n += 1
        acc[s] = n
        anchor[s] = target[s, n]
        commits.append(target[s, :n + 1])
    offs = np.zeros(n_seq + 1, dtype=np.int32)
    for s in range(n_seq):
        offs[s + 1] = offs[s] + acc[s] + 1
    toks = np.concatenate(commits).astype(np.int32) if commits else np.zeros(0, np.int32)
    return acc, anchor, offs, toks
