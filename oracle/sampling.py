"""Oracle of temperature sampling and of speculative-sampling verification (the
temperature-1 rows of the paper's result tables).  Test infrastructure only.

The paper reports acceptance at temperature 1 (Tables 2 and 3, Sec. 3) without
spelling out the verification rule.  Reading taken here: the standard speculative
sampling rule of the speculative-decoding literature it builds on.  Draft token x_i
(block slot i+1, drawn from the draft distribution q_i) is accepted with probability
min(1, p_i(x_i) / q_i(x_i)), where p_i is the target's distribution at that
position; at the first rejection (slot n) the next token is drawn from
max(0, p_n - q_n) renormalised; when all K drafts are accepted it is drawn from p_K
(the bonus token).  Both distributions are softmax(logits / T).

Random numbers (so that the GPU path and this oracle draw the same ones): the
counter-based generator Philox4x64-10 (Salmon, Moraes, Dror, Shaw, "Parallel random
numbers: as easy as 1, 2, 3", SC'11) with key (seed, stream) and counter
(row, v // 8, purpose, 0); of the block's four 64-bit words, word (v % 8) // 2 gives
two uniforms, one from each 32-bit half (the high half for even v, the low half for
odd v): u = (top 24 bits of the half + 1/2) / 2^24, in (0, 1).  Purposes: 0 = Gumbel noise of draft
sampling (row = logits row, v = vocabulary index), 1 = acceptance uniforms
(row = sequence, v = slot), 2 = Gumbel noise of the residual or bonus sample
(row = sequence, v = vocabulary index).  A sample from softmax(s) is
argmax_v (s_v + g_v) with g_v = -log(-log u_v) (the Gumbel-max construction).
"""
from __future__ import annotations

import numpy as np

PURPOSE_DRAFT, PURPOSE_ACCEPT, PURPOSE_RESAMPLE = 0, 1, 2

_M0, _M1 = np.uint64(0xD2E7470EE14C6C93), np.uint64(0xCA5A826395121157)
_W0, _W1 = np.uint64(0x9E3779B97F4A7C15), np.uint64(0xBB67AE8584CAA73B)
_LO32 = np.uint64(0xFFFFFFFF)
_S32 = np.uint64(32)


def _mulhilo(a: np.ndarray, b: np.uint64):
    """128-bit product of uint64 arrays a and a constant b: (high word, low word)."""
    a_lo, a_hi = a & _LO32, a >> _S32
    b_lo, b_hi = b & _LO32, b >> _S32
    t = a_lo * b_lo
    u = a_hi * b_lo + (t >> _S32)
    w = a_lo * b_hi + (u & _LO32)
    hi = a_hi * b_hi + (u >> _S32) + (w >> _S32)
    lo = (w << _S32) | (t & _LO32)
    return hi, lo


def philox4x64_10(ctr: np.ndarray, key: np.ndarray) -> np.ndarray:
    """Philox4x64 with 10 rounds.  ctr [..., 4] uint64, key [..., 2] uint64 ->
    [..., 4] uint64."""
    c = [np.asarray(ctr[..., i], dtype=np.uint64) for i in range(4)]
    k0 = np.asarray(key[..., 0], dtype=np.uint64)
    k1 = np.asarray(key[..., 1], dtype=np.uint64)
    with np.errstate(over="ignore"):
        for r in range(10):
            if r > 0:
                k0 = k0 + _W0
                k1 = k1 + _W1
            hi0, lo0 = _mulhilo(c[0], _M0)
            hi1, lo1 = _mulhilo(c[2], _M1)
            c = [hi1 ^ c[1] ^ k0, lo1, hi0 ^ c[3] ^ k1, lo0]
    return np.stack(c, axis=-1)


def uniforms(seed: int, stream: int, rows, vs, purpose: int) -> np.ndarray:
    """u for every (row, v) pair (broadcast shapes), float64 in (0, 1)."""
    rows, vs = np.broadcast_arrays(np.asarray(rows, dtype=np.uint64),
                                   np.asarray(vs, dtype=np.uint64))
    ctr = np.stack([rows, vs >> np.uint64(3), np.full(rows.shape, purpose, dtype=np.uint64),
                    np.zeros(rows.shape, dtype=np.uint64)], axis=-1)
    key = np.broadcast_to(np.array([seed, stream], dtype=np.uint64), rows.shape + (2,))
    out = philox4x64_10(ctr, key)
    j = ((vs & np.uint64(7)) >> np.uint64(1)).astype(np.int64)
    word = np.take_along_axis(out, j[..., None], axis=-1)[..., 0]
    half = np.where((vs & np.uint64(1)) == 0, word >> np.uint64(32), word & _LO32)
    return ((half >> np.uint64(8)).astype(np.float64) + 0.5) / float(1 << 24)


def gumbel(u: np.ndarray) -> np.ndarray:
    return -np.log(-np.log(u))


def _lse(s: np.ndarray) -> np.ndarray:
    m = s.max(axis=-1, keepdims=True)
    return (m + np.log(np.exp(s - m).sum(axis=-1, keepdims=True)))[..., 0]


def sample_tokens(logits, temperature: float, seed: int, stream: int, rows=None):
    """Draws one token per row from softmax(logits / T).

    logits [R, V]; rows: the row ids used as Philox counters (default 0..R-1).
    Returns (tokens [R] int32, lse [R] = logsumexp(logits / T), margin [R] = gap
    between the best and second-best perturbed score)."""
    z = np.asarray(logits, dtype=np.float64) / temperature
    R, V = z.shape
    rows = np.arange(R) if rows is None else np.asarray(rows)
    g = gumbel(uniforms(seed, stream, rows[:, None], np.arange(V)[None, :], PURPOSE_DRAFT))
    score = z + g
    tok = np.argmax(score, axis=1)
    top2 = np.sort(score, axis=1)[:, -2:]
    return tok.astype(np.int32), _lse(z), top2[:, 1] - top2[:, 0]


def accept_sample(drafts, draft_logits, target_logits, temperature: float, seed: int,
                  stream: int):
    """Speculative-sampling verification of a batch of blocks.

    drafts [n, K] int; draft_logits [n, K, V] (the draft logits of slots 1..K);
    target_logits [n, K+1, V] (row i: the target's logits for the token at slot i+1,
    row K: for the token after the last draft).
    Returns (accept_len [n], next_token [n], commit_offsets [n+1],
             commit_tokens [sum(n_s + 1)], decision_margin [n], sample_margin [n]):
    the committed tokens of sequence s are its accepted drafts then next_token;
    decision_margin is the smallest |u q - p| / max(p, q) over the decisions taken and
    sample_margin the top-2 gap of the final draw (for tolerant comparisons)."""
    drafts = np.asarray(drafts)
    n, K = drafts.shape
    V = np.asarray(target_logits).shape[-1]
    zt = np.asarray(target_logits, dtype=np.float64) / temperature
    acc = np.zeros(n, dtype=np.int32)
    nxt = np.zeros(n, dtype=np.int32)
    dmarg = np.full(n, np.inf)
    smarg = np.zeros(n)
    toks = []
    for s in range(n):
        lp = zt[s] - _lse(zt[s])[:, None]                       # log p_i, [K+1, V]
        if K > 0:
            zd = np.asarray(draft_logits[s], dtype=np.float64) / temperature
            lq = zd - _lse(zd)[:, None]                          # log q_i, [K, V]
        u = uniforms(seed, stream, s, np.arange(K), PURPOSE_ACCEPT) if K > 0 else []
        k = 0
        while k < K:
            x = int(drafts[s, k])
            p, q = np.exp(lp[k, x]), np.exp(lq[k, x])
            dmarg[s] = min(dmarg[s], abs(u[k] * q - p) / max(p, q))
            if u[k] * q < p:
                k += 1
            else:
                break
        g = gumbel(uniforms(seed, stream, s, np.arange(V), PURPOSE_RESAMPLE))
        if k < K:
            w = np.maximum(0.0, np.exp(lp[k]) - np.exp(lq[k]))
            if np.any(w > 0):
                with np.errstate(divide="ignore"):
                    score = np.where(w > 0, np.log(w), -np.inf) + g
            else:
                score = lp[k] + g
        else:
            score = lp[K] + g
        t = int(np.argmax(score))
        top2 = np.sort(score)[-2:]
        smarg[s] = top2[1] - top2[0]
        acc[s], nxt[s] = k, t
        toks.extend([int(x) for x in drafts[s, :k]] + [t])
    offs = np.concatenate([[0], np.cumsum(acc + 1)]).astype(np.int32)
    return acc, nxt, offs, np.asarray(toks, dtype=np.int32), dmarg, smarg
