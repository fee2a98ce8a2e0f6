"""Chained drafting rounds over the paged KV cache (paper_2606_26744_amd.decode):
every round is checked against the oracle given the GPU's own state before it (its
cache rows, lengths and anchors), so a near-tie flipping one draft cannot make later
rounds diverge from what is checked.

Per round: the reduced rows, the cache rows the round appends (pages taken from a
shuffled pool as the sequences grow), the block states, the LM head's argmax on the
GPU's block states (exact outside 1e-2 top-2 margins) and the acceptance (exact)."""
import numpy as np
import pytest
import torch

import synth
from oracle.accept import accept as ref_accept
from oracle.drafter import context_kv, draft_block as ref_draft
from oracle.lm_head import lm_head_argmax as ref_lm
from oracle.numerics import as_f64
from oracle.reducer import hc_reduce as ref_reduce
from paper_2606_26744_amd import hdf
from paper_2606_26744_amd.decode import PagedDecoder
from tests._case import bits
from tests._tol import assert_bf16_close, assert_bf16_state_close, assert_f32_rows_close
from oracle.drafter import Weights

pytestmark = pytest.mark.gpu


def _targets_fn(p, V, seed):
    """Stand-in for the target model: copies each draft with probability p, otherwise a
    different token; the last slot (the token after the drafts) is uniform."""
    def fn(drafts):
        g = torch.Generator(device=drafts.device).manual_seed(seed)
        n, K = drafts.shape
        u = torch.rand((n, K), generator=g, device=drafts.device)
        off = torch.randint(0, V - 1, (n, K), generator=g, device=drafts.device, dtype=torch.int64)
        other = ((drafts.long() + 1 + off) % V).to(torch.int32)
        t = torch.where(u < p, drafts, other)
        bonus = torch.randint(0, V, (n, 1), generator=g, device=drafts.device, dtype=torch.int64)
        return torch.cat([t, bonus.to(torch.int32)], dim=1).contiguous()
    return fn


def _oracle_weights(w, dr, dtype, theta):
    wb = {k: ([bits(x) for x in v] if isinstance(v, list) else bits(v)) for k, v in w.items()}
    return Weights(wb, d=dr.d, n_layers=dr.n_layers, n_heads=dr.n_heads, head_dim=dr.head_dim,
                   d_ff=dr.d_ff, vocab=dr.vocab, eps=dr.eps, rope_theta=theta, dtype=dtype)


def _run(wl, prompts, rounds, p, seed, check_seqs):
    dr = wl.drafter
    n_seq, B = len(prompts), wl.block
    max_ctx = max(prompts) + rounds * B
    w = synth.drafter_weights(wl, device="cuda")
    h = hdf.DrafterHandle(w, n_layers=dr.n_layers, d=dr.d, n_heads=dr.n_heads,
                          head_dim=dr.head_dim, d_ff=dr.d_ff, vocab=dr.vocab, eps=dr.eps,
                          rope_theta=dr.rope_theta, rope_max_pos=max_ctx + B)
    n_pages = sum((t + rounds * B + 63) // 64 for t in prompts) + 7
    order = np.random.default_rng(seed).permutation(n_pages)
    dec = PagedDecoder(h, n_seq, B, max_ctx, n_pages, max(sum(prompts), n_seq * B),
                       page_order=order)
    dec.set_anchors(torch.as_tensor(np.random.default_rng(seed + 1).integers(0, dr.vocab, n_seq),
                                    dtype=torch.int32).cuda())
    W = _oracle_weights(w, dr, wl.dtype, dr.rope_theta)
    wlm = bits(w["w_lm"])
    counts = np.asarray(prompts, dtype=np.int64)
    total_acc = []
    for r in range(rounds):
        n_new = int(counts.sum())
        red = synth.reducer_inputs(wl, n_new, device="cuda", sub=100 + r)
        before = dec.ctx.copy()
        prefix = {}
        for s in check_seqs:
            per_layer = []
            for l in range(dr.n_layers):
                k, v = hdf.read_kv_rows_paged(dec.kv_k, dec.kv_vt, l, dec.pages[s], int(before[s]))
                per_layer.append((bits(k), bits(v)))
            prefix[s] = per_layer
        print(f"[decode] {wl.name} round {r} new rows {counts.tolist()} ctx {before.tolist()}",
              flush=True)
        out = dec.round(red["H"], counts, red["W_g"], red["b_g"], _targets_fn(p, dr.vocab, seed + r))
        torch.cuda.synchronize()
        offs = np.concatenate([[0], np.cumsum(counts)])
        Hn, Wg, bg = bits(red["H"]), bits(red["W_g"]), bits(red["b_g"])
        toks = bits(out["tokens"])
        ys = [None] * n_seq
        for s in check_seqs:
            y_ref = ref_reduce(Hn[offs[s]:offs[s + 1]], Wg, bg, dtype=wl.dtype)[0]
            y_gpu = bits(out["Y"][offs[s]:offs[s + 1]])
            if wl.dtype == "bf16":
                assert_bf16_close(as_f64(y_gpu), y_ref, "Y")
            else:
                assert_f32_rows_close(y_gpu, y_ref, "Y")
            ys[s] = y_gpu
            # cache rows this round appended
            kv = context_kv(W, as_f64(y_gpu), np.arange(before[s], before[s] + counts[s]))
            for l in range(dr.n_layers):
                kk, vv = hdf.read_kv_rows_paged(dec.kv_k, dec.kv_vt, l, dec.pages[s],
                                                int(dec.ctx[s]))
                k, v = kk[int(before[s]):], vv[int(before[s]):]
                if wl.dtype == "bf16":
                    assert_bf16_state_close(as_f64(bits(k.contiguous())), kv[l][0], "cache K")
                    assert_bf16_state_close(as_f64(bits(v.contiguous())), kv[l][1], "cache V")
                else:
                    assert_f32_rows_close(k.cpu().numpy(), kv[l][0], "cache K")
                    assert_f32_rows_close(v.cpu().numpy(), kv[l][1], "cache V")
        hid_ref = ref_draft(W, ys, toks, kv_prefix=[prefix.get(s) for s in range(n_seq)],
                            seqs=check_seqs)
        rows = np.concatenate([np.arange(s * B, (s + 1) * B) for s in check_seqs])
        hid = bits(out["hidden"][torch.as_tensor(rows).cuda()])
        if wl.dtype == "bf16":
            assert_bf16_state_close(as_f64(hid), hid_ref, "hidden")
        else:
            assert_f32_rows_close(hid, hid_ref, "hidden")
        # LM head on the GPU's own block states
        am_ref, _, margin = ref_lm(hid, wlm)
        am = out["argmax"].cpu().numpy()[rows]
        ok = margin >= (1e-2 if wl.dtype == "bf16" else 1e-4)
        assert ok.mean() > 0.8
        assert np.array_equal(am[ok], am_ref[ok])
        # acceptance on the GPU's drafts and targets: exact
        drafts = out["drafts"].cpu().numpy()
        tg = out["targets"].cpu().numpy()
        r_acc, r_anc, r_offs, r_toks = ref_accept(drafts, tg)
        acc = out["accept_len"].cpu().numpy()
        assert np.array_equal(acc, r_acc) and np.array_equal(out["next_anchor"].cpu().numpy(), r_anc)
        assert np.array_equal(out["commit_offsets"].cpu().numpy(), r_offs)
        assert np.array_equal(out["commit_tokens"].cpu().numpy()[:r_offs[-1]], r_toks)
        total_acc.append(acc)
        counts = dec.next_counts(out["accept_len"])
        assert np.array_equal(counts, acc + 1)
    # the cache holds every committed position of every sequence, pages never shared
    allp = [p for s in range(n_seq) for p in dec.pages[s]]
    assert len(allp) == len(set(allp))
    assert all(len(dec.pages[s]) == (int(dec.ctx[s]) + 63) // 64 for s in range(n_seq))
    return np.array(total_acc)


def test_small_bf16_six_rounds():
    wl = synth.small_bf16()
    acc = _run(wl, [100, 37, 64, 250], rounds=6, p=0.7, seed=5, check_seqs=[0, 1, 2, 3])
    print("accept lengths per round", acc.tolist(), flush=True)


def test_tiny_fp32_rounds():
    wl = synth.tiny_fp32()
    wl.drafter = synth.DrafterShape(d=256, n_layers=2, n_heads=4, head_dim=64, d_ff=512,
                                    vocab=500)
    _run(wl, [70, 5], rounds=4, p=0.9, seed=6, check_seqs=[0, 1])


def _chained_decoder(wl, prompts, rounds, seed, sentinel=None):
    """A decoder whose sequences have cached prompts[s] - B positions (pages from a
    shuffled pool); the first chained round projects the last B of every prompt."""
    dr = wl.drafter
    n_seq, B = len(prompts), wl.block
    max_ctx = max(prompts) + (rounds + 1) * B
    w = synth.drafter_weights(wl, device="cuda")
    h = hdf.DrafterHandle(w, n_layers=dr.n_layers, d=dr.d, n_heads=dr.n_heads,
                          head_dim=dr.head_dim, d_ff=dr.d_ff, vocab=dr.vocab, eps=dr.eps,
                          rope_theta=dr.rope_theta, rope_max_pos=max_ctx + B)
    n_pages = n_seq * ((max_ctx + 63) // 64) + 5
    order = np.random.default_rng(seed).permutation(n_pages)
    dec = PagedDecoder(h, n_seq, B, max_ctx, n_pages, n_seq * B, page_order=order)
    if sentinel is not None:
        dec.kv_k.fill_(sentinel)
        dec.kv_vt.fill_(sentinel)
    pre = [t - B for t in prompts]
    dec.preload(pre)
    for s in range(n_seq):
        for l in range(dr.n_layers):
            k, v = synth.kv_prefix(wl, pre[s], l, device="cuda", sub=50 + s)
            if sentinel is not None:   # whole tiles: the rows past the prefix keep the sentinel
                pad = (-pre[s]) % 64
                k = torch.cat([k, torch.full((pad, k.shape[1]), sentinel, dtype=k.dtype,
                                             device=k.device)])
                v = torch.cat([v, torch.full((pad, v.shape[1]), sentinel, dtype=v.dtype,
                                             device=v.device)])
            hdf.write_kv_rows_paged(dec.kv_k, dec.kv_vt, l, dec.pages[s], k, v)
    dec.set_anchors(torch.as_tensor(np.random.default_rng(seed + 1).integers(0, dr.vocab, n_seq),
                                    dtype=torch.int32).cuda())
    dec.start_chain([B] * n_seq)
    return dec, w


def test_chained_rounds_match_oracle():
    """Chained rounds (lengths and row counts stay on the device, launches sized for B
    rows per sequence): every round against the oracle given the GPU's own state; the
    rows past each sequence's new rows are never written (the pool starts as a sentinel
    and every row outside the sequences' committed positions still holds it)."""
    wl = synth.small_bf16()
    dr = wl.drafter
    prompts, rounds, B = [100, 37, 64, 250], 6, wl.block
    n_seq = len(prompts)
    sentinel = -3.0
    dec, w = _chained_decoder(wl, prompts, rounds, seed=8, sentinel=sentinel)
    W = _oracle_weights(w, dr, wl.dtype, dr.rope_theta)
    wlm = bits(w["w_lm"])
    for r in range(rounds):
        torch.cuda.synchronize()
        T = dec.chain_ctx.cpu().numpy().astype(np.int64)
        cnt = dec.chain_counts.cpu().numpy().astype(np.int64)
        before = T - cnt
        prefix = {}
        for s in range(n_seq):
            prefix[s] = [tuple(bits(x) for x in hdf.read_kv_rows_paged(
                dec.kv_k, dec.kv_vt, l, dec.pages[s], int(before[s]))) for l in range(dr.n_layers)]
        print(f"[decode chained] round {r} ctx {T.tolist()} new rows {cnt.tolist()}", flush=True)
        red = synth.reducer_inputs(wl, n_seq * B, device="cuda", sub=300 + r)
        out = dec.chained_round(red["H"], red["W_g"], red["b_g"], _targets_fn(0.7, dr.vocab, 40 + r),
                                record=True)
        torch.cuda.synchronize()
        assert np.array_equal(out["ctx_len"].cpu().numpy(), T)
        assert np.array_equal(out["new_counts"].cpu().numpy(), cnt)
        Hn, Wg, bg = bits(red["H"]), bits(red["W_g"]), bits(red["b_g"])
        ys = []
        for s in range(n_seq):
            rows = slice(s * B, s * B + int(cnt[s]))
            y_gpu = bits(out["Y"][rows])
            assert_bf16_close(as_f64(y_gpu), ref_reduce(Hn[rows], Wg, bg, dtype=wl.dtype)[0], "Y")
            ys.append(y_gpu)
            kv = context_kv(W, as_f64(y_gpu), np.arange(before[s], T[s]))
            for l in range(dr.n_layers):
                kk, vv = hdf.read_kv_rows_paged(dec.kv_k, dec.kv_vt, l, dec.pages[s], int(T[s]))
                assert_bf16_state_close(as_f64(bits(kk[int(before[s]):].contiguous())), kv[l][0],
                                        "cache K")
                assert_bf16_state_close(as_f64(bits(vv[int(before[s]):].contiguous())), kv[l][1],
                                        "cache V")
        toks = bits(out["tokens"])
        hid_ref = ref_draft(W, ys, toks, kv_prefix=[prefix[s] for s in range(n_seq)],
                            seqs=list(range(n_seq)))
        hid = bits(out["hidden"])
        assert_bf16_state_close(as_f64(hid), hid_ref, "hidden")
        am_ref, _, margin = ref_lm(hid, wlm)
        am = out["argmax"].cpu().numpy()
        ok = margin >= 1e-2
        assert ok.mean() > 0.8 and np.array_equal(am[ok], am_ref[ok])
        r_acc, r_anc, r_offs, r_toks = ref_accept(out["drafts"].cpu().numpy(),
                                                  out["targets"].cpu().numpy())
        acc = out["accept_len"].cpu().numpy()
        assert np.array_equal(acc, r_acc)
        assert np.array_equal(out["next_anchor"].cpu().numpy(), r_anc)
        assert np.array_equal(out["commit_tokens"].cpu().numpy()[:r_offs[-1]], r_toks)
        assert np.array_equal(dec.chain_ctx.cpu().numpy(), T + acc + 1)
        assert np.array_equal(dec.chain_counts.cpu().numpy(), acc + 1)
    # every row outside the committed positions still holds the sentinel
    T = dec.sync_lengths()
    assert np.array_equal(T, dec.chain_ctx.cpu().numpy())
    used = np.zeros((dec.kv_k.shape[2], 64), dtype=bool)
    for s in range(n_seq):
        for i in range(int(T[s])):
            used[dec.pages[s][i // 64], i % 64] = True
    # the tail rows of every sequence's pages, through the layout helper
    for s in range(n_seq):
        pages = dec.pages[s]
        n_rows = len(pages) * 64
        for l in range(dr.n_layers):
            kk, vv = hdf.read_kv_rows_paged(dec.kv_k, dec.kv_vt, l, pages, n_rows)
            assert bool((kk[int(T[s]):].float() == sentinel).all())
            assert bool((vv[int(T[s]):].float() == sentinel).all())
    # and every page no sequence holds
    untouched = [p for p in range(dec.kv_k.shape[2]) if not used[p].any()]
    assert bool((dec.kv_k[:, :, untouched].float() == sentinel).all())
    assert bool((dec.kv_vt[:, :, untouched].float() == sentinel).all())


def test_chained_rounds_need_no_host_wait():
    """Twelve chained rounds launched back to back with no synchronisation give results
    bit-identical to the same rounds with the host synchronising (and tightening its
    page bound) after every one: the host never needs the accepted lengths."""
    wl = synth.small_bf16()
    dr = wl.drafter
    prompts, rounds, B = [300, 37, 90], 12, wl.block
    outs = []
    for wait in (False, True):
        dec, _ = _chained_decoder(wl, prompts, rounds, seed=9)
        red = [synth.reducer_inputs(wl, len(prompts) * B, device="cuda", sub=500 + r)
               for r in range(rounds)]
        torch.cuda.synchronize()
        accs = []
        for r in range(rounds):
            o = dec.chained_round(red[r]["H"], red[r]["W_g"], red[r]["b_g"],
                                  _targets_fn(0.8, dr.vocab, 70 + r))
            accs.append(o["accept_len"].clone())
            if wait:
                torch.cuda.synchronize()
                dec.sync_lengths()
        torch.cuda.synchronize()
        T = dec.sync_lengths()
        rows = []
        for s in range(len(prompts)):
            for l in range(dr.n_layers):
                kk, vv = hdf.read_kv_rows_paged(dec.kv_k, dec.kv_vt, l, dec.pages[s], int(T[s]))
                rows.append((bits(kk), bits(vv)))
        outs.append((T, torch.stack(accs).cpu().numpy(), rows, bits(dec.hidden), bits(dec.tokens)))
        del dec
        torch.cuda.empty_cache()
    (Ta, aa, ra, ha, ta), (Tb, ab, rb, hb, tb) = outs
    print("accept lengths per round", aa.tolist(), flush=True)
    assert np.array_equal(Ta, Tb) and np.array_equal(aa, ab)
    assert np.array_equal(ha, hb) and np.array_equal(ta, tb)
    for (ka, va), (kb, vb) in zip(ra, rb):
        assert np.array_equal(ka, kb) and np.array_equal(va, vb)
    assert (Ta == np.asarray(prompts) + (aa + 1).sum(axis=0)).all()
