#!/usr/bin/env python3
"""Benchmark of one HyperDFlash drafter step on one MI355X.

A step is one pass of the whole hot path over one batch of synthetic input:
    gated reduce of the newest context rows -> block draft (context K/V append,
    attention over cached context + block, MLP) -> LM head argmax -> acceptance.
Workload (default): the full-size warm step -- 8 sequences with 2048 context
positions each, 16 of them new this round (reduced and projected), a drafter of
d=4096 (32 heads x 128, SiLU MLP 12288), vocabulary 129280, block B=16; bf16 storage
with fp32 accumulation; seeded synthetic weights and inputs already resident in HBM.

Prints ONE JSON line (rank 0 of a single process).  Extras: per-stage times, the LM
head's roofline (the dominant kernel, timed live with HIP events on the stream it runs
on), the reducer at its bandwidth-stress size, and the CPU oracle timed on a bounded
sample on this host.
"""
import argparse
import gc
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
# HBM bytes of one 128-row LM-head GEMM launch (hdf_lm_head_argmax_keys) from the two
# rocprofv3 --pmc runs recorded in profiles/lm_head_argmax_hbm_counters.md:
# FETCH_SIZE x 1.99997 + WRITE_SIZE x 1.000 KiB, the factors a 2 GiB device copy reads on
# the same counters.  Valid only for the kernel source it was measured on: reported as
# null once the code of gemm.hip or common.hpp changes.
LM_HEAD_TRAFFIC = {"source_sha": "edfa26705c1ac61f",
                   "bytes": (521553.1 * 1.99997 + 253.0 * 1.000) * 1024}
BF16_PEAK_TFLOPS = 2500.0
METRIC = "draft blocks/sec at d=4096,B=16,V=129280; reducer HBM GB/s; MFMA util %"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-reducer-stress", action="store_true")
    ap.add_argument("--no-m-sweep", action="store_true")
    ap.add_argument("--ragged", action="store_true",
                    help="(default; kept for old command lines) time the 64-sequence ragged "
                         "decode workload")
    ap.add_argument("--no-ragged", action="store_true",
                    help="skip the 64-sequence ragged decode workload")
    ap.add_argument("--cold", action="store_true",
                    help="also time the cold step (every context row reduced and projected)")
    ap.add_argument("--ragged-cold", action="store_true",
                    help="also time the cold step of the ragged workload (about 540K context "
                         "rows reduced and projected)")
    ap.add_argument("--no-cold-cache", action="store_true",
                    help="skip the headline step timed with the caches flushed before each step")
    ap.add_argument("--decode", type=int, default=0, metavar="R",
                    help="also time R chained rounds of the paged decode loop (8 sequences "
                         "from 2048 positions, n+1 committed positions appended per round)")
    ap.add_argument("--temperature", type=float, default=0.0, metavar="T",
                    help="also time the step at temperature T > 0 (draws from softmax(z / T) and "
                         "speculative-sampling verification against synthetic target logits)")
    ap.add_argument("--kl", action="store_true",
                    help="also time the KL-distillation forward on the full-size blocks")
    ap.add_argument("--fc-reducer", action="store_true",
                    help="also time the generic fc reducer beside the gated one (warm-step "
                         "rows and the reducer-stress shape)")
    ap.add_argument("--blas-ref", action="store_true",
                    help="also time the vendor BLAS (torch.matmul) on the matrix-core bound "
                         "GEMM shapes, for context")
    ap.add_argument("--copy-probe", action="store_true",
                    help="also run a plain 2 GiB device copy (counter calibration)")
    return ap.parse_args()


def build_workload(torch, synth, hdf, wl=None):
    """Device inputs of one warm step of workload wl (default: the full-size step): drafter
    weights, a KV cache holding every sequence's earlier context rows, the reducer inputs
    of the newest rows, block tokens and the step's buffers."""
    from paper_2606_26744_amd.step import StepBuffers
    wl = wl or synth.drafter_full()
    dr = wl.drafter
    n_seq, B = wl.n_seq, wl.block
    lens = [int(t) for t in wl.ctx_lens]
    news = lens if wl.cold else [wl.new_rows] * n_seq      # rows reduced/projected per step
    T = max(lens)
    dev = "cuda"
    w = synth.drafter_weights(wl, device=dev)
    h = hdf.DrafterHandle(w, n_layers=dr.n_layers, d=dr.d, n_heads=dr.n_heads,
                          head_dim=dr.head_dim, d_ff=dr.d_ff, vocab=dr.vocab, eps=dr.eps,
                          rope_theta=dr.rope_theta, rope_max_pos=T + B)
    offs = hdf.kv_slot_offsets(lens)
    kv_k, kv_vt = h.alloc_kv(offs[-1])
    for s in range(n_seq):          # rows of earlier rounds, already in the cache
        if lens[s] - news[s] <= 0:
            continue
        for l in range(dr.n_layers):
            k, v = synth.kv_prefix(wl, lens[s] - news[s], l, device=dev, sub=s)
            hdf.write_kv_rows(kv_k, kv_vt, l, offs[s], k, v)
            del k, v
    n_new = sum(news)
    red = synth.reducer_inputs(wl, n_new, device=dev)
    i32 = dict(dtype=torch.int32, device=dev)
    new_offsets = [0]
    for n in news:
        new_offsets.append(new_offsets[-1] + n)
    args = dict(H_new=red["H"], W_g=red["W_g"], b_g=red["b_g"],
                new_offsets=torch.tensor(new_offsets, **i32),
                ctx_len=torch.tensor(lens, **i32), max_ctx=T,
                kv_offsets=torch.tensor(offs, **i32), kv_k=kv_k, kv_vt=kv_vt,
                tokens=synth.block_tokens(wl, device=dev))
    bufs = StepBuffers(h, n_seq, B, n_new, T, wl.m)
    return wl, h, bufs, args, red, w, offs


def step_targets(torch, synth, hdf, wl, h, bufs, args):
    """Targets for greedy acceptance: copies of one untimed step's drafts with the
    workload's per-sequence probability, so acceptance lengths are geometric."""
    from paper_2606_26744_amd.step import drafter_step
    out = drafter_step(h, bufs, targets=None, **args)
    torch.cuda.synchronize()
    drafts = out["argmax"].view(wl.n_seq, wl.block)[:, 1:].cpu().numpy()
    return torch.as_tensor(synth.make_targets(drafts, wl.match_p, wl.drafter.vocab,
                                              seed=wl.seed)).cuda()


def ragged_leg(torch, synth, hdf, steps, warmup, wl=None, cpu_seqs=None):
    """A further step workload, timed like the headline step: by default the batched ragged
    decode workload (64 sequences, contexts U[1024, 16384]), warm-step blocks/s.  With
    cpu_seqs, the oracle's time on those sequences of the same step is reported beside it
    (a bounded sample of the workload, scaled to blocks/s)."""
    from paper_2606_26744_amd.step import drafter_step
    wl, h, bufs, args, red, w, offs = build_workload(torch, synth, hdf,
                                                     wl or synth.ragged_decode())
    tg = step_targets(torch, synth, hdf, wl, h, bufs, args)
    for _ in range(warmup):
        drafter_step(h, bufs, targets=tg, **args)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(steps):
        out = drafter_step(h, bufs, targets=tg, **args)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    acc = out["accept_len"].float()
    res = {"n_seq": wl.n_seq, "context_total": int(sum(wl.ctx_lens)),
           "context_min": int(min(wl.ctx_lens)), "context_max": int(max(wl.ctx_lens)),
           "blocks_per_s": round(wl.n_seq / (ms * 1e-3), 1), "ms_per_step": round(ms, 4),
           "steps": steps, "mean_accept_len": round(float(acc.mean()), 3)}
    if wl.cold:
        res["context_rows_projected"] = int(sum(wl.ctx_lens))
    if cpu_seqs is not None:
        res["cpu_baseline"] = cpu_baseline(torch, synth, wl, h, w, red, args, offs, seqs=cpu_seqs,
                                           budget_s=10.0)
    del wl, h, bufs, args, red, w
    gc.collect()
    torch.cuda.empty_cache()
    return res


def lm_head_m_sweep(torch, synth, hdf, h, d):
    """hdf_lm_head_argmax over the full vocabulary at M = 64 .. 2048 rows: time and the
    fraction of the bf16 matrix-core peak (the knee between the weight stream and the
    matrix cores)."""
    out = []
    for M in (64, 128, 192, 256, 384, 512, 1024, 2048):
        hid = synth.normal([M, d], 1.0, 7, 50, M, dtype="bf16", device="cuda")
        ws = torch.zeros(hdf.lm_head_workspace(M, h.V), dtype=torch.uint8, device="cuda")
        am = torch.empty(M, dtype=torch.int32, device="cuda")
        for _ in range(2):
            hdf.lm_head_argmax(hid, h.w_lm, ws=ws, out=(am, None), want_max=False)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        n = 10
        torch.cuda.synchronize()
        e0.record()
        for _ in range(n):
            hdf.lm_head_argmax(hid, h.w_lm, ws=ws, out=(am, None), want_max=False)
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) / n * 1e3
        tf = 2.0 * M * d * h.V / (us * 1e-6) / 1e12
        gbs = (h.V * d * 2 + M * d * 2) / (us * 1e-6) / 1e9
        out.append({"M": M, "us": round(us, 1), "TFLOP/s": round(tf, 1),
                    "mfma_frac": round(tf / BF16_PEAK_TFLOPS, 4), "GB/s": round(gbs, 1)})
        del hid, ws, am
    return out


def decode_leg(torch, synth, hdf, rounds, warmup):
    """Chained drafting rounds of the full-size drafter over the paged cache: 8
    sequences whose first 2032 context positions are already cached (pages taken in a
    shuffled order), a first round projecting the last 16, then one round after another
    appending each sequence's n_s + 1 committed positions.  The target model is stood in
    for by device-side tokens that copy each draft with probability 0.8.  Timed: the
    rounds end to end with their page bookkeeping, twice: chained on the device (the
    accepted lengths never leave it; the host takes pages ahead of an upper bound) and,
    for comparison, with the host reading the accepted lengths back after every round."""
    import numpy as np
    from paper_2606_26744_amd.decode import PagedDecoder
    wl = synth.drafter_full()
    dr = wl.drafter
    n_seq, B = wl.n_seq, wl.block
    T0 = int(wl.ctx_lens[0])
    max_ctx = T0 + (warmup + rounds + 1) * B
    w = synth.drafter_weights(wl, device="cuda")
    h = hdf.DrafterHandle(w, n_layers=dr.n_layers, d=dr.d, n_heads=dr.n_heads,
                          head_dim=dr.head_dim, d_ff=dr.d_ff, vocab=dr.vocab, eps=dr.eps,
                          rope_theta=dr.rope_theta, rope_max_pos=max_ctx + B)
    n_pages = n_seq * ((max_ctx + 63) // 64) + 8
    order = np.random.default_rng(wl.seed).permutation(n_pages)
    pre = T0 - wl.new_rows
    red = synth.reducer_inputs(wl, n_seq * B, device="cuda")
    V, p = dr.vocab, 0.8
    gen = torch.Generator(device="cuda").manual_seed(wl.seed)
    # The target's draws of every round, made before the timed rounds: whether it keeps
    # each draft (probability p), the token it has instead (uniform; equal to the draft
    # with probability 1/V) and the token after the block.
    n_rounds = 2 * (warmup + rounds)
    keep = torch.rand((n_rounds, n_seq, B - 1), generator=gen, device="cuda") < p
    other = torch.randint(0, V, (n_rounds, n_seq, B - 1), generator=gen, device="cuda",
                          dtype=torch.int32)
    tgt = torch.randint(0, V, (n_rounds, n_seq, B), generator=gen, device="cuda",
                        dtype=torch.int32)
    rnd = [0]

    def targets(drafts):
        r = rnd[0]
        rnd[0] += 1
        torch.where(keep[r], drafts, other[r], out=tgt[r, :, :B - 1])   # one kernel
        return tgt[r]

    def decoder():
        dec = PagedDecoder(h, n_seq, B, max_ctx, n_pages, n_seq * B, page_order=order)
        dec.preload(np.full(n_seq, pre, dtype=np.int64))     # the cached prefix of every sequence
        for s in range(n_seq):
            for l in range(dr.n_layers):
                k, v = synth.kv_prefix(wl, pre, l, device="cuda", sub=s)
                hdf.write_kv_rows_paged(dec.kv_k, dec.kv_vt, l, dec.pages[s], k, v)
                del k, v
        dec.set_anchors(synth.block_tokens(wl, device="cuda")[:, 0])
        return dec

    # host-synchronised rounds
    dec = decoder()
    counts = np.full(n_seq, wl.new_rows, dtype=np.int64)

    def one(counts):
        n_new = int(counts.sum())
        out = dec.round(red["H"][:n_new], counts, red["W_g"], red["b_g"], targets)
        return dec.next_counts(out["accept_len"])

    for _ in range(warmup):
        counts = one(counts)
    torch.cuda.synchronize()
    committed = 0
    t0 = time.perf_counter()
    for _ in range(rounds):
        counts = one(counts)
        committed += int(counts.sum())
    torch.cuda.synchronize()
    dt_sync = time.perf_counter() - t0
    sync_res = {"ms_per_round": round(dt_sync / rounds * 1e3, 4),
                "blocks_per_s": round(n_seq * rounds / dt_sync, 1),
                "committed_tokens_per_s": round(committed / dt_sync, 1),
                "mean_accept_len": round(committed / (rounds * n_seq) - 1, 3)}
    del dec
    gc.collect()
    torch.cuda.empty_cache()

    # chained rounds
    dec = decoder()
    dec.start_chain(np.full(n_seq, wl.new_rows, dtype=np.int64))
    H = red["H"][:n_seq * B]
    for _ in range(warmup):
        dec.chained_round(H, red["W_g"], red["b_g"], targets)
    torch.cuda.synchronize()
    c0 = dec.sync_lengths()
    t0 = time.perf_counter()
    for _ in range(rounds):
        dec.chained_round(H, red["W_g"], red["b_g"], targets)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    c1 = dec.sync_lengths()
    committed = int((c1 - c0).sum())
    res = {"n_seq": n_seq, "rounds": rounds, "mode": "chained on the device",
           "ms_per_round": round(dt / rounds * 1e3, 4),
           "blocks_per_s": round(n_seq * rounds / dt, 1),
           "committed_tokens_per_s": round(committed / dt, 1),
           "mean_accept_len": round(committed / (rounds * n_seq) - 1, 3),
           "context_end": [int(x) for x in c1], "pages_used": n_pages - dec.pool.free,
           "host_synchronised": sync_res}
    del dec, h, w, red
    gc.collect()
    torch.cuda.empty_cache()
    return res


def sampled_leg(torch, synth, hdf, wl, h, bufs, args, T, steps, warmup):
    """The full-size step at temperature T: the same step with the LM head's logits kept,
    a draw for every slot and speculative-sampling verification.  The target's logits are
    synthetic: the draft logits of an untimed step plus N(0, 0.5) noise."""
    from paper_2606_26744_amd.step import SampledStepBuffers, drafter_step_sampled
    n_seq, B, V = wl.n_seq, wl.block, h.V
    sb = SampledStepBuffers(h, n_seq, B)
    kw = {k: v for k, v in args.items()}
    tgt = torch.zeros((n_seq, B, V), dtype=torch.float32, device="cuda")
    out = drafter_step_sampled(h, bufs, sb, target_logits=tgt, temperature=T, **kw)
    g = torch.Generator(device="cuda").manual_seed(wl.seed)
    lg = out["logits"].view(n_seq, B, V)
    tgt[:, :B - 1] = lg[:, 1:] + 0.5 * torch.randn((n_seq, B - 1, V), generator=g, device="cuda")
    tgt[:, B - 1] = lg[:, 0]
    for r in range(warmup):
        drafter_step_sampled(h, bufs, sb, target_logits=tgt, temperature=T, round_id=r, **kw)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    accs = torch.empty((steps, n_seq), dtype=torch.int32, device="cuda")
    torch.cuda.synchronize()
    e0.record()
    for r in range(steps):
        out = drafter_step_sampled(h, bufs, sb, target_logits=tgt, temperature=T,
                                   round_id=warmup + r, **kw)
        accs[r].copy_(out["accept_len"])
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    acc = accs.float()
    res = {"temperature": T, "ms_per_step": round(ms, 4), "blocks_per_s": round(n_seq / (ms * 1e-3), 1),
           "steps": steps, "mean_accept_len": round(float(acc.mean()), 3)}
    del sb, tgt
    gc.collect()
    torch.cuda.empty_cache()
    return res


def kl_leg(torch, synth, hdf, wl, h):
    """hdf_kl_forward on the full-size blocks (8 x 16 slots, P = 2, vocabulary 129280):
    the teacher LM head over 16 pooled target states, the KL and cross-entropy passes.
    HIP events around 10 calls."""
    n, B, P, m, d, V = wl.n_seq, wl.block, 2, wl.m, wl.d, h.V
    H = synth.normal([n, P, m, d], 1.0, wl.seed, 80, device="cuda")
    g = torch.Generator(device="cuda").manual_seed(wl.seed)
    z = torch.randn((n * B, V), generator=g, device="cuda")
    lab = torch.randint(0, V, (n, B - 1), generator=g, device="cuda").to(torch.int32)
    ws = torch.empty(int(hdf.lib().hdf_kl_forward_workspace(n, B, P, d, V, hdf.HDF_BF16)),
                     dtype=torch.uint8, device="cuda")
    fn = lambda: hdf.kl_forward(H, h.w_lm, z, B=B, P=P, labels=lab, temperature=1.0, alpha=0.1,
                                ws=ws)
    for _ in range(2):
        fn()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(10):
        out = fn()
    e1.record()
    torch.cuda.synchronize()
    res = {"n_seq": n, "B": B, "P": P, "vocab": V, "us": round(e0.elapsed_time(e1) / 10 * 1e3, 1),
           "loss": [round(float(x), 4) for x in out[2].cpu()]}
    del H, z, lab, ws
    gc.collect()
    torch.cuda.empty_cache()
    return res


def fc_reducer_leg(torch, synth, hdf):
    """The generic fc reducer (a dense m*d -> d projection, 67M parameters at m = 4,
    d = 4096) beside the gated reducer on the same H: the full-size step's 128 new rows
    and the 65536 x 4 x 7168 stress shape.  HIP events around 10 calls each."""
    out = []
    for name, wl, n in (("drafter_full rows", synth.drafter_full(), 128),
                        ("reducer_stress", synth.reducer_stress(), None)):
        n = n or wl.n_tok
        ri = synth.reducer_inputs(wl, n, device="cuda")
        m, d = wl.m, wl.d
        W = synth.normal([d, m * d], wl.w_std, wl.seed, 73, dtype=wl.dtype, device="cuda")
        Wp = hdf.pack_weight(W)
        del W
        Y = torch.empty((n, d), dtype=torch.bfloat16, device="cuda")
        ws = torch.empty(max(int(hdf.lib().hdf_fc_reduce_workspace(n, m, d, hdf.HDF_BF16)), 1),
                         dtype=torch.uint8, device="cuda")
        row = {"case": name, "n_tok": n, "m": m, "d": d}
        for kind, fn in (("gated", lambda: hdf.hc_reduce(ri["H"], ri["W_g"], ri["b_g"], Y=Y)),
                         ("fc", lambda: hdf.fc_reduce(ri["H"], Wp, Y=Y, ws=ws))):
            for _ in range(2):
                fn()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record()
            for _ in range(10):
                fn()
            e1.record()
            torch.cuda.synchronize()
            row[kind + "_us"] = round(e0.elapsed_time(e1) / 10 * 1e3, 1)
        row["fc_params"] = m * d * d
        row["gated_params"] = m * m * d + m
        row["fc_TFLOP/s"] = round(2.0 * n * m * d * d / (row["fc_us"] * 1e-6) / 1e12, 1)
        out.append(row)
        del ri, Wp, Y, ws
        gc.collect()
        torch.cuda.empty_cache()
    return out


def blas_reference(torch):
    """torch.matmul (the vendor BLAS) on the matrix-core bound GEMM shapes of the drafter,
    with the bench's value distributions (activations N(0, 1), weights N(0, 0.02), bf16):
    what the library reaches on the same shapes and data, beside this path's own kernels."""
    shapes = [("lm_head", 1024, 4096, 129280), ("gate_up", 1024, 4096, 24576),
              ("down", 1024, 12288, 4096), ("qkv", 1024, 4096, 12288),
              ("ctx_kv_cold", 16384, 4096, 8192)]
    g = torch.Generator(device="cuda").manual_seed(7)
    out = []
    for name, M, K, N in shapes:
        a = torch.randn((M, K), generator=g, device="cuda").to(torch.bfloat16)
        w = (torch.randn((N, K), generator=g, device="cuda") * 0.02).to(torch.bfloat16)
        wt = w.t()
        for _ in range(3):
            c = torch.matmul(a, wt)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        n = 10
        torch.cuda.synchronize()
        e0.record()
        for _ in range(n):
            c = torch.matmul(a, wt)
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) / n * 1e3
        tf = 2.0 * M * N * K / (us * 1e-6) / 1e12
        out.append({"gemm": name, "M": M, "K": K, "N": N, "us": round(us, 1),
                    "TFLOP/s": round(tf, 1), "mfma_frac": round(tf / BF16_PEAK_TFLOPS, 4)})
        del a, w, wt, c
        gc.collect()
        torch.cuda.empty_cache()
    return out


def _kernel_source_sha():
    """Hash of the LM-head kernel's code (gemm.hip + common.hpp) with comments and
    blank space removed, so that the measured traffic stays attached to the code it was
    measured on and not to its comments."""
    import hashlib
    import re

    def code(path):
        text = open(path).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        text = re.sub(r"//[^\n]*", "", text)
        return "\n".join(l.strip() for l in text.splitlines() if l.strip())

    c = os.path.join(ROOT, "paper_2606_26744_amd", "csrc")
    data = code(os.path.join(c, "gemm.hip")) + "\n" + code(os.path.join(c, "common.hpp"))
    return hashlib.sha256(data.encode()).hexdigest()[:16]


def _blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        return len(os.sched_getaffinity(0))


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(torch, synth, wl, h, w, red, args, offs, seqs=None, budget_s=10.0):
    """The oracle as it stands on the whole step of sequences `seqs` (default: all of
    them), blocks/s; the same inputs the GPU step took, the cached rows read back from
    the GPU's cache.  Repeats for about budget_s seconds (at least twice), median."""
    import numpy as np
    from oracle.accept import accept
    from oracle.drafter import Weights, draft_block
    from oracle.lm_head import lm_head_argmax
    from oracle.reducer import hc_reduce
    dr = wl.drafter
    b = synth.to_numpy_bits
    B = wl.block
    seqs = list(range(wl.n_seq)) if seqs is None else list(seqs)
    lens = [int(t) for t in wl.ctx_lens]
    news = lens if wl.cold else [wl.new_rows] * wl.n_seq
    no = np.concatenate([[0], np.cumsum(news)])
    wb = {k: ([b(x) for x in v] if isinstance(v, list) else b(v)) for k, v in w.items()}
    W = Weights(wb, d=dr.d, n_layers=dr.n_layers, n_heads=dr.n_heads, head_dim=dr.head_dim,
                d_ff=dr.d_ff, vocab=dr.vocab, eps=dr.eps, rope_theta=dr.rope_theta, dtype="bf16")
    from paper_2606_26744_amd import hdf
    pre = []
    for s in seqs:
        t0 = lens[s] - news[s]
        per = []
        for l in range(dr.n_layers):
            k, v = hdf.read_kv_rows(args["kv_k"], args["kv_vt"], l, offs[s], t0)
            per.append((b(k), b(v)))
        pre.append(per)
    H = [b(red["H"][int(no[s]):int(no[s + 1])]) for s in seqs]
    Wg, bg = b(red["W_g"]), b(red["b_g"])
    toks = b(args["tokens"])[seqs]
    p = [wl.match_p[s] for s in seqs]
    times = []
    t_total = 0.0
    while len(times) < 2 or (t_total < budget_s and len(times) < 20):
        t_start = time.perf_counter()
        ys = [hc_reduce(Hs, Wg, bg, dtype="bf16")[0] for Hs in H]
        hid = draft_block(W, ys, toks, kv_prefix=pre)
        am, _, _ = lm_head_argmax(hid, W.w_lm)
        drafts = am.reshape(len(seqs), B)[:, 1:]
        tg = synth.make_targets(drafts, p, dr.vocab, seed=wl.seed)
        accept(drafts, tg)
        times.append(time.perf_counter() - t_start)
        t_total += times[-1]
    t = statistics.median(times)
    ctx = ("every context row reduced and projected" if wl.cold
           else f"{news[seqs[0]]} new context rows each reduced and projected")
    return {"value": round(len(seqs) / t, 4), "unit": "blocks/s", "cores": int(_blas_threads()),
            "kind": "oracle",
            "sample": f"{wl.name}: the whole step of {len(seqs)} of its {wl.n_seq} sequences "
                      f"(contexts {[lens[s] for s in seqs]}, {ctx}, B={B}, full-vocabulary "
                      f"argmax, acceptance); median of {len(times)} runs ({t_total:.1f} s in "
                      f"total), {t:.2f} s per step; float64 NumPy; host CPU {_cpu_model()}; "
                      f"affinity {len(os.sched_getaffinity(0))} cores"}


def cpu_reducer_baseline(synth, sw, ri, n_sample=2048):
    """The oracle's gated reducer (Eq. 1, float64 NumPy) on n_sample tokens of the stress
    shape, with every BLAS thread and with one, as GB/s of the reducer's algorithmic
    bytes (the same unit as the GPU figure)."""
    from oracle.reducer import hc_reduce
    b = synth.to_numpy_bits
    H = b(ri["H"][:n_sample])
    Wg, bg = b(ri["W_g"]), b(ri["b_g"])
    nbytes = n_sample * sw.m * sw.d * 2 + n_sample * sw.d * 2
    out = {}

    def timed():
        ts = []
        for _ in range(3):
            t0 = time.perf_counter()
            hc_reduce(H, Wg, bg, dtype="bf16")
            ts.append(time.perf_counter() - t0)
        return statistics.median(ts)

    t_all = timed()
    out["all_cores"] = {"value": round(nbytes / t_all / 1e9, 3), "unit": "GB/s",
                        "cores": int(_blas_threads()), "kind": "oracle",
                        "sample": f"{n_sample} of the {sw.n_tok} tokens x {sw.m} x {sw.d}, "
                                  f"median of 3, {t_all * 1e3:.0f} ms each; host CPU "
                                  f"{_cpu_model()}"}
    try:
        from threadpoolctl import threadpool_limits
        with threadpool_limits(1):
            t_one = timed()
        out["single_thread"] = {"value": round(nbytes / t_one / 1e9, 3), "unit": "GB/s",
                                "cores": 1, "kind": "oracle",
                                "sample": f"same sample, BLAS limited to one thread, "
                                          f"{t_one * 1e3:.0f} ms each"}
    except Exception as e:  # pragma: no cover
        out["single_thread"] = {"error": str(e)}
    return out


def rw_probe(torch, sw, ri, Y):
    """The memory-system probe (libhdf_probe.so): the reducer's exact traffic with no
    arithmetic, read-only and with the 4:1 writes, each the best of the one- and
    two-token ring depths; GB/s of the bytes moved."""
    import ctypes
    path = os.path.join(ROOT, "paper_2606_26744_amd", "libhdf_probe.so")
    if not os.path.exists(path):
        return {"error": "libhdf_probe.so not built"}
    L = ctypes.CDLL(path)
    L.hdf_probe_rw.restype = ctypes.c_int
    L.hdf_probe_rw.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int,
                               ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                               ctypes.c_void_p, ctypes.c_void_p]
    sink = torch.zeros(4, dtype=torch.int32, device="cuda")
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    grid = torch.cuda.get_device_properties(0).multi_processor_count
    H, n, m, d = ri["H"], sw.n_tok, sw.m, sw.d
    res = {}
    for write in (0, 1):
        best = 0.0
        for pf in (1, 2):
            def go():
                rc = L.hdf_probe_rw(ctypes.c_void_p(H.data_ptr()), ctypes.c_void_p(Y.data_ptr()),
                                    n, m, d, write, pf, grid, ctypes.c_void_p(sink.data_ptr()), st)
                if rc != 0:
                    raise RuntimeError(f"hdf_probe_rw returned {rc}")
            for _ in range(5):
                go()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record()
            for _ in range(20):
                go()
            e1.record()
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) / 20 * 1e3
            nbytes = n * m * d * 2 + (n * d * 2 if write else 0)
            best = max(best, nbytes / (us * 1e-6) / 1e9)
        res["read_4to1_GB/s" if write else "read_only_GB/s"] = round(best, 1)
    return res


def mfma_probe(torch):
    """The matrix-core probe (libhdf_probe.so): back-to-back v_mfma_f32_32x32x16_bf16 from
    registers on every SIMD, four waves per SIMD and four accumulator chains per wave, on
    random operands, no memory traffic: the rate the matrix-core bound kernels can reach
    at the clock the chip holds under that load (with near-constant operands it holds a
    higher one: 2.45 PFLOP/s measured, against 1.7-1.8 on random data)."""
    import ctypes
    path = os.path.join(ROOT, "paper_2606_26744_amd", "libhdf_probe.so")
    if not os.path.exists(path):
        return {"error": "libhdf_probe.so not built"}
    L = ctypes.CDLL(path)
    L.hdf_probe_mfma.restype = ctypes.c_int
    L.hdf_probe_mfma.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    blocks = 4 * torch.cuda.get_device_properties(0).multi_processor_count
    sink = torch.zeros(blocks, dtype=torch.float32, device="cuda")
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    iters = 20000

    def go():
        rc = L.hdf_probe_mfma(blocks, iters, ctypes.c_void_p(sink.data_ptr()), st)
        if rc != 0:
            raise RuntimeError(f"hdf_probe_mfma returned {rc}")
    for _ in range(3):    # about 18 ms: the clock settles under the load first
        go()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(3):
        go()
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) / 3 * 1e3
    tf = blocks * 4 * 4 * iters * 32768.0 / (us * 1e-6) / 1e12
    return {"TFLOP/s": round(tf, 1), "frac_of_peak": round(tf / BF16_PEAK_TFLOPS, 4),
            "us": round(us, 1)}


def cold_cache_step(torch, h, bufs, args, tg, steps):
    """The headline step with the caches flushed before every step: a 512 MiB device copy
    (1 GiB of traffic, well above the 256 MB last-level cache and the L2s) runs ahead of
    each step, and each step is timed by its own events, so no step finds the previous
    one's weights in a cache."""
    from paper_2606_26744_amd.step import drafter_step
    src = torch.empty(1 << 29, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    for i in range(steps):
        dst.copy_(src)
        ev[i][0].record()
        drafter_step(h, bufs, targets=tg, **args)
        ev[i][1].record()
    torch.cuda.synchronize()
    ms = statistics.mean(a.elapsed_time(b) for a, b in ev)
    del src, dst
    gc.collect()
    torch.cuda.empty_cache()
    return {"ms_per_step": round(ms, 4), "steps": steps,
            "flush": "512 MiB device copy before every step"}


def timed_steps(torch, h, bufs, args, tg, steps, warmup):
    """W untimed warm-up steps, then K steps timed between synchronisations.  Inside the
    timed region only the LM head (the roofline kernel) is bracketed by events, on the
    stream its kernels run on, in every LM_SAMPLE-th step: each recorded event leaves the
    GPU idle for about 3 us (a kernel trace shows the gap at every record), so bracketing
    every step would add about 6 us to each timed step.  Returns (ms per step, mean LM-head
    us, LM-head launches timed, the last step's outputs)."""
    from paper_2606_26744_amd.step import drafter_step
    for _ in range(warmup):
        drafter_step(h, bufs, targets=tg, **args)
    ev = lambda: torch.cuda.Event(enable_timing=True)
    LM_SAMPLE = 4
    lm_marks = [[None, None, ev(), ev(), None] if i % LM_SAMPLE == 0 else None
                for i in range(steps)]
    t_start, t_end = ev(), ev()
    torch.cuda.synchronize()
    t_start.record()
    for i in range(steps):
        out = drafter_step(h, bufs, targets=tg, marks=lm_marks[i], **args)
    t_end.record()
    torch.cuda.synchronize()
    sampled = [m for m in lm_marks if m is not None]
    lm_us = statistics.mean(m[2].elapsed_time(m[3]) * 1e3 for m in sampled)
    return t_start.elapsed_time(t_end) / steps, lm_us, len(sampled), out


def main():
    a = parse()
    if a.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {a.gpus}); the drafter step "
              f"shards by sequence with no exchange, so run one process per GPU.", file=sys.stderr)
        sys.exit(2)
    import torch
    import synth
    from paper_2606_26744_amd import hdf
    from paper_2606_26744_amd.step import drafter_step
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    hdf.lib()
    wl, h, bufs, args, red, w, offs = build_workload(torch, synth, hdf)
    n_seq, B = wl.n_seq, wl.block
    # Python's cyclic garbage collector stays paused from here on (collected now and where
    # a leg frees its workload): a full pass over this process's heap takes tens of
    # milliseconds, and a pass inside a timed loop leaves the GPU idle while the host is
    # not enqueuing (a 20-step run once measured 4.0 ms a step for 0.38 ms of work).
    gc.collect()
    gc.disable()
    # Targets: copies of the drafts with probability 0.8 per position (drafts from one
    # untimed step), so acceptance lengths are geometric as in the workload description.
    tg = step_targets(torch, synth, hdf, wl, h, bufs, args)
    # The same W + K steps twice.  First on a GPU fresh from idle: its power management
    # raises the clocks over about 25 ms of load (successive 20-step windows measure
    # 0.41, 0.38, 0.37 ms, then 0.369 ms; 50 ms of idle drops them again), so that run
    # mostly measures the ramp.  The headline run follows it with no idle gap, on a GPU
    # that has been serving steps.
    idle = timed_steps(torch, h, bufs, args, tg, a.steps, a.warmup)
    ms, lm_head_us, n_lm, out = timed_steps(torch, h, bufs, args, tg, a.steps, a.warmup)
    ev = lambda: torch.cuda.Event(enable_timing=True)
    # Per-stage breakdown from a further, untimed pass with events between all stages
    # (medians: a host-side pause inside one step shows in that step's intervals only).
    marks = [[ev() for _ in range(5)] for _ in range(a.steps)]
    for i in range(a.steps):
        drafter_step(h, bufs, targets=tg, marks=marks[i], **args)
    torch.cuda.synchronize()
    names = ["reduce", "draft_block", "lm_head_argmax", "accept"]
    stage_us = {n: statistics.median(m[j].elapsed_time(m[j + 1]) * 1e3 for m in marks)
                for j, n in enumerate(names)}
    cold = None if a.no_cold_cache else cold_cache_step(torch, h, bufs, args, tg, a.steps)
    sweep = None if a.no_m_sweep else lm_head_m_sweep(torch, synth, hdf, h, wl.d)
    acc = out["accept_len"].cpu().numpy()
    # LM head roofline: algorithmic bytes of one hdf_lm_head_argmax_keys call, the LM-head
    # GEMM (weights + hidden states + the per-row argmax keys it leaves).
    d, V, M = wl.d, wl.drafter.vocab, n_seq * B
    lm_bytes = V * d * 2 + M * d * 2 + M * 8
    lm_us = lm_head_us
    lm_gbs = lm_bytes / (lm_us * 1e-6) / 1e9
    lm_tflops = 2.0 * M * d * V / (lm_us * 1e-6) / 1e12
    res = {
        "metric": METRIC, "value": round(n_seq / (ms * 1e-3), 1), "unit": "blocks/s",
        "n_gpus": 1, "steps": a.steps, "warmup": a.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded; random-init weights of the drafter shape)",
        "config": {"workload": "drafter_full_warm", "n_seq": n_seq, "context": wl.ctx_lens[0],
                   "new_rows_per_seq": wl.new_rows, "d": d, "heads": wl.drafter.n_heads,
                   "head_dim": wl.drafter.head_dim, "d_ff": wl.drafter.d_ff, "vocab": V,
                   "block": B, "m_paths": wl.m, "layers": wl.drafter.n_layers,
                   "parallelism": "single GPU"},
        "stages_us": {k: round(v, 2) for k, v in stage_us.items()},
        "roofline": {"kernel": "lm_head_argmax", "bound": "hbm", "achieved": round(lm_gbs, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(lm_gbs / HBM_PEAK_GBS, 4),
                     "traffic": (round(LM_HEAD_TRAFFIC["bytes"])
                                 if _kernel_source_sha() == LM_HEAD_TRAFFIC["source_sha"] else None),
                     "bytes_per_launch": lm_bytes,
                     "timed_launches": n_lm,
                     "mfma_tflops": round(lm_tflops, 1),
                     "mfma_frac": round(lm_tflops / BF16_PEAK_TFLOPS, 4)},
        "mean_accept_len": float(acc.mean()), "tau": float(acc.mean() + 1),
        "from_idle": {"ms_per_step": round(idle[0], 4),
                      "blocks_per_s": round(n_seq / (idle[0] * 1e-3), 1),
                      "lm_head_us": round(idle[1], 1),
                      "note": "the same W + K steps, run first, on a GPU fresh from idle"},
    }
    if sweep is not None:
        res["lm_head_m_sweep"] = sweep
        probe = mfma_probe(torch)
        res["mfma_probe"] = probe
        if "TFLOP/s" in probe:
            for e in sweep:
                e["frac_of_mfma_probe"] = round(e["TFLOP/s"] / probe["TFLOP/s"], 4)
    if cold is not None:
        res["cold_cache_step"] = cold
        cold["blocks_per_s"] = round(n_seq / (cold["ms_per_step"] * 1e-3), 1)
    if not a.no_reducer_stress:
        sw = synth.reducer_stress()
        ri = synth.reducer_inputs(sw, sw.n_tok, device="cuda")
        Y = torch.empty((sw.n_tok, sw.d), dtype=torch.bfloat16, device="cuda")
        # 30 untimed launches first: under sustained load the GPU needs about 20 ms to
        # reach its steady memory throughput (the first 20 launches run about 10% slower)
        for _ in range(30):
            hdf.hc_reduce(ri["H"], ri["W_g"], ri["b_g"], Y=Y)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        n_it = 20
        for _ in range(n_it):
            hdf.hc_reduce(ri["H"], ri["W_g"], ri["b_g"], Y=Y)
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) / n_it * 1e3
        rb = sw.n_tok * sw.m * sw.d * 2 + sw.n_tok * sw.d * 2 + sw.m * sw.m * sw.d * 2
        gbs = rb / (us * 1e-6) / 1e9
        res["reducer_stress"] = {"n_tok": sw.n_tok, "m": sw.m, "d": sw.d, "us": round(us, 1),
                                 "GB/s": round(gbs, 1),
                                 "frac_hbm": round(gbs / HBM_PEAK_GBS, 4),
                                 "bytes_per_launch": rb}
        pr = rw_probe(torch, sw, ri, Y)
        res["reducer_stress"]["probe"] = pr
        if "read_4to1_GB/s" in pr:
            res["reducer_stress"]["frac_of_probe_4to1"] = round(gbs / pr["read_4to1_GB/s"], 4)
        if not a.no_cpu_baseline:
            res["reducer_stress"]["cpu_baseline"] = cpu_reducer_baseline(synth, sw, ri)
        del ri, Y
        gc.collect()
        torch.cuda.empty_cache()
    if a.copy_probe:
        x = torch.empty(1 << 31, dtype=torch.uint8, device="cuda")
        y = torch.empty_like(x)
        for _ in range(5):
            y.copy_(x)
        torch.cuda.synchronize()
        del x, y
    if not a.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(torch, synth, wl, h, w, red, args, offs)
    if a.temperature > 0:
        res["sampled_step"] = sampled_leg(torch, synth, hdf, wl, h, bufs, args, a.temperature,
                                          a.steps, 3)
    if a.kl:
        res["kl_forward"] = kl_leg(torch, synth, hdf, wl, h)
    if a.fc_reducer:
        res["fc_reducer"] = fc_reducer_leg(torch, synth, hdf)
    if a.blas_ref:
        res["blas_reference"] = blas_reference(torch)
        if "TFLOP/s" in res.get("mfma_probe", {}):
            for e in res["blas_reference"]:
                e["frac_of_mfma_probe"] = round(e["TFLOP/s"] / res["mfma_probe"]["TFLOP/s"], 4)
    if not a.no_ragged or a.cold or a.ragged_cold or a.decode:
        del bufs, args
        gc.collect()
        torch.cuda.empty_cache()
    if not a.no_ragged:
        res["ragged_decode"] = ragged_leg(torch, synth, hdf, max(a.steps // 5, 5), 3,
                                          cpu_seqs=None if a.no_cpu_baseline else [0, 1])
    if a.ragged_cold:
        res["ragged_decode_cold"] = ragged_leg(torch, synth, hdf, 3, 1, synth.ragged_decode_cold())
    if a.cold:
        res["drafter_full_cold"] = ragged_leg(torch, synth, hdf, max(a.steps // 5, 5), 3,
                                              synth.drafter_full_cold())
    if a.decode:
        res["paged_decode"] = decode_leg(torch, synth, hdf, a.decode, 5)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
