"""GPU parity of hdf_draft_block (the one-pass block drafter) against the CPU oracle:
final-normed block states and the KV-cache rows it writes."""
import numpy as np
import pytest
import torch

import synth
from oracle.drafter import context_kv, draft_block as ref_draft
from oracle.numerics import as_f64
from paper_2606_26744_amd import hdf
from tests._case import DraftCase, bits
from tests._tol import assert_bf16_state_close, assert_f32_rows_close

pytestmark = pytest.mark.gpu


def _compare(case, seqs=None, check_cache=True):
    print(f"[draft_block] {case.wl.name} dtype={case.wl.dtype} ctx={case.ctx[:6]} "
          f"new={case.new[:6]} B={case.B} seqs={seqs}", flush=True)
    hidden = case.run()
    torch.cuda.synchronize()
    W = case.oracle_weights()
    ys, toks = case.oracle_inputs()
    seqs = list(range(len(case.ctx))) if seqs is None else list(seqs)
    ref = ref_draft(W, ys, toks, kv_prefix=case.prefix, seqs=seqs)
    B = case.B
    got = np.concatenate([bits(hidden[s * B:(s + 1) * B]) for s in seqs])
    if case.wl.dtype == "bf16":
        flips, worst = assert_bf16_state_close(as_f64(got), ref, "hidden")
        print(f"  hidden: {flips} of {ref.size} elements differ; worst row RMS rel {worst:.2e}",
              flush=True)
    else:
        assert_f32_rows_close(got, ref, "hidden")
    if check_cache:
        dr = case.wl.drafter
        for s in seqs[:3]:
            T, n = case.ctx[s], case.new[s]
            if n == 0:
                continue
            kv = context_kv(W, as_f64(case.y_rows(s)), np.arange(T - n, T))
            for l in range(dr.n_layers):
                kk, vv = case.read_cache(s, l)
                k, v = kk[T - n:], vv[T - n:]
                if case.wl.dtype == "bf16":
                    assert_bf16_state_close(as_f64(bits(k.contiguous())), kv[l][0], "cache K")
                    assert_bf16_state_close(as_f64(bits(v.contiguous())), kv[l][1], "cache V")
                else:
                    assert_f32_rows_close(k.cpu().numpy(), kv[l][0], "cache K")
                    assert_f32_rows_close(v.cpu().numpy(), kv[l][1], "cache V")
    return hidden


def test_tiny_fp32_cold():
    wl = synth.tiny_fp32()
    _compare(DraftCase(wl, [64], [64]))


def test_small_bf16_cold_and_warm():
    wl = synth.small_bf16()
    _compare(DraftCase(wl, [512] * 4, [512] * 4))
    _compare(DraftCase(wl, [512] * 4, [16] * 4, sub=1))


def test_ragged_lengths_and_two_query_groups():
    wl = synth.small_bf16()
    ctx = [1, 63, 64, 65, 200, 513, 1030]
    new = [1, 5, 64, 16, 0, 513, 7]
    _compare(DraftCase(wl, ctx, new, B=20, sub=2))


def test_block_of_one():
    wl = synth.small_bf16()
    _compare(DraftCase(wl, [100, 7], [100, 7], B=1, sub=3))


def test_largest_block_and_ragged_query_groups():
    """B = 64, the largest block (four 16-query groups; the block's key tile is all valid
    keys), and B = 33 (a last query group of one query), at head dims 64 and 128."""
    wl = synth.small_bf16()
    _compare(DraftCase(wl, [200, 70], [30, 70], B=64, sub=31))
    _compare(DraftCase(wl, [129, 1, 600], [129, 1, 16], B=33, sub=32))
    wl.drafter = synth.DrafterShape(d=512, n_layers=1, n_heads=4, head_dim=128, d_ff=1024,
                                    vocab=1000)
    wl.d = 512
    _compare(DraftCase(wl, [300, 64], [40, 64], B=64, sub=33))


def test_head_dim_128_and_loose_max_ctx():
    wl = synth.small_bf16()
    wl.drafter = synth.DrafterShape(d=512, n_layers=1, n_heads=4, head_dim=128, d_ff=1024,
                                    vocab=1000)
    wl.d = 512
    _compare(DraftCase(wl, [300, 1500, 64], [20, 1500, 64], sub=4, max_ctx=3000))


def test_many_sequences_attention_chunks():
    """More (sequence, head) pairs than the 256 CUs: the attention takes several chunks
    per sequence merged by the combine kernel (contexts up to 1100), then one chunk per
    sequence written directly (contexts up to 500, one of them empty)."""
    wl = synth.small_bf16()
    rng = np.random.default_rng(17)
    ctx = [int(x) for x in rng.integers(1, 1100, size=20)]
    _compare(DraftCase(wl, ctx, [min(c, 16) for c in ctx], sub=12), seqs=[0, 7, 19])
    ctx = [int(x) for x in rng.integers(1, 500, size=20)]
    ctx[5] = 0
    _compare(DraftCase(wl, ctx, [min(c, 16) for c in ctx], sub=13), seqs=[3, 5, 11])


def test_longest_first_dispatch_every_sequence():
    """40 sequences x 16 heads in 512-key chunks (1920 attention workgroups, more than two
    rounds): each workgroup slot takes the sequence of its rank by context length, ties by
    index.  Lengths with ties and an empty context; every sequence against the oracle."""
    wl = synth.small_bf16()
    rng = np.random.default_rng(41)
    ctx = [int(x) for x in rng.integers(1, 600, size=40)]
    ctx[3] = ctx[17] = ctx[29] = 333          # equal lengths: ranked by sequence index
    ctx[8] = 0
    _compare(DraftCase(wl, ctx, [min(c, 16) for c in ctx], sub=19))


def test_longest_first_dispatch_several_query_groups():
    """The same ranking with B = 33: three 16-query groups per sequence slot (the last
    holds one query), and every group's workgroup must take the slot's sequence.  Ties, an
    empty context; every sequence against the oracle."""
    wl = synth.small_bf16()
    rng = np.random.default_rng(43)
    ctx = [int(x) for x in rng.integers(1, 600, size=40)]
    ctx[2] = ctx[21] = ctx[30] = 250
    ctx[11] = 0
    _compare(DraftCase(wl, ctx, [min(c, 33) for c in ctx], B=33, sub=20))


def test_many_sequences_attention_chunks_head_dim_128():
    wl = synth.small_bf16()
    wl.drafter = synth.DrafterShape(d=1024, n_layers=1, n_heads=8, head_dim=128, d_ff=2048,
                                    vocab=1000)
    rng = np.random.default_rng(18)
    ctx = [int(x) for x in rng.integers(1, 1500, size=40)]
    _compare(DraftCase(wl, ctx, [min(c, 16) for c in ctx], sub=14, paged=True, spare_pages=7),
             seqs=[2, 30])


def test_fused_epilogue_several_rounds():
    """Warm steps with up to 128 projected rows and B <= 16, so the projection epilogue runs
    inside the attention kernel, in several 16-row rounds for the longer sequences (70, 33
    and 17 new rows): every new cache row and the block states against the oracle, at head
    dims 64 and 128, contiguous and paged."""
    wl = synth.small_bf16()
    _compare(DraftCase(wl, [300, 90, 45], [70, 33, 17], sub=21))
    _compare(DraftCase(wl, [300, 90, 45], [70, 33, 17], sub=22, paged=True, spare_pages=3))
    wl.drafter = synth.DrafterShape(d=512, n_layers=1, n_heads=4, head_dim=128, d_ff=1024,
                                    vocab=1000)
    wl.d = 512
    _compare(DraftCase(wl, [200, 129, 40], [80, 29, 19], sub=23))


def test_no_rope_fp32_multilayer():
    wl = synth.tiny_fp32()
    wl.drafter = synth.DrafterShape(d=256, n_layers=3, n_heads=4, head_dim=64, d_ff=512,
                                    vocab=500)
    _compare(DraftCase(wl, [40, 9], [10, 9], rope=False, sub=5))


def test_full_size_warm_sampled():
    """Full-size warm step: 8 sequences x 2048 context, 16 new rows each; the oracle
    evaluates two sequences."""
    wl = synth.drafter_full()
    case = DraftCase(wl, [2048] * 8, [16] * 8, random_norms=False)
    _compare(case, seqs=[0, 5])
    del case
    torch.cuda.empty_cache()


def test_full_size_cold_sampled():
    """Full-size cold step: every one of the 8 x 2048 context rows is projected in the call
    (a 16384-row context projection on the matrix cores, grouped with the block's QKV);
    the oracle evaluates one sequence and all 2048 of its cache rows."""
    wl = synth.drafter_full()
    case = DraftCase(wl, [2048] * 8, [2048] * 8, random_norms=False, sub=8)
    _compare(case, seqs=[6])
    del case
    torch.cuda.empty_cache()


def test_ragged_long_contexts_sampled():
    wl = synth.ragged_decode()
    ctx = [1024, 16384, 5000, 777 + 1024]
    case = DraftCase(wl, ctx, [16] * 4, random_norms=False, sub=6, max_ctx=16384)
    _compare(case, seqs=[1, 3])
    del case
    torch.cuda.empty_cache()


def test_long_cold_contexts_across_projection_chunks():
    """Full-size drafter, three cold sequences of 13000, 9000 and 700 positions: 22700
    context rows projected in one call, in two chunks of the context projection (16384
    rows, then 6316), the chunk boundary inside sequence 1.  Sampled cache rows of every
    sequence (each boundary, the chunk boundary and random rows), read back through
    hdf_kv_read_rows, against oracle.context_kv of the same reduced rows."""
    wl = synth.drafter_full()
    ctx = [13000, 9000, 700]
    print(f"[cold chunks] drafter_full contexts {ctx}", flush=True)
    case = DraftCase(wl, ctx, ctx, random_norms=False, sub=17)
    case.run()
    torch.cuda.synchronize()
    W = case.oracle_weights()
    offs = case.kv_offsets.tolist()
    rng = np.random.default_rng(17)
    chunk_row = 16384 - ctx[0]            # local row of sequence 1 where the second chunk starts
    for s, T in enumerate(ctx):
        pick = {0, 1, 63, 64, T - 2, T - 1}
        if s == 1:
            pick |= {chunk_row - 1, chunk_row, chunk_row + 1}
        pick |= set(rng.choice(T, 120, replace=False).tolist())
        rows = np.array(sorted(r for r in pick if 0 <= r < T))
        ys = case.y_rows(s)[rows]
        ref = context_kv(W, as_f64(ys), rows)
        k, v = hdf.kv_read_rows(case.kv_k, case.kv_vt, 0, len(rows),
                                rows=torch.as_tensor(offs[s] + rows, dtype=torch.int32).cuda())
        assert_bf16_state_close(as_f64(bits(k)), ref[0][0], f"K seq {s}")
        assert_bf16_state_close(as_f64(bits(v)), ref[0][1], f"V seq {s}")
    del case
    torch.cuda.empty_cache()


def test_cold_rows_projected_into_the_cache_by_the_gemm_epilogue():
    """8192 cold context rows at head_dim 64 over a paged pool: one K split, so RoPE and
    the cache stores happen in the projection GEMM's epilogue (no fp32 rows in memory)."""
    wl = synth.small_bf16()
    case = DraftCase(wl, [4096, 4096], [4096, 4096], sub=15, paged=True, spare_pages=3)
    _compare(case, seqs=[1])
    del case
    torch.cuda.empty_cache()


def test_device_row_counts_through_the_gemm_epilogue():
    """Device row counts on 8192 rows (4096 per sequence, 3000 and 1 of them new): the
    cold rows go through the projection GEMM's K/V epilogue, the rows past each count are
    neither stored nor used (the oracle sees only the new rows), and every cache row past
    a sequence's context keeps what it held."""
    wl = synth.small_bf16()
    case = DraftCase(wl, [3050, 701], [3000, 1], sub=16, paged=True, spare_pages=2, stride=4096)
    dr = wl.drafter

    def tails():
        out = []
        for s, T in enumerate(case.ctx):
            n_rows = len(case.pages[s]) * 64
            for l in range(dr.n_layers):
                kk, vv = hdf.read_kv_rows_paged(case.kv_k, case.kv_vt, l, case.pages[s], n_rows)
                out.append((bits(kk[T:].contiguous()), bits(vv[T:].contiguous())))
        return out
    before = tails()
    _compare(case, seqs=[0, 1])
    for (kb, vb), (ka, va) in zip(before, tails()):
        assert np.array_equal(kb, ka) and np.array_equal(vb, va)
    del case
    torch.cuda.empty_cache()


def test_paged_cache_scattered_pages():
    """Paged cache: every sequence's 64-row tiles sit at random pages of a shared pool
    (with spare pages in between); warm and cold rows, ragged lengths, one and two
    query groups."""
    wl = synth.small_bf16()
    ctx = [1, 63, 64, 65, 200, 513, 1030]
    new = [1, 5, 64, 16, 0, 513, 7]
    _compare(DraftCase(wl, ctx, new, B=20, sub=9, paged=True, spare_pages=11))


def test_paged_cache_fp32_multilayer():
    wl = synth.tiny_fp32()
    wl.drafter = synth.DrafterShape(d=256, n_layers=2, n_heads=4, head_dim=64, d_ff=512,
                                    vocab=500)
    _compare(DraftCase(wl, [130, 9, 64], [10, 9, 64], sub=10, paged=True, spare_pages=3))


def test_paged_matches_contiguous_full_size():
    """The full-size warm step over a paged pool gives bit-identical block states to the
    contiguous cache with the same rows (same kernels, only the tile addresses differ)."""
    wl = synth.drafter_full()
    a = DraftCase(wl, [2048] * 8, [16] * 8, random_norms=False, sub=11)
    ha = a.run().clone()
    del a
    b = DraftCase(wl, [2048] * 8, [16] * 8, random_norms=False, sub=11, paged=True,
                  spare_pages=5)
    hb = b.run().clone()
    del b
    torch.cuda.empty_cache()
    assert torch.equal(ha, hb)


def test_determinism():
    wl = synth.small_bf16()
    case = DraftCase(wl, [700, 300], [16, 300], sub=7)
    h1 = case.run().clone()
    h2 = case.run().clone()
    assert torch.equal(h1, h2)
