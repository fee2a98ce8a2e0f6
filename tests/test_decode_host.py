"""Host bookkeeping of the paged decode loop (no GPU): the page allocator."""
import pytest

from paper_2606_26744_amd.decode import PagePool


def test_page_pool_order_and_reuse():
    pool = PagePool(4, order=[2, 0, 3, 1])
    assert [pool.take() for _ in range(3)] == [2, 0, 3]
    assert pool.free == 1
    pool.release([0])
    assert pool.take() == 0 and pool.take() == 1
    with pytest.raises(MemoryError):
        pool.take()


def test_page_pool_rejects_bad_order():
    with pytest.raises(ValueError):
        PagePool(3, order=[0, 0, 1])


def test_lengths_past_max_ctx_are_rejected():
    """A context may fill its last page only up to max_ctx: the drafter call is launched
    with max_ctx, which sizes the RoPE table, so the host bound is max_ctx itself and not
    the page capacity (max_pages * 64)."""
    import numpy as np
    from paper_2606_26744_amd.decode import pages_for
    assert pages_for([0, 1, 64, 65, 100], 100).tolist() == [0, 1, 1, 2, 2]
    with pytest.raises(ValueError, match="sequence 1 outgrows max_ctx=100"):
        pages_for(np.array([100, 101]), 100)   # 101 still fits two pages of 64


class _NoWait:
    def synchronize(self):
        pass


def _host_only_decoder(max_ctx, n_seq=2):
    """The decoder's host bookkeeping without device buffers (the bound checks run before
    anything is copied to the device)."""
    import numpy as np
    from paper_2606_26744_amd.decode import PagedDecoder
    dec = PagedDecoder.__new__(PagedDecoder)
    dec.n_seq, dec.B, dec.max_ctx = n_seq, 16, max_ctx
    dec.max_pages = (max_ctx + 63) // 64
    dec.pool = PagePool(n_seq * dec.max_pages)
    dec.pages = [[] for _ in range(n_seq)]
    dec.ctx = np.zeros(n_seq, dtype=np.int64)
    dec._pt_host = np.full((n_seq, dec.max_pages), -1, dtype=np.int32)
    dec._copied = _NoWait()
    dec._rb_pending = []
    dec._rounds = 0
    return dec


def test_decoder_grow_stops_at_max_ctx():
    import numpy as np
    dec = _host_only_decoder(100)
    with pytest.raises(ValueError, match="outgrows max_ctx=100"):
        dec._grow(np.array([10, 101]))
    assert dec.pages == [[], []] and dec.pool.free == 4   # nothing taken


def test_chained_bound_stops_at_max_ctx():
    """Chained rounds raise the host's upper bound by B a round; once it passes max_ctx
    (and no read-back can tighten it) the next round is refused, although the last page
    would still hold the rows."""
    import numpy as np
    dec = _host_only_decoder(100)
    dec._ctx_hi = np.array([90, 101], dtype=np.int64)
    with pytest.raises(ValueError, match="sequence 1 outgrows max_ctx=100"):
        dec._reserve()
    assert dec.pages == [[], []]
