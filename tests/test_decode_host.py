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
