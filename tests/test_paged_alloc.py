"""Host-side page bookkeeping of the paged KV cache (no GPU): pages cover
every position a slot holds, no page belongs to two slots or to a slot and
the free list at once, rollback and release return pages, and a request
that does not fit fails without changing anything."""

import numpy as np
import pytest

from paper_2408_00539_amd.paged import PageAllocator, PoolExhausted


def _check_invariants(a):
    owned = [p for held in a.held for p in held]
    assert len(owned) == len(set(owned))
    assert sorted(owned + a._free) == list(range(a.num_pages))
    for s, held in enumerate(a.held):
        assert len(held) >= -(-int(a.lens[s]) // a.page_size)
        assert list(a.table[s, :len(held)]) == held


def test_reserve_grows_page_by_page():
    a = PageAllocator(num_pages=10, page_size=64, slots=3, max_pages=4)
    a.reserve(0, 1)
    assert a.held[0] == [0]
    a.reserve(0, 64)
    assert a.held[0] == [0]
    a.reserve(0, 65)
    assert a.held[0] == [0, 1]
    a.reserve(1, 200)
    assert a.held[1] == [2, 3, 4, 5]
    _check_invariants(a)


def test_rollback_and_release_return_pages():
    a = PageAllocator(num_pages=8, page_size=64, slots=2, max_pages=8)
    a.reserve(0, 300)
    a.lens[0] = 300
    a.rollback(0, 129)          # keeps 3 pages
    assert len(a.held[0]) == 3 and a.lens[0] == 129
    assert a.free_pages() == 5
    a.rollback(0, 128)          # exactly 2 pages
    assert len(a.held[0]) == 2
    with pytest.raises(ValueError):
        a.rollback(0, 129)      # cannot grow by rolling back
    a.release(0)
    assert a.held[0] == [] and a.lens[0] == 0 and a.free_pages() == 8
    assert np.all(a.table[0] == 0)
    _check_invariants(a)


def test_freed_pages_are_reused():
    a = PageAllocator(num_pages=4, page_size=64, slots=2, max_pages=4)
    a.reserve(0, 256)
    a.lens[0] = 256
    with pytest.raises(PoolExhausted):
        a.reserve(1, 1)
    a.release(0)
    a.reserve(1, 130)
    assert sorted(a.held[1]) == a.held[1] and len(a.held[1]) == 3
    _check_invariants(a)


def test_failed_requests_change_nothing():
    a = PageAllocator(num_pages=5, page_size=64, slots=2, max_pages=3)
    a.reserve(0, 192)              # 3 pages, 2 left
    before = (a.table.copy(), [list(h) for h in a.held], list(a._free))
    with pytest.raises(ValueError):
        a.reserve(1, 3 * 64 + 1)   # beyond max_pages x page_size
    with pytest.raises(PoolExhausted):
        a.reserve(1, 192)          # needs 3 pages
    assert (a.table == before[0]).all()
    assert [list(h) for h in a.held] == before[1] and a._free == before[2]


def test_random_churn_keeps_invariants():
    rng = np.random.default_rng(3)
    a = PageAllocator(num_pages=40, page_size=64, slots=6, max_pages=12)
    for _ in range(2000):
        s = int(rng.integers(6))
        op = rng.integers(3)
        try:
            if op == 0:
                n = int(a.lens[s] + rng.integers(1, 150))
                a.reserve(s, n)
                a.lens[s] = n
            elif op == 1:
                a.rollback(s, int(rng.integers(0, a.lens[s] + 1)))
            else:
                a.release(s)
        except (PoolExhausted, ValueError):
            pass
        _check_invariants(a)


def test_cache_reservation_is_all_or_nothing():
    """PagedKVCache reserves the pages of all its slots or of none (no GPU:
    only the host bookkeeping runs before the launch)."""
    from paper_2408_00539_amd.paged import PagedKVCache
    cache = PagedKVCache.__new__(PagedKVCache)
    cache.alloc = PageAllocator(num_pages=4, page_size=64, slots=3, max_pages=4)
    cache.alloc.reserve(2, 128)
    cache.alloc.lens[2] = 128
    free_before = cache.alloc.free_pages()
    with pytest.raises(PoolExhausted):
        cache._reserve_all([0, 1], [64, 129])   # 1 page, then 3: only 2 are free
    assert cache.alloc.held[0] == [] and cache.alloc.held[1] == []
    assert cache.alloc.free_pages() == free_before
    with pytest.raises(ValueError):
        cache._reserve_all([0, 0], [1, 1])
