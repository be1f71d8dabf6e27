"""Checkpoint and resume of the serving state. Across turns the KV cache is
the whole state the method carries (Sec. 2.3: the history cache is reused
and extended); after a prefill and some decode steps, a copy of the cache
(and of the lengths, and for the paged pool of its table) taken to host
memory and loaded into fresh device tensors continues exactly like the live
cache: the next decode steps and the next turn's prefill give the same bits
and leave the same cache."""

import copy

import numpy as np
import pytest

from tests._gpu import announce, torch_cuda

pytestmark = pytest.mark.gpu


def _inputs(torch, seed, B, hq, hkv, d, new):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    r = lambda *s: torch.randn(s, generator=g, device="cuda").to(torch.bfloat16)  # noqa: E731
    Tn = sum(new)
    turn1 = (r(Tn, hq, d), r(Tn, hkv, d), r(Tn, hkv, d))
    steps = [(r(B, hq, d), r(B, hkv, d), r(B, hkv, d)) for _ in range(5)]
    new2 = [n // 2 + 1 for n in new]
    T2 = sum(new2)
    turn2 = (r(T2, hq, d), r(T2, hkv, d), r(T2, hkv, d))
    return turn1, steps, new2, turn2


def _cu(torch, lens):
    return torch.tensor(np.concatenate([[0], np.cumsum(lens)]), dtype=torch.int32, device="cuda")


@pytest.mark.parametrize("hq,hkv", [(4, 4), (8, 1)])
def test_dense_cache_resume(hq, hkv):
    torch = torch_cuda()
    from paper_2408_00539_amd import ops
    B, d, cap = 3, 128, 1024
    hist = [200, 37, 512]
    new = [70, 129, 5]
    turn1, steps, new2, turn2 = _inputs(torch, 40 + hq, B, hq, hkv, d, new)
    announce("resume dense", hq, hkv, hist, new)
    g = torch.Generator(device="cuda")
    g.manual_seed(41)
    kc = torch.randn((B, hkv, cap, d), generator=g, device="cuda").to(torch.bfloat16)
    vc = torch.randn((B, hkv, cap, d), generator=g, device="cuda").to(torch.bfloat16)
    lens = torch.tensor(hist, dtype=torch.int32, device="cuda")
    sc = d ** -0.5
    ops.prefill_cached(*turn1, kc, vc, lens, _cu(torch, new), max(new), sc)
    lens += torch.tensor(new, dtype=torch.int32, device="cuda")
    for q, k, v in steps[:3]:
        ops.decode(q, k, v, kc, vc, lens, 0, sc)
        lens += 1
    torch.cuda.synchronize()
    # checkpoint: the whole state, in host memory
    ck = (kc.cpu(), vc.cpu(), lens.cpu())

    def continue_from(kc, vc, lens):
        outs = []
        for q, k, v in steps[3:]:
            outs += list(ops.decode(q, k, v, kc, vc, lens, 0, sc))
            lens += 1
        outs += list(ops.prefill_cached_segment(*turn2, kc, vc, lens, _cu(torch, new2),
                                                max(new2), False, sc))
        torch.cuda.synchronize()
        return outs

    live = continue_from(kc, vc, lens)
    kc2, vc2, lens2 = (x.cuda() for x in ck)  # a fresh copy, as after a reload
    resumed = continue_from(kc2, vc2, lens2)
    for a, b in zip(live, resumed):
        assert torch.equal(a, b)
    assert torch.equal(kc, kc2) and torch.equal(vc, vc2) and torch.equal(lens, lens2)


def test_paged_cache_resume():
    torch = torch_cuda()
    from paper_2408_00539_amd import paged
    B, hq, hkv, d = 3, 8, 2, 128
    new = [300, 64, 129]
    turn1, steps, new2, turn2 = _inputs(torch, 42, B, hq, hkv, d, new)
    announce("resume paged", hq, hkv, new)
    cache = paged.PagedKVCache(num_pages=24, page_size=64, slots=4, max_pages=12, hkv=hkv, d=d)
    slots = [2, 0, 3]
    sc = d ** -0.5
    cache.prefill(slots, *turn1, new, True, sc)
    for q, k, v in steps[:3]:
        cache.decode(slots, q, k, v, sc)
    torch.cuda.synchronize()
    # checkpoint: pages in host memory plus the allocator's table and lengths
    ck = (cache.k_pages.cpu(), cache.v_pages.cpu(), copy.deepcopy(cache.alloc))

    def continue_from(c):
        outs = []
        for q, k, v in steps[3:]:
            outs += list(c.decode(slots, q, k, v, sc))
        outs += list(c.prefill(slots, *turn2, new2, False, sc))
        torch.cuda.synchronize()
        return outs

    live = continue_from(cache)
    fresh = paged.PagedKVCache(num_pages=24, page_size=64, slots=4, max_pages=12, hkv=hkv, d=d)
    fresh.k_pages.copy_(ck[0])
    fresh.v_pages.copy_(ck[1])
    fresh.alloc = ck[2]
    resumed = continue_from(fresh)
    for a, b in zip(live, resumed):
        assert torch.equal(a, b)
    assert torch.equal(cache.k_pages, fresh.k_pages) and torch.equal(cache.v_pages, fresh.v_pages)
    assert np.array_equal(cache.alloc.table, fresh.alloc.table)
    assert np.array_equal(cache.alloc.lens, fresh.alloc.lens)
