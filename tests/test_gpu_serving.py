"""GPU parity of multi-turn serving over the paged KV cache (Sec. 2.3: each
turn reuses the dialogue's cache, prefills the new query segment against it,
then generates the answer, which extends the cache).

* A serving loop over several dialogue slots sharing one page pool: per turn
  a query segment (Eq. 5 first two cases), then the answer as one decode
  step, a chunk of answer tokens prefilled causally (third case), and more
  decode steps; a finished dialogue is released and a new one reuses its
  pages. Every output is compared with the fp64 oracle's stepwise path
  (``oracle.prefill_cached`` / ``oracle.decode_step``) on the same history.
* Verification of drafted tokens (speculative decoding): k drafts prefilled
  as one answer chunk give, row by row, what k decode steps give; rejected
  drafts are rolled back and decoding continues from the accepted prefix.
"""

import numpy as np
import pytest

import oracle
from paper_2408_00539_amd import workloads as W
from tests._gpu import announce, compare, dev_bf16, f64, host_f64, torch_cuda

pytestmark = pytest.mark.gpu


def _bits(rng, *shape):
    return W.to_bf16_bits(rng.standard_normal(shape, dtype=np.float32))


class _Ref:
    """The oracle's per-dialogue history (fp64, [p, hkv, d])."""

    def __init__(self, hkv, d):
        self.k, self.v = {}, {}
        self.hkv, self.d = hkv, d

    def reset(self, s):
        self.k[s] = np.zeros((0, self.hkv, self.d))
        self.v[s] = np.zeros((0, self.hkv, self.d))

    def prefill(self, s, q, k, v, scale, is_query):
        o, lse, self.k[s], self.v[s] = oracle.prefill_cached(
            self.k[s], self.v[s], f64(q), f64(k), f64(v), scale, new_is_query=is_query)
        return o, lse

    def decode(self, s, q, k, v, scale):
        o, lse, self.k[s], self.v[s] = oracle.decode_step(self.k[s], self.v[s], f64(q),
                                                          f64(k), f64(v), scale)
        return o, lse


def _prefill_turn(cache, ref, rng, slots, lens, hq, hkv, d, scale, is_query, tag):
    q, k, v = (_bits(rng, sum(lens), hq, d), _bits(rng, sum(lens), hkv, d),
               _bits(rng, sum(lens), hkv, d))
    announce(tag, slots, lens, is_query)
    o, lse = cache.prefill(slots, dev_bf16(q), dev_bf16(k), dev_bf16(v), lens, is_query, scale)
    o, lse = host_f64(o), host_f64(lse)
    r = 0
    for s, n in zip(slots, lens):
        ro, rl = ref.prefill(s, q[r:r + n], k[r:r + n], v[r:r + n], scale, is_query)
        compare(f"{tag} O slot {s}", o[r:r + n], ro)
        compare(f"{tag} LSE slot {s}", lse[:, r:r + n], rl)
        r += n


def _decode_step(cache, ref, rng, slots, hq, hkv, d, scale, tag, splits=0):
    q, k, v = (_bits(rng, len(slots), hq, d), _bits(rng, len(slots), hkv, d),
               _bits(rng, len(slots), hkv, d))
    announce(tag, slots)
    o, lse = cache.decode(slots, dev_bf16(q), dev_bf16(k), dev_bf16(v), scale, splits)
    o, lse = host_f64(o), host_f64(lse)
    for i, s in enumerate(slots):
        ro, rl = ref.decode(s, q[i], k[i], v[i], scale)
        compare(f"{tag} O slot {s}", o[i], ro)
        compare(f"{tag} LSE slot {s}", lse[:, i], rl)


@pytest.mark.parametrize("hq,hkv,d,page_size", [(8, 2, 128, 64), (4, 4, 64, 128)])
def test_serving_loop_over_turns(hq, hkv, d, page_size):
    torch_cuda()
    from paper_2408_00539_amd.paged import PagedKVCache
    rng = np.random.default_rng(hq * 10 + d + page_size)
    slots, max_pages = 4, 12
    # the pool is smaller than slots x max_pages; a released dialogue's pages
    # are the next ones handed out
    cache = PagedKVCache(num_pages=40, page_size=page_size, slots=slots,
                         max_pages=max_pages, hkv=hkv, d=d)
    ref = _Ref(hkv, d)
    for s in range(slots):
        ref.reset(s)
    scale = 1 / np.sqrt(d)
    active = list(range(slots))
    freed = []
    for turn in range(3):
        qlens = [int(x) for x in rng.integers(1, 90, size=len(active))]
        _prefill_turn(cache, ref, rng, active, qlens, hq, hkv, d, scale, True, f"turn {turn} query")
        _decode_step(cache, ref, rng, active, hq, hkv, d, scale, f"turn {turn} answer token 0")
        alens = [int(x) for x in rng.integers(1, 70, size=len(active))]
        _prefill_turn(cache, ref, rng, active, alens, hq, hkv, d, scale, False,
                      f"turn {turn} answer chunk")
        for t in range(3):
            _decode_step(cache, ref, rng, active, hq, hkv, d, scale,
                         f"turn {turn} answer token {t + 1}", splits=[0, 2, 5][t])
        if turn == 0:
            # dialogue 1 ends; a new dialogue starts in its slot on its pages
            freed = list(cache.alloc.held[1])
            cache.release(1)
            ref.reset(1)
    # the new dialogue in slot 1 (or another slot's growth) took freed pages
    assert freed and set(freed) & {p for h in cache.alloc.held for p in h}
    assert all(int(cache.lens[s]) == ref.k[s].shape[0] for s in range(slots))


@pytest.mark.parametrize("hq,hkv,d", [(8, 2, 128), (4, 1, 64)])
def test_draft_verification_and_rollback(hq, hkv, d):
    torch = torch_cuda()
    from paper_2408_00539_amd.paged import PagedKVCache
    rng = np.random.default_rng(7 * hq + d)
    cache = PagedKVCache(num_pages=16, page_size=64, slots=2, max_pages=8, hkv=hkv, d=d)
    ref = _Ref(hkv, d)
    scale = 1 / np.sqrt(d)
    for s in range(2):
        ref.reset(s)
    _prefill_turn(cache, ref, rng, [0, 1], [100, 63], hq, hkv, d, scale, True, "history")
    _decode_step(cache, ref, rng, [0, 1], hq, hkv, d, scale, "first answer token")
    k_draft = 6
    q, k, v = (_bits(rng, 2 * k_draft, hq, d), _bits(rng, 2 * k_draft, hkv, d),
               _bits(rng, 2 * k_draft, hkv, d))
    base = [int(cache.lens[0]), int(cache.lens[1])]
    announce("verify drafts", k_draft)
    o, lse = cache.prefill([0, 1], dev_bf16(q), dev_bf16(k), dev_bf16(v), [k_draft, k_draft],
                           False, scale)
    o, lse = host_f64(o), host_f64(lse)
    # row r of the chunk equals decoding draft r after drafts 0..r-1
    kd, vd = dict(ref.k), dict(ref.v)
    for s in range(2):
        for r in range(k_draft):
            i = s * k_draft + r
            ro, rl, kd[s], vd[s] = oracle.decode_step(kd[s], vd[s], f64(q[i]), f64(k[i]),
                                                      f64(v[i]), scale)
            compare(f"draft {r} slot {s} O", o[i], ro)
            compare(f"draft {r} slot {s} LSE", lse[:, i], rl)
    # accept 2 drafts in slot 0 and none in slot 1, then keep decoding
    accepted = [2, 0]
    for s in range(2):
        cache.rollback(s, base[s] + accepted[s])
        n = accepted[s]
        ref.k[s] = np.concatenate([ref.k[s], f64(k[s * k_draft:s * k_draft + n])])
        ref.v[s] = np.concatenate([ref.v[s], f64(v[s * k_draft:s * k_draft + n])])
    for t in range(4):
        _decode_step(cache, ref, rng, [0, 1], hq, hkv, d, scale, f"after rollback {t}")
    torch.cuda.synchronize()
    assert [int(x) for x in cache.lens] == [base[0] + 2 + 4, base[1] + 4]
