"""Multi-turn serving over the paged KV cache.

Sec. 2.3: with ISM a dialogue's KV cache is reused across turns, and every
turn extends it: the new query segment is prefilled against the cache (Eq. 5
first two cases), then the answer is generated token by token (third case,
f(j) = j). ``PagedKVCache`` runs those turns for many dialogues at once over
one pool of fixed-size pages, each call one launch sequence of the paged
entry points (``ops.prefill_paged``, ``ops.decode_paged``):

* ``prefill(slots, ..., seg_is_query=True)``: a new query segment;
* ``prefill(slots, ..., seg_is_query=False)``: a chunk of answer tokens, each
  row seeing the cache and the chunk's rows up to itself. A chunk of k
  drafted tokens is the same call: one launch verifies them (row r gives
  what decoding the r-th draft would give);
* ``decode(slots, ...)``: one answer token per dialogue;
* ``rollback(slot, length)``: drop rejected drafts (positions past
  ``length`` are no longer part of the dialogue; the next append overwrites
  them);
* ``release(slot)``: the dialogue ended; its pages return to the pool.

``PageAllocator`` is the host-side bookkeeping (no GPU): a free list of page
indices and each dialogue slot's block table row and length.
"""

from __future__ import annotations

import numpy as np

from . import ops


class PoolExhausted(RuntimeError):
    """No free page is left for a dialogue's growth."""


class PageAllocator:
    """Free list over ``num_pages`` pages of ``page_size`` positions; slot b
    holds ``lens[b]`` positions in pages ``table[b, :npages(b)]``."""

    def __init__(self, num_pages, page_size, slots, max_pages):
        if num_pages < 1 or page_size < 1 or slots < 1 or max_pages < 1:
            raise ValueError("num_pages, page_size, slots and max_pages must be positive")
        self.num_pages, self.page_size = int(num_pages), int(page_size)
        self.max_pages = int(max_pages)
        self._free = list(range(self.num_pages - 1, -1, -1))  # pop() -> lowest
        self.table = np.zeros((slots, self.max_pages), dtype=np.int32)
        self.held = [[] for _ in range(slots)]
        self.lens = np.zeros(slots, dtype=np.int64)

    @property
    def capacity(self):
        """Positions one slot can hold."""
        return self.max_pages * self.page_size

    def free_pages(self):
        return len(self._free)

    def reserve(self, slot, length):
        """Make pages cover positions [0, length) of ``slot``; all or nothing."""
        if length > self.capacity:
            raise ValueError(f"slot {slot}: {length} positions exceed the capacity "
                             f"{self.capacity} (max_pages x page_size)")
        held = self.held[slot]
        grow = -(-int(length) // self.page_size) - len(held)
        if grow > len(self._free):
            raise PoolExhausted(f"slot {slot} needs {grow} more pages, {len(self._free)} free")
        for _ in range(max(grow, 0)):
            page = self._free.pop()
            self.table[slot, len(held)] = page
            held.append(page)

    def rollback(self, slot, length):
        """Shorten ``slot`` to ``length`` positions; pages past them return."""
        if not 0 <= length <= self.lens[slot]:
            raise ValueError(f"slot {slot}: rollback to {length} outside [0, {self.lens[slot]}]")
        self.lens[slot] = length
        keep = -(-int(length) // self.page_size)
        held = self.held[slot]
        while len(held) > keep:
            self._free.append(held.pop())
            self.table[slot, len(held)] = 0

    def release(self, slot):
        self.rollback(slot, 0)


class PagedKVCache:
    """Device page pools, one block table row per dialogue slot, and the turn
    operations above. Pools are ``[num_pages, hkv, page_size, d]`` bf16. Each
    call uploads the block table rows and lengths of its slots (a small
    synchronous host-to-device copy): a reference loop, not a graph-captured
    one."""

    def __init__(self, num_pages, page_size, slots, max_pages, hkv, d, device="cuda"):
        import torch
        self.alloc = PageAllocator(num_pages, page_size, slots, max_pages)
        self.hkv, self.d, self.device = hkv, d, device
        shape = (num_pages, hkv, page_size, d)
        self.k_pages = torch.zeros(shape, dtype=torch.bfloat16, device=device)
        self.v_pages = torch.zeros(shape, dtype=torch.bfloat16, device=device)
        self._ws = None

    @property
    def lens(self):
        return self.alloc.lens

    def _reserve_all(self, slots, lengths):
        """Reserve pages for every slot or, if one request fails, for none
        (the pages reserved by this call go back to the pool)."""
        if len(set(slots)) != len(slots):
            raise ValueError("a slot appears twice in one call")
        done = []
        try:
            for s, n in zip(slots, lengths):
                self.alloc.reserve(s, n)
                done.append(s)
        except Exception:
            for s in done:
                self.alloc.rollback(s, int(self.alloc.lens[s]))
            raise

    def _views(self, slots):
        import torch
        tab = torch.from_numpy(self.alloc.table[slots]).to(self.device)
        lens = torch.from_numpy(self.alloc.lens[slots].astype(np.int32)).to(self.device)
        return tab, lens

    def prefill(self, slots, q_new, k_new, v_new, new_lens, seg_is_query=True, scale=None):
        """New segment of ``new_lens[i]`` >= 1 tokens for each slot in
        ``slots`` (rows packed in slot order). Returns (o, lse)."""
        import torch
        slots = list(slots)
        new_lens = [int(n) for n in new_lens]
        if len(new_lens) != len(slots) or min(new_lens, default=1) < 1:
            raise ValueError("one new length >= 1 per slot")
        self._reserve_all(slots, [self.alloc.lens[s] + n for s, n in zip(slots, new_lens)])
        tab, lens = self._views(slots)
        cu = torch.tensor(np.concatenate([[0], np.cumsum(new_lens)]), dtype=torch.int32,
                          device=self.device)
        out = ops.prefill_paged(q_new, k_new, v_new, self.k_pages, self.v_pages, tab, lens,
                                cu, max(new_lens), seg_is_query, scale)
        for s, n in zip(slots, new_lens):
            self.alloc.lens[s] += n
        return out

    def decode(self, slots, q, k_new, v_new, scale=None, num_splits=0):
        """One answer token for each slot in ``slots``. Returns (o, lse)."""
        import torch
        slots = list(slots)
        self._reserve_all(slots, [self.alloc.lens[s] + 1 for s in slots])
        tab, lens = self._views(slots)
        need = ops.workspace_size(ops.ISM_OP_DECODE, len(slots), 0, self.alloc.capacity,
                                  q.shape[1], self.hkv, self.d, num_splits)
        if self._ws is None or self._ws.numel() < need:
            self._ws = torch.empty(need, dtype=torch.uint8, device=self.device)
        out = ops.decode_paged(q, k_new, v_new, self.k_pages, self.v_pages, tab, lens, 0,
                               scale, num_splits, workspace=self._ws)
        for s in slots:
            self.alloc.lens[s] += 1
        return out

    def rollback(self, slot, length):
        self.alloc.rollback(slot, length)

    def release(self, slot):
        self.alloc.release(slot)
