"""Seeded synthetic inputs shaped like the paper's multi-turn dialogues.

This module only draws random numbers and lays them out; it holds none of the
attention arithmetic, so both the HIP path's tests and the oracle may read its
output. Dialogues alternate query and answer segments and start with a query
segment (the prompt and the first query form one bidirectional block, Eq. 5
first case). Lengths follow the laws of the five workloads below; tensors are
i.i.d. N(0, 1) drawn in float32 and rounded to bfloat16 (round to nearest
even) on the host, stored as raw uint16 bit patterns.

Random streams (numpy PCG64): the segment layout uses SeedSequence([seed, 0]);
every tensor of every dialogue has its own stream SeedSequence([seed, 1, code,
b]) so that one dialogue's slice can be regenerated without the rest.

Workloads (all dialogue turns are [query, answer] pairs):

0. forward, 1 dialogue of 4 turns, 1 head, head_dim 64; query lengths
   uniform in [8, 32], answer lengths uniform in [16, 48] (<= 320 tokens).
1. forward, 8 dialogues x 4096 tokens, 32 heads, head_dim 128, 8 turns each;
   query lengths lognormal(median 96, sigma 0.8), answer lengths
   lognormal(median 320, sigma 0.7), rescaled to sum to 4096.
2. forward with grouped KV heads (32 query / 8 KV heads), head_dim 128,
   2 dialogues x 16384 tokens, 24 turns, the laws of workload 1.
3. KV-cache reuse: 32 dialogues, 32 heads, head_dim 128, a history of 8192
   cached tokens (16 turns, laws of workload 1), a new query segment of
   length uniform in [64, 512] per dialogue, then 256 single-token answer
   decode steps.
4. backward, 4 dialogues x 8192 tokens, 32 heads, head_dim 128, 16 turns,
   laws of workload 1; upstream gradient dO i.i.d. N(0, 1).
"""

from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

# stream codes for per-tensor random streams
Q, K, V, DO, Q_NEW, K_NEW, V_NEW, K_HIST, V_HIST, Q_DEC, K_DEC, V_DEC = range(12)

DECODE_STEPS = 256
CACHE_CAP = 9216


# --------------------------------------------------------------------------
# bfloat16 helpers (bit patterns as uint16)
# --------------------------------------------------------------------------

def to_bf16_bits(x, out=None):
    """float32 array -> bfloat16 bit patterns (round to nearest even).

    Written with in-place steps to keep large conversions to two passes of
    fresh memory; ``out`` (uint16, same shape) receives the result if given.
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = u >> np.uint32(16)
    r &= np.uint32(1)
    r += np.uint32(0x7FFF)
    r += u
    r >>= np.uint32(16)
    if out is None:
        return r.astype(np.uint16)
    np.copyto(out, r, casting="unsafe")
    return out


def bf16_bits_to_f32(b):
    """bfloat16 bit patterns -> float32 (exact)."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


# --------------------------------------------------------------------------
# Lengths
# --------------------------------------------------------------------------

def rescale_lengths(x, total):
    """Scale positive reals x to integers >= 1 summing exactly to ``total``.

    x * total / sum(x), floored, clamped to >= 1; the residual is handed out
    one token at a time by largest fractional part (or, when the clamp made
    the sum too large, taken back from the smallest fractional parts among
    entries above 1).
    """
    x = np.asarray(x, dtype=np.float64)
    if total < len(x):
        raise ValueError("total smaller than the number of segments")
    y = x * (total / x.sum())
    f = np.maximum(np.floor(y), 1).astype(np.int64)
    frac = y - np.floor(y)
    res = total - int(f.sum())
    order = np.argsort(-frac, kind="stable")
    i = 0
    while res > 0:
        f[order[i % len(f)]] += 1
        res -= 1
        i += 1
    order = np.argsort(frac, kind="stable")
    i = 0
    while res < 0:
        j = order[i % len(f)]
        if f[j] > 1:
            f[j] -= 1
            res += 1
        i += 1
    assert int(f.sum()) == total and f.min() >= 1
    return f


def _lognormal_turns(rng, turns, total):
    q = rng.lognormal(math.log(96.0), 0.8, size=turns)
    a = rng.lognormal(math.log(320.0), 0.7, size=turns)
    x = np.empty(2 * turns)
    x[0::2], x[1::2] = q, a
    return rescale_lengths(x, total)


def _uniform_turns(rng, turns):
    q = rng.integers(8, 33, size=turns)
    a = rng.integers(16, 49, size=turns)
    x = np.empty(2 * turns, dtype=np.int64)
    x[0::2], x[1::2] = q, a
    return x


@dataclass
class Segments:
    """Dialogue structure of a packed batch (int32 / uint8 host arrays)."""
    cu_seqlens: np.ndarray
    cu_segs: np.ndarray
    seg_is_query: np.ndarray

    @property
    def batch(self):
        return len(self.cu_seqlens) - 1

    @property
    def num_segs(self):
        return len(self.seg_is_query)

    @property
    def total(self):
        return int(self.cu_seqlens[-1])

    @property
    def max_seqlen(self):
        return int(np.max(np.diff(self.cu_seqlens))) if self.batch else 0


def segments_from_lengths(per_dialogue):
    """Build packed metadata from a list of dialogues, each a list of
    (length, is_query) segments."""
    cu_seqlens = [0]
    cu_segs = [0]
    flags = []
    for dia in per_dialogue:
        for n, isq in dia:
            cu_segs.append(cu_segs[-1] + int(n))
            flags.append(1 if isq else 0)
        cu_seqlens.append(cu_segs[-1])
    return Segments(np.asarray(cu_seqlens, dtype=np.int32),
                    np.asarray(cu_segs, dtype=np.int32),
                    np.asarray(flags, dtype=np.uint8))


def alternating(lengths, first_is_query=True):
    """[(len, is_query)] for segments that alternate query / answer."""
    return [(int(n), (i % 2 == 0) == first_is_query)
            for i, n in enumerate(lengths)]


def prefix_expansion(segs):
    """The multi-sample layout a prefix-mask model trains on (Sec. 1): every
    dialogue [Q_1, A_1, ..., Q_n, A_n] becomes n samples, sample k being the
    history up to Q_k as one bidirectional prefix (Eq. 3) followed by A_k as
    a causal answer. ISM covers the same answers in one pass over the
    dialogue.

    Returns (expanded Segments, src) where src[t] is the token of the
    original packed axis that expanded token t copies (so expanded tensors
    are gathers of the original ones). Dialogues must alternate query /
    answer segments starting with a query; a trailing query segment without
    an answer yields no sample.
    """
    cu, cs, fl = segs.cu_seqlens, segs.cu_segs, segs.seg_is_query
    samples, src = [], []
    g = 0
    for b in range(segs.batch):
        s, e = int(cu[b]), int(cu[b + 1])
        while g < len(fl) and cs[g] < e:
            a, c = int(cs[g]), int(cs[g + 1])
            if not fl[g]:
                raise ValueError("dialogues must alternate query / answer "
                                 "segments starting with a query")
            if g + 1 < len(fl) and cs[g + 1] < e:
                if fl[g + 1]:
                    raise ValueError("two adjacent query segments")
                a2 = int(cs[g + 2])
                samples.append([(c - s, True), (a2 - c, False)])
                src.append(np.arange(s, a2, dtype=np.int64))
                g += 2
            else:
                g += 1
    exp = segments_from_lengths(samples)
    return exp, (np.concatenate(src) if src else np.zeros(0, np.int64))


# --------------------------------------------------------------------------
# Tensors
# --------------------------------------------------------------------------

def normal_bf16(seed, code, b, shape, out=None):
    """N(0,1) bf16 bits of one dialogue's slice of one tensor."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(
        [int(seed), 1, int(code), int(b)])))
    return to_bf16_bits(rng.standard_normal(shape, dtype=np.float32), out=out)


def _pmap(fn, items):
    """Run fn over items on a few threads (numpy's generators and
    element-wise passes release the GIL)."""
    items = list(items)
    workers = max(1, min(16, len(os.sched_getaffinity(0)), len(items)))
    if workers == 1:
        return [fn(i) for i in items]
    with ThreadPoolExecutor(max_workers=workers) as ex:
        return list(ex.map(fn, items))


def packed_tensor(seed, code, cu_seqlens, heads, d):
    """[T, heads, d] bf16 bits, generated dialogue by dialogue."""
    cu = np.asarray(cu_seqlens)
    out = np.empty((int(cu[-1]), heads, d), dtype=np.uint16)

    def one(b):
        normal_bf16(seed, code, b, (int(cu[b + 1] - cu[b]), heads, d),
                    out=out[cu[b]:cu[b + 1]])

    _pmap(one, range(len(cu) - 1))
    return out


@dataclass
class Workload:
    """One synthetic workload. Tensors are bf16 bit patterns (uint16)."""
    index: int
    seed: int
    name: str
    hq: int
    hkv: int
    d: int
    segs: Segments = None
    q: np.ndarray = None
    k: np.ndarray = None
    v: np.ndarray = None
    do: np.ndarray = None
    # KV-cache reuse (workload 3)
    hist: Segments = None              # history segments, one dialogue each
    hist_len: int = 0
    cache_cap: int = 0
    new_lens: np.ndarray = None        # [B] new query lengths
    cu_new: np.ndarray = None          # [B+1]
    q_new: np.ndarray = None
    k_new: np.ndarray = None
    v_new: np.ndarray = None
    k_cache: np.ndarray = None         # [B, Hkv, cap, d], history filled
    v_cache: np.ndarray = None
    steps: int = 0
    q_dec: np.ndarray = None           # [steps, B, Hq, d]
    k_dec: np.ndarray = None           # [steps, B, Hkv, d]
    v_dec: np.ndarray = None
    extra: dict = field(default_factory=dict)

    @property
    def scale(self):
        return 1.0 / math.sqrt(self.d)


def _layout_rng(seed):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(
        [int(seed), 0])))


def make_segments(index, seed):
    """Segment layout of workload ``index`` (no tensors)."""
    rng = _layout_rng(seed)
    if index == 0:
        return segments_from_lengths([alternating(_uniform_turns(rng, 4))])
    if index == 1:
        return segments_from_lengths(
            [alternating(_lognormal_turns(rng, 8, 4096)) for _ in range(8)])
    if index == 2:
        return segments_from_lengths(
            [alternating(_lognormal_turns(rng, 24, 16384)) for _ in range(2)])
    if index == 4:
        return segments_from_lengths(
            [alternating(_lognormal_turns(rng, 16, 8192)) for _ in range(4)])
    raise ValueError(f"workload {index} has no packed segment layout")


def make_workload(index, seed=None, tensors=True, steps=DECODE_STEPS,
                  batch=None):
    """Build workload ``index`` (0..4) with ``seed`` (default: the index).

    ``tensors=False`` returns the layout only. For workload 3, ``batch``
    may shrink the number of dialogues (the first ``batch`` dialogues of the
    full workload, same values) and ``steps`` the number of decode steps.
    """
    seed = index if seed is None else seed
    if index in (0, 1, 2, 4):
        shapes = {0: (1, 1, 64), 1: (32, 32, 128), 2: (32, 8, 128),
                  4: (32, 32, 128)}
        hq, hkv, d = shapes[index]
        names = {0: "ism_fwd_1x<=320_h1_d64", 1: "ism_fwd_8x4096_h32_d128",
                 2: "ism_fwd_gqa_2x16384_h32kv8_d128",
                 4: "ism_bwd_4x8192_h32_d128"}
        w = Workload(index, seed, names[index], hq, hkv, d)
        w.segs = make_segments(index, seed)
        if tensors:
            cu = w.segs.cu_seqlens
            w.q = packed_tensor(seed, Q, cu, hq, d)
            w.k = packed_tensor(seed, K, cu, hkv, d)
            w.v = packed_tensor(seed, V, cu, hkv, d)
            if index == 4:
                w.do = packed_tensor(seed, DO, cu, hq, d)
        return w
    if index == 3:
        return _make_cache_workload(seed, tensors, steps, batch)
    raise ValueError(f"unknown workload {index}")


def _make_cache_workload(seed, tensors, steps, batch):
    B_full, H, d, C = 32, 32, 128, 8192
    rng = _layout_rng(seed)
    hist = [alternating(_lognormal_turns(rng, 16, C)) for _ in range(B_full)]
    new_lens = rng.integers(64, 513, size=B_full)
    B = B_full if batch is None else int(batch)
    hist, new_lens = hist[:B], new_lens[:B]
    w = Workload(3, seed, "ism_cache_b32_h32_d128_ctx8192", H, H, d)
    w.hist = segments_from_lengths(hist)
    w.hist_len = C
    w.cache_cap = CACHE_CAP
    w.new_lens = new_lens.astype(np.int32)
    w.cu_new = np.concatenate([[0], np.cumsum(new_lens)]).astype(np.int32)
    w.steps = steps
    if tensors:
        w.q_new = packed_tensor(seed, Q_NEW, w.cu_new, H, d)
        w.k_new = packed_tensor(seed, K_NEW, w.cu_new, H, d)
        w.v_new = packed_tensor(seed, V_NEW, w.cu_new, H, d)
        w.k_cache = np.zeros((B, H, w.cache_cap, d), dtype=np.uint16)
        w.v_cache = np.zeros((B, H, w.cache_cap, d), dtype=np.uint16)

        def hist_one(job):
            b, code = job
            dst = w.k_cache if code == K_HIST else w.v_cache
            dst[b, :, :C] = history_slice(seed, code, b, H, C, d)

        _pmap(hist_one, [(b, c) for b in range(B) for c in (K_HIST, V_HIST)])
        w.q_dec = np.stack([normal_bf16(seed, Q_DEC, b, (steps, H, d))
                            for b in range(B)], axis=1)
        w.k_dec = np.stack([normal_bf16(seed, K_DEC, b, (steps, H, d))
                            for b in range(B)], axis=1)
        w.v_dec = np.stack([normal_bf16(seed, V_DEC, b, (steps, H, d))
                            for b in range(B)], axis=1)
    return w


def history_slice(seed, code, b, heads, length, d):
    """Cached history of dialogue b, in cache layout [heads, length, d]."""
    return normal_bf16(seed, code, b, (heads, length, d))
