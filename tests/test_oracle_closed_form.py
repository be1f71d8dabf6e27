"""Pins of the oracle's Q = 0 closed forms and of seer (who sees a key).

The closed forms are derived from Eq. 4/5 with softmax (uniform weights over
a row's visible keys); here they are pinned to the oracle's general forward
and backward (themselves pinned by brute force, library attention, finite
differences and the paper's invariants) and seer to the dense mask.
"""

import math

import numpy as np
import pytest

import oracle
from paper_2408_00539_amd.workloads import alternating, segments_from_lengths


def _random_layout(rng, n_dialogues, max_len):
    dias = []
    for _ in range(n_dialogues):
        n = int(rng.integers(1, max_len + 1))
        parts, left = [], n
        while left:
            ln = int(rng.integers(1, left + 1))
            parts.append(ln)
            left -= ln
        dias.append([(p, bool(rng.integers(0, 2))) for p in parts])
    return segments_from_lengths(dias)


def _args(segs):
    return segs.cu_seqlens, segs.cu_segs, segs.seg_is_query


@pytest.mark.parametrize("seed", range(20))
def test_seer_is_first_row_of_each_mask_column(seed):
    """seer(i) = first row of the dense Eq. 5 mask whose column i is set, and
    every later row of the dialogue sees i as well (so seer alone decides
    visibility below the diagonal's look-ahead)."""
    rng = np.random.default_rng(seed)
    segs = _random_layout(rng, int(rng.integers(1, 4)), 40)
    se = oracle.seer(*_args(segs))
    cu = segs.cu_seqlens
    for b in range(len(cu) - 1):
        s, e = int(cu[b]), int(cu[b + 1])
        M = oracle.mask_dense(*_args(segs), b)
        for i in range(e - s):
            rows = np.nonzero(M[:, i])[0]
            assert rows[0] + s == se[s + i]
            assert np.array_equal(rows, np.arange(rows[0], e - s))


def test_seer_hand_layout():
    """[Q 3, A 2, Q 2] then [A 2, Q 1]: a query key is first seen by its
    segment's first token, an answer key by itself."""
    segs = segments_from_lengths([alternating([3, 2, 2]), [(2, False), (1, True)]])
    assert list(oracle.seer(*_args(segs))) == [0, 0, 0, 3, 4, 5, 5, 7, 8, 9]


@pytest.mark.parametrize("seed,hq,hkv", [(0, 1, 1), (1, 4, 2), (2, 3, 1), (3, 2, 2),
                                         (4, 6, 3), (5, 1, 1)])
def test_uniform_fwd_equals_general_forward(seed, hq, hkv):
    rng = np.random.default_rng(100 + seed)
    segs = _random_layout(rng, int(rng.integers(1, 4)), 60)
    T, d = segs.total, 8
    k, v = rng.standard_normal((T, hkv, d)), rng.standard_normal((T, hkv, d))
    o, lse = oracle.fwd(np.zeros((T, hq, d)), k, v, *_args(segs), 0.37)
    ou, lu = oracle.uniform_fwd(v, *_args(segs))
    G = hq // hkv
    for h in range(hq):
        np.testing.assert_allclose(o[:, h], ou[:, h // G], rtol=0, atol=1e-12)
        np.testing.assert_allclose(lse[h], lu, rtol=0, atol=1e-12)


@pytest.mark.parametrize("seed,hq,hkv", [(0, 1, 1), (1, 4, 2), (2, 3, 1), (3, 2, 2),
                                         (4, 6, 3)])
def test_uniform_bwd_equals_general_backward(seed, hq, hkv):
    rng = np.random.default_rng(200 + seed)
    segs = _random_layout(rng, int(rng.integers(1, 4)), 50)
    T, d, scale = segs.total, 8, 1 / math.sqrt(8)
    k, v = rng.standard_normal((T, hkv, d)), rng.standard_normal((T, hkv, d))
    dq, dk, dv = oracle.bwd(np.zeros((T, hq, d)), k, v, np.ones((T, hq, d)),
                            *_args(segs), scale)
    uq, uk, uv = oracle.uniform_bwd(k, v, hq, scale, *_args(segs))
    np.testing.assert_allclose(uq, dq, rtol=0, atol=1e-11)
    np.testing.assert_allclose(uk, dk, rtol=0, atol=1e-12)
    np.testing.assert_allclose(uv, dv, rtol=0, atol=1e-11)


def test_uniform_bwd_row_weight_replaces_dv_weights_only():
    """row_weight changes dV (sum of the weights of the rows that see each
    key) and nothing else."""
    segs = segments_from_lengths([alternating([4, 3, 5])])
    rng = np.random.default_rng(3)
    T = segs.total
    k, v = rng.standard_normal((T, 1, 4)), rng.standard_normal((T, 1, 4))
    w = np.arange(1, T + 1, dtype=np.float64)
    q1, _, v1 = oracle.uniform_bwd(k, v, 1, 0.5, *_args(segs))
    q2, _, v2 = oracle.uniform_bwd(k, v, 1, 0.5, *_args(segs), row_weight=w)
    np.testing.assert_array_equal(q1, q2)
    se = oracle.seer(*_args(segs))
    for i in range(T):
        assert v2[i, 0, 0] == pytest.approx(w[se[i]:].sum())
