"""Pins of the 2-D rotary-position oracle (ChatGLM-style positions kept under
ISM, Sec. 2.3): hand-derived values, positions of a hand-built layout, the
properties every rotary embedding has, and the chain rule that maps
gradients of rotated queries/keys back to the unrotated ones."""

import os

import numpy as np
import pytest

import oracle
from oracle.rope2d import positions_2d, rope2d

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    rows = [ln.split() for ln in open(os.path.join(GOLDEN, name))
            if ln.strip() and not ln.startswith("#")]
    d, base, p1, p2 = int(rows[0][0]), float(rows[0][1]), int(rows[0][2]), int(rows[0][3])
    x = np.array(rows[1], dtype=np.float64).reshape(1, 1, d)
    want = np.array(rows[2], dtype=np.float64).reshape(1, 1, d)
    return x, base, p1, p2, want


@pytest.mark.parametrize("name", ["rope2d_d4.txt", "rope2d_d8.txt"])
def test_hand_derived_values(name):
    x, base, p1, p2, want = _golden(name)
    got = rope2d(x, [p1], [p2], base)
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-11)


def test_positions_of_a_hand_built_layout():
    # dialogue 0: Q(3) A(2) Q(1) A(4); dialogue 1: Q(2) A(1)
    cu_seqlens = [0, 10, 13]
    cu_segs = [0, 3, 5, 6, 10, 12, 13]
    p1, p2 = positions_2d(cu_seqlens, cu_segs)
    assert p1.tolist() == [0, 0, 0, 1, 1, 2, 3, 3, 3, 3, 0, 0, 1]
    assert p2.tolist() == [0, 1, 2, 0, 1, 0, 0, 1, 2, 3, 0, 1, 0]


def _rand(rng, T=7, H=3, d=16):
    x = rng.standard_normal((T, H, d))
    p1 = rng.integers(0, 40, size=T)
    p2 = rng.integers(0, 3000, size=T)
    return x, p1, p2


def test_position_zero_is_identity():
    x, _, _ = _rand(np.random.default_rng(1))
    z = np.zeros(x.shape[0], dtype=np.int64)
    np.testing.assert_array_equal(rope2d(x, z, z), x)


@pytest.mark.parametrize("d", [4, 8, 64, 128])
def test_orthogonal_and_invertible(d):
    rng = np.random.default_rng(d)
    x, p1, p2 = _rand(rng, d=d)
    y = rope2d(x, p1, p2)
    # each pair is rotated, so every pair's norm and the whole norm are kept
    np.testing.assert_allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1),
                               rtol=1e-12)
    np.testing.assert_allclose(rope2d(y, p1, p2, inverse=True), x, rtol=0, atol=1e-12)
    # the two halves use their own positions: swapping them changes the result
    assert np.max(np.abs(rope2d(x, p2, p1) - y)) > 1e-3


def test_scores_depend_on_position_differences_only():
    rng = np.random.default_rng(2)
    T, H, d = 5, 2, 32
    q = rng.standard_normal((T, H, d))
    k = rng.standard_normal((T, H, d))
    p1, p2 = rng.integers(0, 20, T), rng.integers(0, 500, T)
    s = np.einsum("ihd,jhd->hij", rope2d(q, p1, p2), rope2d(k, p1, p2))
    s_shift = np.einsum("ihd,jhd->hij", rope2d(q, p1 + 13, p2 + 777),
                        rope2d(k, p1 + 13, p2 + 777))
    np.testing.assert_allclose(s_shift, s, rtol=0, atol=1e-9)


def test_gradients_through_the_rotation():
    """Attention on rotated queries and keys: the gradient with respect to
    the unrotated q (k) is the inverse rotation of the gradient with respect
    to the rotated one; checked by central differences."""
    rng = np.random.default_rng(4)
    cu_seqlens = np.array([0, 7])
    cu_segs = np.array([0, 3, 5, 7])
    isq = np.array([1, 0, 1], dtype=np.uint8)
    T, hq, hkv, d = 7, 2, 1, 8
    q = rng.standard_normal((T, hq, d))
    k = rng.standard_normal((T, hkv, d))
    v = rng.standard_normal((T, hkv, d))
    do = rng.standard_normal((T, hq, d))
    p1, p2 = positions_2d(cu_seqlens, cu_segs)
    scale = 0.4

    def loss(qq, kk):
        o, _ = oracle.fwd(rope2d(qq, p1, p2), rope2d(kk, p1, p2), v, cu_seqlens, cu_segs,
                          isq, scale)
        return float(np.sum(o * do))

    gq, gk, _ = oracle.bwd(rope2d(q, p1, p2), rope2d(k, p1, p2), v, do, cu_seqlens, cu_segs,
                           isq, scale)
    dq = rope2d(gq, p1, p2, inverse=True)
    dk = rope2d(gk, p1, p2, inverse=True)
    eps = 1e-6
    for arr, grad in ((q, dq), (k, dk)):
        num = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            old = arr[idx]
            arr[idx] = old + eps
            up = loss(q, k)
            arr[idx] = old - eps
            dn = loss(q, k)
            arr[idx] = old
            num[idx] = (up - dn) / (2 * eps)
        np.testing.assert_allclose(grad, num, rtol=0, atol=1e-7)
