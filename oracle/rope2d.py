"""fp64 CPU oracle of ChatGLM-style 2-D rotary positions for ISM (Sec. 2.3,
the prefix-backbone adaptation). TEST INFRASTRUCTURE: only the test suite,
the smoke check and the benchmark's CPU-baseline leg may use this module.

The paper adapts ISM to ChatGLM and keeps its 2-D positional scheme: one
position encodes the span a token belongs to, the other its offset inside
the span; its figure of the layout is not available. Readings fixed here:

* a span is a segment of the dialogue (the prompt merged with the first
  query, as for Eq. 5): ``pos1(j)`` is the index of j's segment counted from
  the first segment of its dialogue, ``pos2(j)`` is j minus the first token
  of its segment (both from 0);
* the two positions enter as rotary embeddings on the two halves of the
  head dimension: dims [0, d/2) rotate by pos1, dims [d/2, d) by pos2. Inside
  a half of width r = d/2, dims k and k + r/2 (k < r/2) form a pair rotated
  by the angle pos * base^(-2k/r) (base 10000 by default):
      x_k'       = x_k cos a - x_{k+r/2} sin a
      x_{k+r/2}' = x_k sin a + x_{k+r/2} cos a;
* the inverse rotation (angle -a) maps gradients with respect to rotated
  queries and keys back to the unrotated ones (the rotation is orthogonal,
  so its transpose is its inverse).

Pinned by ``tests/test_oracle_rope.py``: hand-derived values at d = 4 and
d = 8 (``tests/golden/``), the identity at position 0, norm preservation,
inverse after forward, the relative-position property of the scores, and
finite differences of attention on rotated inputs.
"""

from __future__ import annotations

import numpy as np


def positions_2d(cu_seqlens, cu_segs):
    """(pos1, pos2) per token of a packed batch: segment index within the
    dialogue and offset within the segment."""
    cu_seqlens = np.asarray(cu_seqlens, dtype=np.int64)
    cu_segs = np.asarray(cu_segs, dtype=np.int64)
    T = int(cu_segs[-1])
    pos1 = np.empty(T, dtype=np.int64)
    pos2 = np.empty(T, dtype=np.int64)
    for b in range(len(cu_seqlens) - 1):
        first = int(np.searchsorted(cu_segs, cu_seqlens[b]))
        g = first
        while g < len(cu_segs) - 1 and cu_segs[g] < cu_seqlens[b + 1]:
            a, c = int(cu_segs[g]), int(cu_segs[g + 1])
            pos1[a:c] = g - first
            pos2[a:c] = np.arange(c - a)
            g += 1
    return pos1, pos2


def rope2d(x, pos1, pos2, base=10000.0, inverse=False):
    """Rotate x [T, H, d] (any float dtype; computed in fp64) by the 2-D
    positions of its tokens. Returns a new fp64 array."""
    x = np.asarray(x, dtype=np.float64)
    T, H, d = x.shape
    if d % 4:
        raise ValueError("d must be a multiple of 4")
    r = d // 2
    k = np.arange(r // 2, dtype=np.float64)
    freq = base ** (-2.0 * k / r)                       # [r/2]
    sign = -1.0 if inverse else 1.0
    out = x.copy()
    for half, pos in ((0, pos1), (1, pos2)):
        ang = sign * np.asarray(pos, dtype=np.float64)[:, None] * freq[None, :]  # [T, r/2]
        c = np.cos(ang)[:, None, :]
        s = np.sin(ang)[:, None, :]
        lo = slice(half * r, half * r + r // 2)
        hi = slice(half * r + r // 2, (half + 1) * r)
        xa, xb = x[:, :, lo], x[:, :, hi]
        out[:, :, lo] = xa * c - xb * s
        out[:, :, hi] = xa * s + xb * c
    return out
