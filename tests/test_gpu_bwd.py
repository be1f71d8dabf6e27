"""GPU parity of ism_attn_bwd against the oracle's textbook gradients.

The GPU backward consumes the GPU forward's O and LSE (as in training); the
oracle recomputes everything from Q, K, V, dO alone.
"""

import zlib

import numpy as np
import pytest

import oracle
from paper_2408_00539_amd import workloads as W
from tests._gpu import announce, compare, dev_bf16, f64, host_f64, torch_cuda

pytestmark = pytest.mark.gpu


def _bits(rng, *shape):
    return W.to_bf16_bits(rng.standard_normal(shape, dtype=np.float32))


def _gpu_grads(segs_h, q, k, v, do, scale, deterministic=True):
    torch = torch_cuda()
    from paper_2408_00539_amd import ops
    segs = ops.Segments.from_host(segs_h.cu_seqlens, segs_h.cu_segs,
                                  segs_h.seg_is_query)
    Q, K, V, DO = dev_bf16(q), dev_bf16(k), dev_bf16(v), dev_bf16(do)
    o, lse = ops.fwd(Q, K, V, segs, scale)
    dq, dk, dv = ops.bwd(Q, K, V, o, lse, DO, segs, scale, deterministic)
    torch.cuda.synchronize()
    return dq, dk, dv


LAYOUTS = {
    "single_token": [[(1, True)]],
    "ragged": [W.alternating([31, 33, 1, 65, 32, 97])],
    "all_answer": [[(200, False)]],
    "all_query": [[(129, True)]],
    "answer_first_adjacent_q": [[(40, False), (30, True), (35, True), (5, False)]],
    "packed_mixed": [W.alternating([5, 9]), [(130, False)],
                     W.alternating([70, 1, 1, 60]), [(33, True)]],
}


@pytest.mark.parametrize("layout", sorted(LAYOUTS))
@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("hq,hkv", [(1, 1), (4, 1), (4, 4), (8, 2), (4, 2), (6, 2)])
def test_small_shapes(layout, d, hq, hkv):
    segs = W.segments_from_lengths(LAYOUTS[layout])
    rng = np.random.default_rng(zlib.crc32(f"bwd/{layout}/{d}/{hq}/{hkv}".encode()))
    T = segs.total
    q, k, v = _bits(rng, T, hq, d), _bits(rng, T, hkv, d), _bits(rng, T, hkv, d)
    do = _bits(rng, T, hq, d)
    scale = 1 / np.sqrt(d)
    announce("bwd small", layout, d, hq, hkv)
    dq, dk, dv = _gpu_grads(segs, q, k, v, do, scale)
    rq, rk, rv = oracle.bwd(f64(q), f64(k), f64(v), f64(do), segs.cu_seqlens,
                            segs.cu_segs, segs.seg_is_query, scale)
    compare("dQ", host_f64(dq), rq)
    compare("dK", host_f64(dk), rk)
    compare("dV", host_f64(dv), rv)


def test_bitwise_repeatable():
    """The backward has no atomics: two runs give identical bits, and the
    deterministic flag (reserved) does not change them."""
    torch = torch_cuda()
    segs = W.segments_from_lengths([W.alternating([100, 300, 80, 200])] * 2)
    rng = np.random.default_rng(12)
    T = segs.total
    q, k, v, do = (_bits(rng, T, 8, 128), _bits(rng, T, 2, 128),
                   _bits(rng, T, 2, 128), _bits(rng, T, 8, 128))
    announce("bwd repeatable")
    a = _gpu_grads(segs, q, k, v, do, 0.088, True)
    b = _gpu_grads(segs, q, k, v, do, 0.088, True)
    c = _gpu_grads(segs, q, k, v, do, 0.088, False)
    for x, y, z in zip(a, b, c):
        assert torch.equal(x, y) and torch.equal(x, z)


def test_workload4_sampled():
    """Full workload 4 (4 x 8192 tokens, 32 heads, d 128) on the GPU; whole
    (dialogue, head) slices of dQ, dK, dV checked against the oracle."""
    torch = torch_cuda()
    from paper_2408_00539_amd import ops
    w = W.make_workload(4)
    announce("bwd workload 4", w.segs.total)
    segs = ops.Segments.from_host(w.segs.cu_seqlens, w.segs.cu_segs,
                                  w.segs.seg_is_query)
    Q, K, V, DO = dev_bf16(w.q), dev_bf16(w.k), dev_bf16(w.v), dev_bf16(w.do)
    o, lse = ops.fwd(Q, K, V, segs, w.scale)
    dq, dk, dv = ops.bwd(Q, K, V, o, lse, DO, segs, w.scale)
    torch.cuda.synchronize()
    for x in (dq, dk, dv):
        assert torch.isfinite(x).all().item()
    pairs = [(0, 0), (3, 29)]
    rq, rk, rv = oracle.bwd(f64(w.q), f64(w.k), f64(w.v), f64(w.do),
                            w.segs.cu_seqlens, w.segs.cu_segs, w.segs.seg_is_query,
                            w.scale, pairs=pairs)
    cu = w.segs.cu_seqlens
    for b, h in pairs:
        s, e = int(cu[b]), int(cu[b + 1])
        compare(f"dQ b{b} h{h}", host_f64(dq[s:e, h]), rq[s:e, h])
        compare(f"dK b{b} h{h}", host_f64(dk[s:e, h]), rk[s:e, h])
        compare(f"dV b{b} h{h}", host_f64(dv[s:e, h]), rv[s:e, h])



def test_mismatched_shapes_raise_before_launch():
    """ops.bwd checks every tensor's shape and the token count against the
    segments before the library is called."""
    torch = torch_cuda()
    from paper_2408_00539_amd import ops
    segs_h = W.segments_from_lengths([W.alternating([20, 30])])
    segs = ops.Segments.from_host(segs_h.cu_seqlens, segs_h.cu_segs, segs_h.seg_is_query)
    T, hq, hkv, d = segs_h.total, 4, 2, 64
    z = lambda *s: torch.zeros(s, dtype=torch.bfloat16, device="cuda")
    q, k, v, o, do = z(T, hq, d), z(T, hkv, d), z(T, hkv, d), z(T, hq, d), z(T, hq, d)
    lse = torch.zeros((hq, T), dtype=torch.float32, device="cuda")
    bad = {"k": (q, z(T - 1, hkv, d), v, o, lse, do), "v": (q, k, z(T, hkv, d + 64), o, lse, do),
           "o": (q, k, v, z(T, hq - 1, d), lse, do), "dout": (q, k, v, o, lse, z(T + 1, hq, d))}
    for name, args in bad.items():
        with pytest.raises(ValueError, match=name):
            ops.bwd(*args, segs)
    other = ops.Segments.from_host(np.array([0, T - 1]), np.array([0, 20, T - 1]),
                                   np.array([1, 0]))
    with pytest.raises(ValueError, match="total_tokens"):
        ops.bwd(q, k, v, o, lse, do, other)
