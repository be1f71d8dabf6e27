"""GPU parity on generated layouts: hypothesis draws packed batches of
dialogues whose segment lengths sit on and around the kernels' tile sizes
(1, 31-33, 63-65, 127-129 and others), with arbitrary query/answer flag
patterns (Eq. 5 for every pattern, R2), head groupings of 1, 2, 4 and 8 and
both head dims, and compares the forward and the backward with the fp64
oracle. Derandomized: the same examples run every time."""

import numpy as np
import pytest

hyp = pytest.importorskip("hypothesis")
from hypothesis import given, settings, strategies as st  # noqa: E402

import oracle  # noqa: E402
from paper_2408_00539_amd import workloads as W  # noqa: E402
from tests._gpu import announce, compare, dev_bf16, f64, host_f64, torch_cuda  # noqa: E402

pytestmark = pytest.mark.gpu

EDGE = [1, 2, 31, 32, 33, 63, 64, 65, 127, 128, 129]
seg_len = st.one_of(st.sampled_from(EDGE), st.integers(1, 200))
dialogue = st.lists(st.tuples(seg_len, st.booleans()), min_size=1, max_size=6)
heads = st.sampled_from([(1, 1), (2, 1), (2, 2), (4, 1), (4, 2), (8, 1), (8, 2), (8, 8)])


@settings(max_examples=60, deadline=None, derandomize=True, database=None)
@given(dialogues=st.lists(dialogue, min_size=1, max_size=3), hh=heads,
       d=st.sampled_from([64, 128]), seed=st.integers(0, 2 ** 31 - 1))
def test_generated_layouts(dialogues, hh, d, seed):
    torch = torch_cuda()
    from paper_2408_00539_amd import ops
    hq, hkv = hh
    segs = W.segments_from_lengths(dialogues)
    T = segs.total
    rng = np.random.default_rng(seed)

    def bits(*shape):
        return W.to_bf16_bits(rng.standard_normal(shape, dtype=np.float32))
    q, k, v, do = bits(T, hq, d), bits(T, hkv, d), bits(T, hkv, d), bits(T, hq, d)
    scale = 1 / np.sqrt(d)
    announce("fuzz", [[n for n, _ in dl] for dl in dialogues], hq, hkv, d, seed)
    dsg = ops.Segments.from_host(segs.cu_seqlens, segs.cu_segs, segs.seg_is_query)
    Q, K, V = dev_bf16(q), dev_bf16(k), dev_bf16(v)
    o, lse = ops.fwd(Q, K, V, dsg, scale)
    dq, dk, dv = ops.bwd(Q, K, V, o, lse, dev_bf16(do), dsg, scale)
    torch.cuda.synchronize()
    args = (segs.cu_seqlens, segs.cu_segs, segs.seg_is_query, scale)
    ro, rl = oracle.fwd(f64(q), f64(k), f64(v), *args)
    rq, rk, rv = oracle.bwd(f64(q), f64(k), f64(v), f64(do), *args)
    compare("O", host_f64(o), ro)
    compare("LSE", host_f64(lse), rl)
    compare("dQ", host_f64(dq), rq)
    compare("dK", host_f64(dk), rk)
    compare("dV", host_f64(dv), rv)
