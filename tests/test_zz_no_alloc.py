"""ism_attn_decode_noalloc (the decode step for callers that cannot allocate)
against ism_attn_decode, through the C ABI: identical bits on two calls in a
row, the second with a smaller input, and a host-side rejection of inputs
whose split partials exceed the fixed scratch."""

import numpy as np
import pytest

from paper_2408_00539_amd import workloads as W
from tests._gpu import announce, dev_bf16, torch_cuda

pytestmark = pytest.mark.gpu


def _case(rng, B, hq, hkv, d, cap, lens):
    torch = torch_cuda()
    bits = lambda *s: dev_bf16(W.to_bf16_bits(rng.standard_normal(s, dtype=np.float32)))
    kc, vc = bits(B, hkv, cap, d), bits(B, hkv, cap, d)
    q, kn, vn = bits(B, hq, d), bits(B, hkv, d), bits(B, hkv, d)
    pos = torch.tensor(lens, dtype=torch.int32, device="cuda")
    return q, kn, vn, kc, vc, pos


@pytest.mark.parametrize("hq,hkv,d", [(32, 8, 128), (8, 8, 64)])
def test_noalloc_matches_decode_twice(hq, hkv, d):
    torch = torch_cuda()
    from paper_2408_00539_amd import ops
    rng = np.random.default_rng(hq * 7 + d)
    # first call: 6 dialogues; second: 3 dialogues, shorter cache
    for B, cap, lens in ((6, 3000, [2999, 0, 1, 1234, 2048, 777]),
                         (3, 1100, [5, 1099, 640])):
        announce("decode_noalloc", hq, hkv, d, B, cap)
        q, kn, vn, kc, vc, pos = _case(rng, B, hq, hkv, d, cap, lens)
        kc2, vc2 = kc.clone(), vc.clone()
        o_ref, l_ref = ops.decode(q, kn, vn, kc, vc, pos)
        o = torch.empty_like(o_ref)
        l = torch.empty_like(l_ref)
        o.fill_(float("nan"))
        l.fill_(float("nan"))
        ops.decode_noalloc(q, kn, vn, kc2, vc2, pos, out=(o, l))
        torch.cuda.synchronize()
        assert torch.equal(o.view(torch.int16), o_ref.view(torch.int16))
        assert torch.equal(l, l_ref)
        assert torch.equal(kc2.view(torch.int16), kc.view(torch.int16))
        assert torch.equal(vc2.view(torch.int16), vc.view(torch.int16))


def test_noalloc_rejects_partials_beyond_scratch():
    """64 dialogues x 64 heads x 64 splits x (128 + 2) x 4 bytes is far above
    the scratch: refused before any launch, outputs untouched."""
    torch = torch_cuda()
    from paper_2408_00539_amd import ops
    B, hq, hkv, d, cap = 64, 64, 64, 128, 64
    q = torch.zeros((B, hq, d), dtype=torch.bfloat16, device="cuda")
    kn = torch.zeros((B, hkv, d), dtype=torch.bfloat16, device="cuda")
    kc = torch.zeros((B, hkv, cap, d), dtype=torch.bfloat16, device="cuda")
    pos = torch.zeros(B, dtype=torch.int32, device="cuda")
    o = torch.full((B, hq, d), 7.0, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(ops.IsmError, match="ISM_ERR_WORKSPACE"):
        ops.decode_noalloc(q, kn, kn, kc, kc, pos, num_splits=64, return_lse=False,
                           out=(o, None))
    torch.cuda.synchronize()
    assert bool((o.float() == 7.0).all())
