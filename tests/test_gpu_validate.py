"""ISM_VALIDATE=1: the entry points copy their device boundary arrays to the
host and reject malformed ones before any launch (outputs untouched); valid
ones give the same results as without validation.

The malformed inputs are chosen so that even unvalidated they would keep
every access inside the tensors: a dialogue boundary moved one token into a
segment (lim of that token then points past its dialogue's end but not past
the batch), and a dialogue with more new tokens than max_new (rows past
max_new are simply not covered)."""

import numpy as np
import pytest

from paper_2408_00539_amd import workloads as W
from tests._gpu import announce, torch_cuda

pytestmark = pytest.mark.gpu

ISM_ERR_SEGMENTS = 4


def _randn(torch, g, *shape):
    return torch.randn(shape, generator=g, device="cuda").to(torch.bfloat16)


def test_validate_packed_boundaries(monkeypatch):
    torch = torch_cuda()
    from paper_2408_00539_amd import ops
    segs = W.segments_from_lengths([W.alternating([40, 70, 30]), W.alternating([50, 20])])
    T, hq, hkv, d = segs.total, 2, 1, 64
    g = torch.Generator(device="cuda")
    g.manual_seed(30)
    q, k, v, do = (_randn(torch, g, T, hq, d), _randn(torch, g, T, hkv, d),
                   _randn(torch, g, T, hkv, d), _randn(torch, g, T, hq, d))
    sc = d ** -0.5
    announce("validate packed", T, hq, hkv, d)
    good = ops.Segments.from_host(segs.cu_seqlens, segs.cu_segs, segs.seg_is_query)
    monkeypatch.delenv("ISM_VALIDATE", raising=False)
    o_ref, lse_ref = ops.fwd(q, k, v, good, sc)
    dq_ref, dk_ref, dv_ref = ops.bwd(q, k, v, o_ref, lse_ref, do, good, sc)
    monkeypatch.setenv("ISM_VALIDATE", "1")
    o, lse = ops.fwd(q, k, v, good, sc)
    dq, dk, dv = ops.bwd(q, k, v, o, lse, do, good, sc)
    torch.cuda.synchronize()
    for a, b in ((o, o_ref), (lse, lse_ref), (dq, dq_ref), (dk, dk_ref), (dv, dv_ref)):
        assert torch.equal(a, b)
    cu = np.array(segs.cu_seqlens, dtype=np.int32)
    cu[1] += 1  # no longer a segment boundary
    bad = ops.Segments.from_host(cu, segs.cu_segs, segs.seg_is_query)
    nan = float("nan")
    o2 = torch.full_like(o_ref, nan)
    lse2 = torch.full_like(lse_ref, nan)
    with pytest.raises(ops.IsmError) as ei:
        ops.fwd(q, k, v, bad, sc, out=(o2, lse2))
    assert ei.value.status == ISM_ERR_SEGMENTS, ei.value
    grads = tuple(torch.full_like(x, nan) for x in (dq_ref, dk_ref, dv_ref))
    with pytest.raises(ops.IsmError) as ei:
        ops.bwd(q, k, v, o_ref, lse_ref, do, bad, sc, out=grads)
    assert ei.value.status == ISM_ERR_SEGMENTS, ei.value
    with pytest.raises(ops.IsmError) as ei:
        ops.visibility(bad)
    assert ei.value.status == ISM_ERR_SEGMENTS, ei.value
    with pytest.raises(ops.IsmError) as ei:
        ops.positions_2d(bad)
    assert ei.value.status == ISM_ERR_SEGMENTS, ei.value
    torch.cuda.synchronize()
    for x in (o2, lse2) + grads:
        assert bool(torch.isnan(x.float()).all())  # nothing launched


def test_validate_new_token_boundaries(monkeypatch):
    torch = torch_cuda()
    from paper_2408_00539_amd import ops
    B, hq, hkv, d, cap = 2, 4, 2, 128, 256
    g = torch.Generator(device="cuda")
    g.manual_seed(31)
    kc, vc = _randn(torch, g, B, hkv, cap, d), _randn(torch, g, B, hkv, cap, d)
    lens = torch.tensor([100, 60], dtype=torch.int32, device="cuda")
    cu = torch.tensor([0, 50, 80], dtype=torch.int32, device="cuda")
    Tn = 80
    qn, kn, vn = _randn(torch, g, Tn, hq, d), _randn(torch, g, Tn, hkv, d), _randn(torch, g, Tn, hkv, d)
    sc = d ** -0.5
    announce("validate prefill", B, hq, hkv, d, cap)
    monkeypatch.setenv("ISM_VALIDATE", "1")
    kc0, vc0 = kc.clone(), vc.clone()
    o_ok, lse_ok = ops.prefill_cached(qn, kn, vn, kc, vc, lens, cu, 50, sc)
    monkeypatch.delenv("ISM_VALIDATE")
    kc1, vc1 = kc0.clone(), vc0.clone()
    o_ref, lse_ref = ops.prefill_cached(qn, kn, vn, kc1, vc1, lens, cu, 50, sc)
    torch.cuda.synchronize()
    assert torch.equal(o_ok, o_ref) and torch.equal(lse_ok, lse_ref)
    assert torch.equal(kc, kc1) and torch.equal(vc, vc1)
    # dialogue 0 has 50 new tokens, more than max_new = 40
    monkeypatch.setenv("ISM_VALIDATE", "1")
    kc2, vc2 = kc0.clone(), vc0.clone()
    o2 = torch.full_like(o_ref, float("nan"))
    lse2 = torch.full_like(lse_ref, float("nan"))
    with pytest.raises(ops.IsmError) as ei:
        ops.prefill_cached(qn, kn, vn, kc2, vc2, lens, cu, 40, sc, out=(o2, lse2))
    assert ei.value.status == ISM_ERR_SEGMENTS, ei.value
    torch.cuda.synchronize()
    assert bool(torch.isnan(o2.float()).all()) and bool(torch.isnan(lse2).all())
    assert torch.equal(kc2, kc0) and torch.equal(vc2, vc0)  # nothing appended
