"""GPU parity of the ChatGLM-style 2-D rotary positions kept under ISM
(Sec. 2.3, prefix-backbone adaptation): positions from the segment layout
(bit-exact), the in-place rotation of bf16 and fp32 tensors and its inverse,
the cached prefill with the rotation fused into the append and the query
load (bit-exact against rotating first, then the plain prefill, and against
the oracle), and training through the rotation (gradients rotated back)."""

import numpy as np
import pytest

import oracle
from oracle.rope2d import positions_2d, rope2d
from paper_2408_00539_amd import workloads as W
from tests._gpu import announce, compare, dev_bf16, f64, host_f64, torch_cuda

pytestmark = pytest.mark.gpu


def _bits(rng, *shape):
    return W.to_bf16_bits(rng.standard_normal(shape, dtype=np.float32))


def _layout():
    return W.segments_from_lengths([W.alternating([40, 70, 33, 65, 1, 129]),
                                    W.alternating([64, 64, 100, 3]),
                                    W.alternating([300])])


def test_positions_match_oracle():
    torch = torch_cuda()
    from paper_2408_00539_amd import ops
    segs = _layout()
    dsg = ops.Segments.from_host(segs.cu_seqlens, segs.cu_segs, segs.seg_is_query)
    announce("positions_2d", segs.total)
    p1, p2 = ops.positions_2d(dsg)
    torch.cuda.synchronize()
    r1, r2 = positions_2d(segs.cu_seqlens, segs.cu_segs)
    np.testing.assert_array_equal(p1.cpu().numpy(), r1)
    np.testing.assert_array_equal(p2.cpu().numpy(), r2)


@pytest.mark.parametrize("d,heads", [(64, 3), (128, 5)])
def test_rotation_bf16_and_fp32(d, heads):
    torch = torch_cuda()
    from paper_2408_00539_amd import ops
    rng = np.random.default_rng(d + heads)
    T = 777
    x = _bits(rng, T, heads, d)
    p1 = rng.integers(0, 60, size=T).astype(np.int32)
    p2 = rng.integers(0, 5000, size=T).astype(np.int32)
    P1, P2 = torch.from_numpy(p1).cuda(), torch.from_numpy(p2).cuda()
    want = rope2d(f64(x), p1, p2)
    announce("rope2d bf16", d, heads)
    xb = ops.rope2d_(dev_bf16(x), P1, P2)
    compare("rotated bf16", host_f64(xb), want)
    announce("rope2d fp32", d, heads)
    xf = torch.from_numpy(f64(x).astype(np.float32)).cuda()
    ops.rope2d_(xf, P1, P2)
    compare("rotated fp32", host_f64(xf), want, max_abs=5e-3, mean_abs=5e-5)
    ops.rope2d_(xf, P1, P2, inverse=True)
    torch.cuda.synchronize()
    compare("inverse of rotated fp32", host_f64(xf), f64(x), max_abs=5e-3, mean_abs=5e-5)


@pytest.mark.parametrize("hq,hkv,d", [(8, 2, 128), (4, 4, 64)])
@pytest.mark.parametrize("seg_is_query", [True, False])
def test_fused_prefill(hq, hkv, d, seg_is_query):
    torch = torch_cuda()
    from paper_2408_00539_amd import ops
    rng = np.random.default_rng(hq + d + int(seg_is_query))
    hist, new, cap = [0, 70, 129, 300], [5, 64, 130, 1], 512
    B = len(hist)
    kc = np.zeros((B, hkv, cap, d), np.uint16)
    vc = np.zeros((B, hkv, cap, d), np.uint16)
    for b, C in enumerate(hist):  # the cache holds rotated keys already
        kc[b, :, :C] = _bits(rng, hkv, C, d)
        vc[b, :, :C] = _bits(rng, hkv, C, d)
    cu = np.concatenate([[0], np.cumsum(new)]).astype(np.int32)
    Tn = int(cu[-1])
    qn, kn, vn = _bits(rng, Tn, hq, d), _bits(rng, Tn, hkv, d), _bits(rng, Tn, hkv, d)
    # positions of the new segment: its index in the dialogue and 0..L-1
    p1 = np.concatenate([np.full(L, 2 * (b + 1), np.int32) for b, L in enumerate(new)])
    p2 = np.concatenate([np.arange(L, dtype=np.int32) for L in new])
    P1, P2 = torch.from_numpy(p1).cuda(), torch.from_numpy(p2).cuda()
    lens = torch.tensor(hist, dtype=torch.int32, device="cuda")
    cu_d = torch.from_numpy(cu).cuda()
    scale = 1 / np.sqrt(d)
    Kf, Vf = dev_bf16(kc), dev_bf16(vc)
    announce("fused rope prefill", hq, hkv, d, seg_is_query)
    of, lf = ops.prefill_cached_rope2d(dev_bf16(qn), dev_bf16(kn), dev_bf16(vn), Kf, Vf, lens,
                                       cu_d, max(new), P1, P2, seg_is_query, scale=scale)
    # unfused: rotate, then the plain cached prefill
    Ku, Vu = dev_bf16(kc), dev_bf16(vc)
    qr = ops.rope2d_(dev_bf16(qn), P1, P2)
    kr = ops.rope2d_(dev_bf16(kn), P1, P2)
    ou, lu = ops.prefill_cached_segment(qr, kr, dev_bf16(vn), Ku, Vu, lens, cu_d, max(new),
                                        seg_is_query, scale)
    torch.cuda.synchronize()
    for a, b in ((of, ou), (Kf, Ku), (Vf, Vu)):
        np.testing.assert_array_equal(a.view(torch.int16).cpu().numpy(),
                                      b.view(torch.int16).cpu().numpy())
    np.testing.assert_array_equal(lf.cpu().numpy(), lu.cpu().numpy())
    of, lf = host_f64(of), host_f64(lf)
    q_rot = rope2d(f64(qn), p1, p2)
    k_rot = rope2d(f64(kn), p1, p2)
    for b, C in enumerate(hist):
        r0, r1 = cu[b], cu[b + 1]
        ro, rl, _, _ = oracle.prefill_cached(
            f64(kc[b, :, :C]).transpose(1, 0, 2), f64(vc[b, :, :C]).transpose(1, 0, 2),
            q_rot[r0:r1], k_rot[r0:r1], f64(vn[r0:r1]), scale, new_is_query=seg_is_query)
        compare(f"O fused b{b}", of[r0:r1], ro)
        compare(f"LSE fused b{b}", lf[:, r0:r1], rl)


@pytest.mark.parametrize("hq,hkv,d", [(4, 2, 128), (2, 1, 64)])
def test_training_through_the_rotation(hq, hkv, d):
    torch = torch_cuda()
    from paper_2408_00539_amd import ops
    rng = np.random.default_rng(5 * hq + d)
    segs = _layout()
    T = segs.total
    q, k, v, do = (_bits(rng, T, hq, d), _bits(rng, T, hkv, d), _bits(rng, T, hkv, d),
                   _bits(rng, T, hq, d))
    dsg = ops.Segments.from_host(segs.cu_seqlens, segs.cu_segs, segs.seg_is_query)
    scale = 1 / np.sqrt(d)
    announce("train through rope", hq, hkv, d)
    P1, P2 = ops.positions_2d(dsg)
    Q, K, V = ops.rope2d_(dev_bf16(q), P1, P2), ops.rope2d_(dev_bf16(k), P1, P2), dev_bf16(v)
    o, lse = ops.fwd(Q, K, V, dsg, scale)
    dq, dk, dv = ops.bwd(Q, K, V, o, lse, dev_bf16(do), dsg, scale)
    ops.rope2d_(dq, P1, P2, inverse=True)
    ops.rope2d_(dk, P1, P2, inverse=True)
    torch.cuda.synchronize()
    p1, p2 = positions_2d(segs.cu_seqlens, segs.cu_segs)
    qr, kr = rope2d(f64(q), p1, p2), rope2d(f64(k), p1, p2)
    ro, _ = oracle.fwd(qr, kr, f64(v), segs.cu_seqlens, segs.cu_segs, segs.seg_is_query, scale)
    gq, gk, gv = oracle.bwd(qr, kr, f64(v), f64(do), segs.cu_seqlens, segs.cu_segs,
                            segs.seg_is_query, scale)
    compare("O", host_f64(o), ro)
    compare("dQ", host_f64(dq), rope2d(gq, p1, p2, inverse=True))
    compare("dK", host_f64(dk), rope2d(gk, p1, p2, inverse=True))
    compare("dV", host_f64(dv), gv)
