"""GPU parity of the paged KV cache (ism_attn_prefill_paged,
ism_attn_decode_paged): the same turns as the dense cache path (Sec. 2.3:
reuse the history cache, append the new segment, then decode the answer one
token at a time), with the cache held in shuffled pages of a shared pool.

Each result is compared with the fp64 oracle on the logical cache, and with
the dense entry points on the same inputs: the kernels visit the same keys in
the same order (the decode cuts each dialogue's key range at the same
chunks), so the two must agree bit for bit. The pages the appends wrote are
read back and compared with the dense cache.
"""

import numpy as np
import pytest

import oracle
from paper_2408_00539_amd import workloads as W
from tests._gpu import announce, compare, dev_bf16, f64, host_f64, torch_cuda

pytestmark = pytest.mark.gpu


def _bits(rng, *shape):
    return W.to_bf16_bits(rng.standard_normal(shape, dtype=np.float32))


def _paged_pool(rng, kc, page_size, spare=3):
    """Scatter dense caches [B, hkv, cap, d] into a shuffled page pool.
    Returns (pool_k [P, hkv, ps, d], block_table [B, cap // ps])."""
    B, hkv, cap, d = kc.shape
    mp = cap // page_size
    P = B * mp + spare
    order = rng.permutation(P)[:B * mp].reshape(B, mp).astype(np.int32)
    pool = np.zeros((P, hkv, page_size, d), np.uint16)
    pool[...] = W.to_bf16_bits(np.array([-777.0], np.float32))[0]
    for b in range(B):
        for j in range(mp):
            pool[order[b, j]] = kc[b, :, j * page_size:(j + 1) * page_size]
    return pool, order


def _gather_dense(pool, table):
    B, mp = table.shape
    _, hkv, ps, d = pool.shape
    out = np.empty((B, hkv, mp * ps, d), pool.dtype)
    for b in range(B):
        for j in range(mp):
            out[b, :, j * ps:(j + 1) * ps] = pool[table[b, j]]
    return out


@pytest.mark.parametrize("page_size", [64, 128])
@pytest.mark.parametrize("hq,hkv,d", [(4, 4, 128), (8, 2, 128), (4, 1, 64), (4, 2, 64),
                                      (8, 1, 128), (8, 1, 64)])
@pytest.mark.parametrize("seg_is_query", [True, False])
def test_paged_turn_matches_dense_and_oracle(page_size, hq, hkv, d, seg_is_query):
    torch = torch_cuda()
    from paper_2408_00539_amd import ops
    rng = np.random.default_rng(page_size + 7 * hq + d + int(seg_is_query))
    hist = [0, 1, 63, 64, 130, 300]
    new = [5, 64, 1, 129, 65, 77]
    steps, cap = 6, 512
    B = len(hist)
    kc = np.zeros((B, hkv, cap, d), np.uint16)
    vc = np.zeros((B, hkv, cap, d), np.uint16)
    for b, C in enumerate(hist):
        kc[b, :, :C] = _bits(rng, hkv, C, d)
        vc[b, :, :C] = _bits(rng, hkv, C, d)
    cu_new = np.concatenate([[0], np.cumsum(new)]).astype(np.int32)
    Tn = int(cu_new[-1])
    qn, kn, vn = _bits(rng, Tn, hq, d), _bits(rng, Tn, hkv, d), _bits(rng, Tn, hkv, d)
    pk, table = _paged_pool(rng, kc, page_size)
    pv = np.zeros_like(pk)  # V in the pages of K's table
    for b in range(B):
        for j in range(table.shape[1]):
            pv[table[b, j]] = vc[b, :, j * page_size:(j + 1) * page_size]
    scale = 1 / np.sqrt(d)
    lens = torch.tensor(hist, dtype=torch.int32, device="cuda")
    cu = torch.from_numpy(cu_new).cuda()
    Kd, Vd = dev_bf16(kc), dev_bf16(vc)
    Kp, Vp = dev_bf16(pk), dev_bf16(pv)
    tab = torch.from_numpy(table).cuda()
    announce("paged prefill", page_size, hq, hkv, d, seg_is_query)
    od, ld = ops.prefill_cached_segment(dev_bf16(qn), dev_bf16(kn), dev_bf16(vn), Kd, Vd,
                                        lens, cu, max(new), seg_is_query, scale)
    op, lp = ops.prefill_paged(dev_bf16(qn), dev_bf16(kn), dev_bf16(vn), Kp, Vp, tab, lens,
                               cu, max(new), seg_is_query, scale)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(op.view(torch.int16).cpu().numpy(),
                                  od.view(torch.int16).cpu().numpy())
    np.testing.assert_array_equal(lp.cpu().numpy(), ld.cpu().numpy())
    op, lp = host_f64(op), host_f64(lp)
    for b, C in enumerate(hist):
        r0, r1 = cu_new[b], cu_new[b + 1]
        ro, rl, _, _ = oracle.prefill_cached(
            f64(kc[b, :, :C]).transpose(1, 0, 2), f64(vc[b, :, :C]).transpose(1, 0, 2),
            f64(qn[r0:r1]), f64(kn[r0:r1]), f64(vn[r0:r1]), scale, new_is_query=seg_is_query)
        compare(f"O paged b{b}", op[r0:r1], ro)
        compare(f"LSE paged b{b}", lp[:, r0:r1], rl)
    # the appends wrote the same cache contents through the pages
    back = _gather_dense(Kp.view(torch.int16).cpu().numpy().view(np.uint16), table)
    np.testing.assert_array_equal(back, Kd.view(torch.int16).cpu().numpy().view(np.uint16))

    # decode: paged against the dense entry point and the oracle's stepwise path
    kref, vref = [], []
    for b, C in enumerate(hist):
        r0, r1 = cu_new[b], cu_new[b + 1]
        kref.append(np.concatenate([f64(kc[b, :, :C]).transpose(1, 0, 2), f64(kn[r0:r1])]))
        vref.append(np.concatenate([f64(vc[b, :, :C]).transpose(1, 0, 2), f64(vn[r0:r1])]))
    pos = np.array([C + n for C, n in zip(hist, new)], np.int32)
    for t in range(steps):
        q, k, v = _bits(rng, B, hq, d), _bits(rng, B, hkv, d), _bits(rng, B, hkv, d)
        announce("paged decode step", t)
        p_dev = torch.from_numpy(pos).cuda()
        splits = [0, 1, 3][t % 3]
        od, ld = ops.decode(dev_bf16(q), dev_bf16(k), dev_bf16(v), Kd, Vd, p_dev, 0, scale,
                            num_splits=splits)
        opd, lpd = ops.decode_paged(dev_bf16(q), dev_bf16(k), dev_bf16(v), Kp, Vp, tab, p_dev,
                                    0, scale, num_splits=splits)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(opd.view(torch.int16).cpu().numpy(),
                                      od.view(torch.int16).cpu().numpy())
        np.testing.assert_array_equal(lpd.cpu().numpy(), ld.cpu().numpy())
        opd, lpd = host_f64(opd), host_f64(lpd)
        for b in range(B):
            ro, rl, kref[b], vref[b] = oracle.decode_step(kref[b], vref[b], f64(q[b]),
                                                          f64(k[b]), f64(v[b]), scale)
            compare(f"O paged decode t{t} b{b}", opd[b], ro)
            compare(f"LSE paged decode t{t} b{b}", lpd[:, b], rl)
        pos += 1
    back = _gather_dense(Kp.view(torch.int16).cpu().numpy().view(np.uint16), table)
    np.testing.assert_array_equal(back, Kd.view(torch.int16).cpu().numpy().view(np.uint16))
    backv = _gather_dense(Vp.view(torch.int16).cpu().numpy().view(np.uint16), table)
    np.testing.assert_array_equal(backv, Vd.view(torch.int16).cpu().numpy().view(np.uint16))
