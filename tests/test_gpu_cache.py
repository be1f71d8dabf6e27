"""GPU parity of the KV-cache reuse path: ism_attn_prefill_cached and
ism_attn_decode against the oracle's stepwise cache path and one-shot
forward (Sec. 2.3 of the paper)."""

import numpy as np
import pytest

import oracle
from paper_2408_00539_amd import workloads as W
from tests._gpu import announce, compare, dev_bf16, f64, host_f64, torch_cuda

pytestmark = pytest.mark.gpu


def _bits(rng, *shape):
    return W.to_bf16_bits(rng.standard_normal(shape, dtype=np.float32))


def _setup(rng, hist, new, hq, hkv, d, cap):
    """Caches [B, hkv, cap, d] with len(hist[b]) history tokens, new segments."""
    B = len(hist)
    kc = np.zeros((B, hkv, cap, d), np.uint16)
    vc = np.zeros((B, hkv, cap, d), np.uint16)
    # poison the unused tail so that reading past the valid range is visible
    kc[...] = W.to_bf16_bits(np.array([1000.0], np.float32))[0]
    vc[...] = W.to_bf16_bits(np.array([1000.0], np.float32))[0]
    for b, C in enumerate(hist):
        kc[b, :, :C] = _bits(rng, hkv, C, d)
        vc[b, :, :C] = _bits(rng, hkv, C, d)
    cu_new = np.concatenate([[0], np.cumsum(new)]).astype(np.int32)
    Tn = int(cu_new[-1])
    return kc, vc, cu_new, _bits(rng, Tn, hq, d), _bits(rng, Tn, hkv, d), \
        _bits(rng, Tn, hkv, d)


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("hq,hkv", [(2, 2), (4, 2), (8, 2), (4, 1), (8, 1),
                                    (3, 1), (12, 1), (16, 2), (6, 3), (5, 1), (32, 1),
                                    (64, 1)])
def test_prefill_then_decode_small(d, hq, hkv):
    torch = torch_cuda()
    from paper_2408_00539_amd import ops
    rng = np.random.default_rng(d * 100 + hq * 10 + hkv)
    hist = [0, 1, 63, 64, 65, 300]
    new = [5, 64, 1, 129, 65, 200]
    steps, cap = 9, 640
    kc, vc, cu_new, qn, kn, vn = _setup(rng, hist, new, hq, hkv, d, cap)
    scale = 1 / np.sqrt(d)
    announce("prefill small", d, hq, hkv)
    Kc, Vc = dev_bf16(kc), dev_bf16(vc)
    lens = torch.tensor(hist, dtype=torch.int32, device="cuda")
    o, lse = ops.prefill_cached(dev_bf16(qn), dev_bf16(kn), dev_bf16(vn), Kc, Vc,
                                lens, torch.from_numpy(cu_new).cuda(), max(new),
                                scale)
    torch.cuda.synchronize()
    o, lse = host_f64(o), host_f64(lse)
    kcache_ref = [None] * len(hist)
    vcache_ref = [None] * len(hist)
    for b, C in enumerate(hist):
        r0, r1 = cu_new[b], cu_new[b + 1]
        ro, rl, kk, vv = oracle.prefill_cached(
            f64(kc[b, :, :C]).transpose(1, 0, 2), f64(vc[b, :, :C]).transpose(1, 0, 2),
            f64(qn[r0:r1]), f64(kn[r0:r1]), f64(vn[r0:r1]), scale)
        compare(f"O prefill b{b}", o[r0:r1], ro)
        compare(f"LSE prefill b{b}", lse[:, r0:r1], rl)
        kcache_ref[b], vcache_ref[b] = kk, vv
    # the append wrote exactly the new rows, bit for bit, and nothing else
    Kh = Kc.view(torch.int16).cpu().numpy().view(np.uint16)
    for b, C in enumerate(hist):
        r0, r1 = cu_new[b], cu_new[b + 1]
        np.testing.assert_array_equal(Kh[b, :, C:C + new[b]],
                                      kn[r0:r1].transpose(1, 0, 2))
        np.testing.assert_array_equal(Kh[b, :, :C], kc[b, :, :C])
        np.testing.assert_array_equal(Kh[b, :, C + new[b]:], kc[b, :, C + new[b]:])

    pos = np.array([C + n for C, n in zip(hist, new)], np.int32)
    B = len(hist)
    for t in range(steps):
        q = _bits(rng, B, hq, d)
        k = _bits(rng, B, hkv, d)
        v = _bits(rng, B, hkv, d)
        announce("decode step", t)
        od, ld = ops.decode(dev_bf16(q), dev_bf16(k), dev_bf16(v), Kc, Vc,
                            torch.from_numpy(pos).cuda(), 0, scale,
                            num_splits=[0, 1, 3][t % 3])
        torch.cuda.synchronize()
        od, ld = host_f64(od), host_f64(ld)
        for b in range(B):
            ro, rl, kcache_ref[b], vcache_ref[b] = oracle.decode_step(
                kcache_ref[b], vcache_ref[b], f64(q[b]), f64(k[b]), f64(v[b]), scale)
            compare(f"O decode t{t} b{b}", od[b], ro)
            compare(f"LSE decode t{t} b{b}", ld[:, b], rl)
        pos += 1


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("hq,hkv", [(2, 2), (8, 2)])
def test_prefill_answer_segment_small(d, hq, hkv):
    """ism_attn_prefill_cached_segment with an answer segment (Eq. 5 third
    case: new row r sees the cache and new rows 0..r) against the oracle;
    the query form of the same entry point against the query oracle."""
    torch = torch_cuda()
    from paper_2408_00539_amd import ops
    rng = np.random.default_rng(7 * d + hq)
    hist = [0, 1, 64, 65, 300, 127]
    new = [1, 64, 130, 65, 200, 33]
    cap = 640
    scale = 1 / np.sqrt(d)
    for isq in (False, True):
        kc, vc, cu_new, qn, kn, vn = _setup(rng, hist, new, hq, hkv, d, cap)
        announce("prefill segment", "query" if isq else "answer", d, hq, hkv)
        o, lse = ops.prefill_cached_segment(
            dev_bf16(qn), dev_bf16(kn), dev_bf16(vn), dev_bf16(kc), dev_bf16(vc),
            torch.tensor(hist, dtype=torch.int32, device="cuda"),
            torch.from_numpy(cu_new).cuda(), max(new), isq, scale)
        torch.cuda.synchronize()
        o, lse = host_f64(o), host_f64(lse)
        for b, C in enumerate(hist):
            r0, r1 = cu_new[b], cu_new[b + 1]
            ro, rl, _, _ = oracle.prefill_cached(
                f64(kc[b, :, :C]).transpose(1, 0, 2),
                f64(vc[b, :, :C]).transpose(1, 0, 2),
                f64(qn[r0:r1]), f64(kn[r0:r1]), f64(vn[r0:r1]), scale,
                new_is_query=isq)
            compare(f"O b{b} q={isq}", o[r0:r1], ro)
            compare(f"LSE b{b} q={isq}", lse[:, r0:r1], rl)


@pytest.mark.parametrize("hq,hkv,B,cap", [(4, 4, 3, 2048), (16, 2, 3, 2048),
                                           (16, 16, 32, 640), (32, 16, 32, 640),
                                           (48, 16, 32, 640)])
def test_decode_split_counts_agree(hq, hkv, B, cap):
    """Any split count merges to the same result (exact merge, R19), for the
    matrix-core kernel (steps of few (dialogue, KV head) slabs: one and 8
    query heads per KV head) and the vector kernel (512 slabs: 1, 2 and 3
    query heads per KV head); with 64 splits most chunks of the shorter
    dialogues are empty."""
    torch = torch_cuda()
    from paper_2408_00539_amd import ops
    rng = np.random.default_rng(77 + hq + B)
    d = 128
    kc = _bits(rng, B, hkv, cap, d)
    vc = _bits(rng, B, hkv, cap, d)
    if B == 3:
        pos = np.array([0, 1000, 2047], np.int32)
    else:  # chunk and tile edges, the last position, and random ones
        pos = rng.integers(0, cap, B).astype(np.int32)
        pos[:6] = [0, 1, 31, 32, 255, 256]
        pos[-1] = cap - 1
    q, k, v = _bits(rng, B, hq, d), _bits(rng, B, hkv, d), _bits(rng, B, hkv, d)
    outs = []
    for splits in [1, 2, 7, 16, 64]:
        announce("decode splits", hq, hkv, B, splits)
        Kc, Vc = dev_bf16(kc), dev_bf16(vc)
        o, l = ops.decode(dev_bf16(q), dev_bf16(k), dev_bf16(v), Kc, Vc,
                          torch.from_numpy(pos).cuda(), 0, 1 / np.sqrt(d),
                          num_splits=splits)
        torch.cuda.synchronize()
        outs.append((host_f64(o), host_f64(l)))
    for b in range(B):
        p = pos[b]
        kk = np.concatenate([f64(kc[b, :, :p]).transpose(1, 0, 2), f64(k[b])[None]])
        vv = np.concatenate([f64(vc[b, :, :p]).transpose(1, 0, 2), f64(v[b])[None]])
        ro, rl, _, _ = oracle.decode_step(kk[:-1], vv[:-1], f64(q[b]), f64(k[b]),
                                          f64(v[b]), 1 / np.sqrt(d))
        for o, l in outs:
            compare(f"O b{b}", o[b], ro)
            compare(f"LSE b{b}", l[:, b], rl)


def test_workload3_one_shot_rows():
    """Full workload 3 on the GPU (32 dialogues, 8192 cached tokens, new
    query segment, 256 decode steps); sampled dialogues are checked against
    the one-shot oracle forward over [history; Q_n; A_n] (P-10 on device)."""
    torch = torch_cuda()
    from paper_2408_00539_amd import ops
    w = W.make_workload(3)
    announce("workload 3 prefill", int(w.cu_new[-1]))
    Kc, Vc = dev_bf16(w.k_cache), dev_bf16(w.v_cache)
    B = len(w.new_lens)
    lens = torch.full((B,), w.hist_len, dtype=torch.int32, device="cuda")
    o, lse = ops.prefill_cached(dev_bf16(w.q_new), dev_bf16(w.k_new),
                                dev_bf16(w.v_new), Kc, Vc, lens,
                                torch.from_numpy(w.cu_new).cuda(),
                                int(w.new_lens.max()), w.scale)
    pos = lens + torch.from_numpy(w.new_lens).cuda()
    qd, kd, vd = dev_bf16(w.q_dec), dev_bf16(w.k_dec), dev_bf16(w.v_dec)
    od = torch.empty_like(qd)
    ld = torch.empty((w.steps, w.hq, B), dtype=torch.float32, device="cuda")
    announce("workload 3 decode", w.steps)
    for t in range(w.steps):
        od[t], ld[t] = ops.decode(qd[t], kd[t], vd[t], Kc, Vc, pos, 0, w.scale)
        pos += 1
    torch.cuda.synchronize()
    del Kc, Vc

    # the same turn through a paged cache (pages of 256 scattered over a
    # shuffled pool) gives the same bits
    ps = 256
    mp = w.cache_cap // ps
    table = torch.from_numpy(np.random.default_rng(9).permutation(B * mp + 5)[:B * mp]
                             .astype(np.int32).reshape(B, mp)).cuda()

    def pool_of(c):
        c = dev_bf16(c)
        pool = torch.zeros((B * mp + 5, w.hkv, ps, w.d), dtype=c.dtype, device="cuda")
        pool[table.view(-1).long()] = (c.view(B, w.hkv, mp, ps, w.d).permute(0, 2, 1, 3, 4)
                                       .reshape(B * mp, w.hkv, ps, w.d))
        return pool
    Kp, Vp = pool_of(w.k_cache), pool_of(w.v_cache)
    announce("workload 3 paged prefill and decode")
    op, lp = ops.prefill_paged(dev_bf16(w.q_new), dev_bf16(w.k_new), dev_bf16(w.v_new), Kp, Vp,
                               table, lens, torch.from_numpy(w.cu_new).cuda(),
                               int(w.new_lens.max()), True, w.scale)
    pos = lens + torch.from_numpy(w.new_lens).cuda()
    same = True
    for t in range(w.steps):
        o_t, l_t = ops.decode_paged(qd[t], kd[t], vd[t], Kp, Vp, table, pos, 0, w.scale)
        same &= bool(torch.equal(o_t.view(torch.int16), od[t].view(torch.int16)))
        same &= bool(torch.equal(l_t, ld[t]))
        pos += 1
    torch.cuda.synchronize()
    assert torch.equal(op.view(torch.int16), o.view(torch.int16)) and torch.equal(lp, lse)
    assert same, "paged decode differs from the dense decode"
    del Kp, Vp
    for b in (0, 13, 31):
        C, L, S = w.hist_len, int(w.new_lens[b]), w.steps
        dia = W.segments_from_lengths([
            [(int(n), bool(f)) for n, f in zip(
                np.diff(w.hist.cu_segs[b * 32:(b + 1) * 32 + 1]),
                w.hist.seg_is_query[b * 32:(b + 1) * 32])] + [(L, True), (S, False)]])
        n = C + L + S
        kk = np.concatenate([f64(w.k_cache[b, :, :C]).transpose(1, 0, 2),
                             f64(w.k_new[w.cu_new[b]:w.cu_new[b + 1]]),
                             f64(w.k_dec[:, b])])
        vv = np.concatenate([f64(w.v_cache[b, :, :C]).transpose(1, 0, 2),
                             f64(w.v_new[w.cu_new[b]:w.cu_new[b + 1]]),
                             f64(w.v_dec[:, b])])
        qq = np.zeros((n, w.hq, w.d))
        qq[C:C + L] = f64(w.q_new[w.cu_new[b]:w.cu_new[b + 1]])
        qq[C + L:] = f64(w.q_dec[:, b])
        for h in (0, 21):
            ro, rl = oracle.fwd_rows(qq, kk, vv, dia.cu_seqlens, dia.cu_segs,
                                     dia.seg_is_query, w.scale, 0, h, rows=(C, n))
            r0, r1 = w.cu_new[b], w.cu_new[b + 1]
            compare(f"O prefill b{b} h{h}", host_f64(o[r0:r1, h]), ro[:L])
            compare(f"LSE prefill b{b} h{h}", host_f64(lse[h, r0:r1]), rl[:L])
            compare(f"O decode b{b} h{h}", host_f64(od[:, b, h]), ro[L:])
            compare(f"LSE decode b{b} h{h}", host_f64(ld[:, h, b]), rl[L:])


def test_out_of_capacity_dialogues_get_nan():
    """Out of contract (the lengths live on the device, so the host cannot
    refuse them): a dialogue whose new segment would end past the cache, or
    whose decode position lies outside it, gets NaN in all its rows and
    nothing of it is written outside the cache; the other dialogues are
    unaffected."""
    torch = torch_cuda()
    from paper_2408_00539_amd import ops
    rng = np.random.default_rng(31)
    hq = hkv = 2
    d, cap = 64, 256
    hist, new = [10, 250, 100], [20, 20, 20]   # dialogue 1 ends at 270 > 256
    kc, vc, cu_new, qn, kn, vn = _setup(rng, hist, new, hq, hkv, d, cap)
    Kc, Vc = dev_bf16(kc), dev_bf16(vc)
    announce("prefill out of capacity")
    o, lse = ops.prefill_cached(dev_bf16(qn), dev_bf16(kn), dev_bf16(vn), Kc, Vc,
                                torch.tensor(hist, dtype=torch.int32, device="cuda"),
                                torch.from_numpy(cu_new).cuda(), max(new), 0.125)
    torch.cuda.synchronize()
    o, lse = host_f64(o), host_f64(lse)
    assert np.all(np.isnan(o[cu_new[1]:cu_new[2]])) and np.all(np.isnan(lse[:, cu_new[1]:cu_new[2]]))
    for b in (0, 2):
        r0, r1 = cu_new[b], cu_new[b + 1]
        C = hist[b]
        ro, rl, _, _ = oracle.prefill_cached(
            f64(kc[b, :, :C]).transpose(1, 0, 2), f64(vc[b, :, :C]).transpose(1, 0, 2),
            f64(qn[r0:r1]), f64(kn[r0:r1]), f64(vn[r0:r1]), 0.125)
        compare(f"O b{b}", o[r0:r1], ro)
        compare(f"LSE b{b}", lse[:, r0:r1], rl)
    Kh = Kc.view(torch.int16).cpu().numpy().view(np.uint16)
    # dialogue 1: the six positions 250..255 inside the cache were appended
    np.testing.assert_array_equal(Kh[1, :, 250:256],
                                  kn[cu_new[1]:cu_new[1] + 6].transpose(1, 0, 2))
    np.testing.assert_array_equal(Kh[1, :, :250], kc[1, :, :250])

    # decode: positions cap (past the end) and -1 are out of contract
    pos = torch.tensor([cap, 40, -1], dtype=torch.int32, device="cuda")
    q, k, v = _bits(rng, 3, hq, d), _bits(rng, 3, hkv, d), _bits(rng, 3, hkv, d)
    before = Kc.clone()
    announce("decode out of capacity")
    od, ld = ops.decode(dev_bf16(q), dev_bf16(k), dev_bf16(v), Kc, Vc, pos, 0, 0.125)
    torch.cuda.synchronize()
    od, ld = host_f64(od), host_f64(ld)
    assert np.all(np.isnan(od[0])) and np.all(np.isnan(od[2]))
    assert np.all(np.isnan(ld[:, 0])) and np.all(np.isnan(ld[:, 2]))
    assert np.all(np.isfinite(od[1])) and np.all(np.isfinite(ld[:, 1]))
    after = Kc.view(torch.int16).cpu().numpy()
    bef = before.view(torch.int16).cpu().numpy()
    np.testing.assert_array_equal(after[0], bef[0])
    np.testing.assert_array_equal(after[2], bef[2])
