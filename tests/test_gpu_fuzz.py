"""GPU parity on generated layouts: hypothesis draws packed batches of
dialogues whose segment lengths sit on and around the kernels' tile sizes
(1, 31-33, 63-65, 127-129 and others), with arbitrary query/answer flag
patterns (Eq. 5 for every pattern, R2), head groupings of 1, 2, 3, 4 and 8
and both head dims, and compares the forward and the backward with the fp64
oracle; the cache-path tests add groupings of 5, 6, 12 and 16 query heads
per KV head (the decode's matrix-core sets), and decode steps of 512
(dialogue, KV head) slabs exercise the vector decode kernel. Derandomized:
the same examples run every time."""

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
heads = st.sampled_from([(1, 1), (2, 1), (2, 2), (4, 1), (4, 2), (8, 1), (8, 2), (8, 8),
                         (3, 1), (6, 2)])
cache_heads = st.sampled_from([(1, 1), (2, 1), (2, 2), (4, 1), (4, 2), (8, 1), (8, 2), (8, 8),
                               (3, 1), (5, 1), (6, 1), (12, 2), (16, 1)])


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


hist_len = st.one_of(st.sampled_from([0, 1, 63, 64, 65, 127, 128, 129, 255, 256, 257]),
                     st.integers(0, 400))
new_len = st.one_of(st.sampled_from([1, 2, 31, 32, 33, 63, 64, 65]), st.integers(1, 150))


@settings(max_examples=40, deadline=None, derandomize=True, database=None)
@given(turns=st.lists(st.tuples(hist_len, new_len), min_size=1, max_size=4),
       is_query=st.booleans(), hh=cache_heads, d=st.sampled_from([64, 128]),
       splits=st.sampled_from([0, 1, 3, 64]), seed=st.integers(0, 2 ** 31 - 1))
def test_generated_cache_turns(turns, is_query, hh, d, splits, seed):
    """Cached prefill of a query or answer segment over generated histories,
    then two decode steps, against the oracle's stepwise path (Sec. 2.3)."""
    torch = torch_cuda()
    from paper_2408_00539_amd import ops
    hq, hkv = hh
    rng = np.random.default_rng(seed)

    def bits(*shape):
        return W.to_bf16_bits(rng.standard_normal(shape, dtype=np.float32))
    hist = [h for h, _ in turns]
    new = [n for _, n in turns]
    B, cap = len(turns), 640
    kc = np.zeros((B, hkv, cap, d), np.uint16)
    vc = np.zeros((B, hkv, cap, d), np.uint16)
    for b, C in enumerate(hist):
        kc[b, :, :C] = bits(hkv, C, d)
        vc[b, :, :C] = bits(hkv, C, d)
    cu = np.concatenate([[0], np.cumsum(new)]).astype(np.int32)
    Tn = int(cu[-1])
    qn, kn, vn = bits(Tn, hq, d), bits(Tn, hkv, d), bits(Tn, hkv, d)
    scale = 1 / np.sqrt(d)
    announce("fuzz cache", turns, is_query, hq, hkv, d, splits, seed)
    Kc, Vc = dev_bf16(kc), dev_bf16(vc)
    lens = torch.tensor(hist, dtype=torch.int32, device="cuda")
    o, lse = ops.prefill_cached_segment(dev_bf16(qn), dev_bf16(kn), dev_bf16(vn), Kc, Vc, lens,
                                        torch.from_numpy(cu).cuda(), max(new), is_query, scale)
    torch.cuda.synchronize()
    o, lse = host_f64(o), host_f64(lse)
    kref, vref = [], []
    for b, C in enumerate(hist):
        r0, r1 = cu[b], cu[b + 1]
        ro, rl, kk, vv = oracle.prefill_cached(
            f64(kc[b, :, :C]).transpose(1, 0, 2), f64(vc[b, :, :C]).transpose(1, 0, 2),
            f64(qn[r0:r1]), f64(kn[r0:r1]), f64(vn[r0:r1]), scale, new_is_query=is_query)
        compare(f"O prefill b{b}", o[r0:r1], ro)
        compare(f"LSE prefill b{b}", lse[:, r0:r1], rl)
        kref.append(kk)
        vref.append(vv)
    pos = torch.tensor([h + n for h, n in turns], dtype=torch.int32, device="cuda")
    for t in range(2):
        q, k, v = bits(B, hq, d), bits(B, hkv, d), bits(B, hkv, d)
        od, ld = ops.decode(dev_bf16(q), dev_bf16(k), dev_bf16(v), Kc, Vc, pos, 0, scale,
                            num_splits=splits)
        torch.cuda.synchronize()
        od, ld = host_f64(od), host_f64(ld)
        for b in range(B):
            ro, rl, kref[b], vref[b] = oracle.decode_step(kref[b], vref[b], f64(q[b]),
                                                          f64(k[b]), f64(v[b]), scale)
            compare(f"O decode t{t} b{b}", od[b], ro)
            compare(f"LSE decode t{t} b{b}", ld[:, b], rl)
        pos += 1


@settings(max_examples=30, deadline=None, derandomize=True, database=None)
@given(turns=st.lists(st.tuples(hist_len, new_len), min_size=1, max_size=4),
       is_query=st.booleans(), hh=cache_heads, d=st.sampled_from([64, 128]),
       page_size=st.sampled_from([64, 128, 192, 256]), splits=st.sampled_from([0, 2, 7]),
       seed=st.integers(0, 2 ** 31 - 1))
def test_generated_paged_equals_dense(turns, is_query, hh, d, page_size, splits, seed):
    """The paged entry points on a shuffled page pool give the dense entry
    points' results bit for bit, for a segment prefill and two decode steps."""
    torch = torch_cuda()
    from paper_2408_00539_amd import ops
    hq, hkv = hh
    rng = np.random.default_rng(seed)

    def bits(*shape):
        return W.to_bf16_bits(rng.standard_normal(shape, dtype=np.float32))
    hist = [h for h, _ in turns]
    new = [n for _, n in turns]
    B = len(turns)
    mp = -(-(max(h + n for h, n in turns) + 2) // page_size)
    cap = mp * page_size
    kc = np.zeros((B, hkv, cap, d), np.uint16)
    vc = np.zeros((B, hkv, cap, d), np.uint16)
    for b, C in enumerate(hist):
        kc[b, :, :C] = bits(hkv, C, d)
        vc[b, :, :C] = bits(hkv, C, d)
    npages = B * mp + 3
    table = rng.permutation(npages)[:B * mp].astype(np.int32).reshape(B, mp)

    def pool_of(c):
        pool = np.zeros((npages, hkv, page_size, d), np.uint16)
        for b in range(B):
            for j in range(mp):
                pool[table[b, j]] = c[b, :, j * page_size:(j + 1) * page_size]
        return dev_bf16(pool)
    cu = torch.from_numpy(np.concatenate([[0], np.cumsum(new)]).astype(np.int32)).cuda()
    Tn = sum(new)
    qn, kn, vn = dev_bf16(bits(Tn, hq, d)), dev_bf16(bits(Tn, hkv, d)), dev_bf16(bits(Tn, hkv, d))
    lens = torch.tensor(hist, dtype=torch.int32, device="cuda")
    Kd, Vd, Kp, Vp = dev_bf16(kc), dev_bf16(vc), pool_of(kc), pool_of(vc)
    tab = torch.from_numpy(table).cuda()
    announce("fuzz paged", turns, is_query, hq, hkv, d, page_size, splits, seed)
    od, ld = ops.prefill_cached_segment(qn, kn, vn, Kd, Vd, lens, cu, max(new), is_query)
    op, lp = ops.prefill_paged(qn, kn, vn, Kp, Vp, tab, lens, cu, max(new), is_query)
    outs = [(od, op), (ld, lp)]
    pos = lens + torch.tensor(new, dtype=torch.int32, device="cuda")
    for t in range(2):
        q, k, v = dev_bf16(bits(B, hq, d)), dev_bf16(bits(B, hkv, d)), dev_bf16(bits(B, hkv, d))
        outs.append(tuple(ops.decode(q, k, v, Kd, Vd, pos, 0, num_splits=splits)))
        outs.append(tuple(ops.decode_paged(q, k, v, Kp, Vp, tab, pos, 0, num_splits=splits)))
        pos += 1
    torch.cuda.synchronize()
    for a, b in outs[:2]:
        assert torch.equal(a.view(torch.int16) if a.dtype == torch.bfloat16 else a,
                           b.view(torch.int16) if b.dtype == torch.bfloat16 else b)
    for (oa, la), (ob, lb) in zip(outs[2::2], outs[3::2]):
        assert torch.equal(oa.view(torch.int16), ob.view(torch.int16)) and torch.equal(la, lb)


@settings(max_examples=20, deadline=None, derandomize=True, database=None)
@given(pos=st.lists(st.one_of(st.sampled_from([0, 1, 31, 32, 63, 64, 255, 256, 319]),
                              st.integers(0, 319)), min_size=32, max_size=32),
       g=st.sampled_from([1, 2, 3]), d=st.sampled_from([64, 128]),
       splits=st.sampled_from([0, 1, 3, 64]), seed=st.integers(0, 2 ** 31 - 1))
def test_generated_decode_many_slabs(pos, g, d, splits, seed):
    """Decode steps of 32 dialogues x 16 KV heads (512 slabs: the vector
    kernel for 1-3 query heads per KV head) at generated positions, against
    the oracle's decode step."""
    torch = torch_cuda()
    from paper_2408_00539_amd import ops
    B, hkv, cap = 32, 16, 320
    hq = g * hkv
    rng = np.random.default_rng(seed)

    def bits(*shape):
        return W.to_bf16_bits(rng.standard_normal(shape, dtype=np.float32))
    kc, vc = bits(B, hkv, cap, d), bits(B, hkv, cap, d)
    q, kn, vn = bits(B, hq, d), bits(B, hkv, d), bits(B, hkv, d)
    p = np.array(pos, np.int32)
    scale = 1 / np.sqrt(d)
    announce("fuzz decode slabs", g, d, splits, seed)
    o, lse = ops.decode(dev_bf16(q), dev_bf16(kn), dev_bf16(vn), dev_bf16(kc), dev_bf16(vc),
                        torch.from_numpy(p).cuda(), 0, scale, num_splits=splits)
    torch.cuda.synchronize()
    o, lse = host_f64(o), host_f64(lse)
    for b in range(B):
        ro, rl, _, _ = oracle.decode_step(f64(kc[b, :, :p[b]]).transpose(1, 0, 2),
                                          f64(vc[b, :, :p[b]]).transpose(1, 0, 2),
                                          f64(q[b]), f64(kn[b]), f64(vn[b]), scale)
        compare(f"O b{b}", o[b], ro)
        compare(f"LSE b{b}", lse[:, b], rl)
