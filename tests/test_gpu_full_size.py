"""Full-size GPU parity: every row, head and tile of the large workloads.

* The Eq. 5 index work as the kernels compute it (lim, seer) equals the
  oracle's bit for bit.
* With Q = 0 every row's softmax is uniform over its visible keys, so each
  row's output is fixed by which keys it sees (tests/_closed_form.py): the
  forward (workloads 1, 2, 4), the backward (workload 4, both modes) and the
  cache path (workload 3, prefill and all 256 decode steps) are checked on
  every row against the oracle's closed forms, tightly enough to catch one
  key too many or too few on the longest rows.
* With the workloads' own random inputs, every element of the forward
  (workloads 1 and 2) and of the backward (workload 4) is compared with the
  fp64 oracle.
Outputs are filled with NaN before each launch, so a tile that no workgroup
writes cannot pass.
"""

import os

import numpy as np
import pytest

import oracle
from paper_2408_00539_amd import workloads as W
from tests._closed_form import (DV_TOL, LSE_TOL, O_ABS, O_REL, bf16_round,
                                close)
from tests._gpu import announce, compare, dev_bf16, f64, host_f64, torch_cuda

pytestmark = pytest.mark.gpu

WORKERS = max(1, min(16, len(os.sched_getaffinity(0))))


def _args(segs):
    return segs.cu_seqlens, segs.cu_segs, segs.seg_is_query


def _segs_dev(segs):
    from paper_2408_00539_amd import ops
    return ops.Segments.from_host(segs.cu_seqlens, segs.cu_segs, segs.seg_is_query)


def _nan(torch, shape, dtype):
    return torch.full(shape, float("nan"), dtype=dtype, device="cuda")


def _random_layout(rng, n_dialogues, max_len):
    dias = []
    for _ in range(n_dialogues):
        n = int(rng.integers(1, max_len + 1))
        parts, left = [], n
        while left:
            ln = int(rng.integers(1, min(left, 300) + 1))
            parts.append(ln)
            left -= ln
        dias.append([(p, bool(rng.integers(0, 2))) for p in parts])
    return W.segments_from_lengths(dias)


LAYOUTS = {f"workload{i}": (lambda i=i: W.make_segments(i, i)) for i in (0, 1, 2, 4)}
LAYOUTS.update({f"random{s}": (lambda s=s: _random_layout(np.random.default_rng(s), 5, 3000))
                for s in range(4)})


@pytest.mark.parametrize("name", sorted(LAYOUTS))
def test_visibility_bit_exact(name):
    torch = torch_cuda()
    from paper_2408_00539_amd import ops
    segs = LAYOUTS[name]()
    announce("visibility", name, segs.total)
    lim_d, seer_d = ops.visibility(_segs_dev(segs))
    torch.cuda.synchronize()
    assert np.array_equal(lim_d.cpu().numpy(), oracle.lim(*_args(segs)))
    assert np.array_equal(seer_d.cpu().numpy(), oracle.seer(*_args(segs)))


def _zero_query_inputs(index):
    torch = torch_cuda()
    w = W.make_workload(index, tensors=False)
    cu = w.segs.cu_seqlens
    k = W.packed_tensor(w.seed, W.K, cu, w.hkv, w.d)
    v = W.packed_tensor(w.seed, W.V, cu, w.hkv, w.d)
    q = torch.zeros((w.segs.total, w.hq, w.d), dtype=torch.bfloat16, device="cuda")
    return w, q, k, v


@pytest.mark.parametrize("index", [1, 2, 4])
def test_fwd_zero_query_every_row(index):
    torch = torch_cuda()
    from paper_2408_00539_amd import ops
    w, q, k, v = _zero_query_inputs(index)
    T, G = w.segs.total, w.hq // w.hkv
    announce("fwd Q=0 workload", index, T, w.hq, w.hkv)
    o = _nan(torch, (T, w.hq, w.d), torch.bfloat16)
    lse = _nan(torch, (w.hq, T), torch.float32)
    ops.fwd(q, dev_bf16(k), dev_bf16(v), _segs_dev(w.segs), w.scale, out=(o, lse))
    torch.cuda.synchronize()
    o_ref, lse_ref = oracle.uniform_fwd(f64(v), *_args(w.segs))
    lse_h = host_f64(lse)
    assert np.all(np.isfinite(lse_h))
    err = np.abs(lse_h - lse_ref[None, :])
    print(f"LSE: max abs err {err.max():.3e} (bar {LSE_TOL})")
    assert err.max() <= LSE_TOL
    for h in range(w.hq):
        close(f"O h{h}", host_f64(o[:, h]), o_ref[:, h // G], O_REL, O_ABS)


def test_bwd_zero_query_every_row():
    """Workload 4 with Q = 0 and dO = 1: dK = 0 exactly;
    dV_i = the sum of the (bf16-rounded, as the device's P operand) weights
    1 / n_j of the rows j that see key i, which pins seer; dQ by its closed
    form."""
    torch = torch_cuda()
    from paper_2408_00539_amd import ops
    w, q, k, v = _zero_query_inputs(4)
    T = w.segs.total
    segs = _segs_dev(w.segs)
    K, V = dev_bf16(k), dev_bf16(v)
    o, lse = ops.fwd(q, K, V, segs, w.scale)
    do = torch.ones_like(q)
    L = oracle.lim(*_args(w.segs))
    cu = w.segs.cu_seqlens
    n = L - cu[oracle.seq_index(cu, T)] + 1
    rq, _, rv = oracle.uniform_bwd(f64(k), f64(v), w.hq, w.scale, *_args(w.segs),
                                   row_weight=bf16_round(1.0 / n))
    announce("bwd Q=0 workload 4")
    dq = _nan(torch, (T, w.hq, w.d), torch.float32)
    dk = _nan(torch, (T, w.hkv, w.d), torch.float32)
    dv = _nan(torch, (T, w.hkv, w.d), torch.float32)
    ops.bwd(q, K, V, o, lse, do, segs, w.scale, out=(dq, dk, dv))
    torch.cuda.synchronize()
    assert bool(torch.isfinite(dk).all()) and int(torch.count_nonzero(dk)) == 0
    for h in range(w.hkv):
        close(f"dV h{h}", host_f64(dv[:, h]), rv[:, h], 0.0, DV_TOL)
    compare("dQ (all elements)", host_f64(dq), rq)


def test_cache_zero_query_every_row():
    """Workload 3 with zero queries: prefill row of dialogue b has
    LSE = ln(C_b + L_b) and O = the mean of all its cached and new values;
    decode step t has LSE = ln(p + 1), O = mean of V[0 .. p], p = C_b + L_b + t."""
    torch = torch_cuda()
    from paper_2408_00539_amd import ops
    w = W.make_workload(3)
    B, H, d, C, S = len(w.new_lens), w.hq, w.d, w.hist_len, w.steps
    Tn = int(w.cu_new[-1])
    announce("cache Q=0 workload 3", B, Tn, S)
    Kc, Vc = dev_bf16(w.k_cache), dev_bf16(w.v_cache)
    lens = torch.full((B,), C, dtype=torch.int32, device="cuda")
    cu_new = torch.from_numpy(w.cu_new).cuda()
    q0 = torch.zeros((Tn, H, d), dtype=torch.bfloat16, device="cuda")
    o = _nan(torch, (Tn, H, d), torch.bfloat16)
    lse = _nan(torch, (H, Tn), torch.float32)
    ops.prefill_cached(q0, dev_bf16(w.k_new), dev_bf16(w.v_new), Kc, Vc, lens, cu_new,
                       int(w.new_lens.max()), w.scale, out=(o, lse))
    pos = lens + torch.from_numpy(w.new_lens).cuda()
    kd, vd = dev_bf16(w.k_dec), dev_bf16(w.v_dec)
    qd0 = torch.zeros((B, H, d), dtype=torch.bfloat16, device="cuda")
    od = _nan(torch, (S, B, H, d), torch.bfloat16)
    ld = _nan(torch, (S, H, B), torch.float32)
    for t in range(S):
        ops.decode(qd0, kd[t], vd[t], Kc, Vc, pos, 0, w.scale, out=(od[t], ld[t]))
        pos += 1
    torch.cuda.synchronize()
    del Kc, Vc
    o_h, lse_h, od_h, ld_h = host_f64(o), host_f64(lse), host_f64(od), host_f64(ld)
    for b in range(B):
        L = int(w.new_lens[b])
        r0, r1 = int(w.cu_new[b]), int(w.cu_new[b + 1])
        vall = np.concatenate([f64(w.v_cache[b, :, :C]).transpose(1, 0, 2),
                               f64(w.v_new[r0:r1]), f64(w.v_dec[:, b])])
        cs = np.cumsum(vall, axis=0)
        npf = C + L
        assert np.max(np.abs(lse_h[:, r0:r1] - np.log(npf))) <= LSE_TOL, b
        close(f"prefill O b{b}", o_h[r0:r1], np.broadcast_to(cs[npf - 1] / npf, (L, H, d)),
              O_REL, O_ABS)
        nd = npf + 1 + np.arange(S)
        assert np.max(np.abs(ld_h[:, :, b] - np.log(nd)[:, None])) <= LSE_TOL, b
        close(f"decode O b{b}", od_h[:, b], cs[npf:npf + S] / nd[:, None, None], O_REL, O_ABS)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("index", [1, 2])
def test_fwd_every_element_vs_oracle(index):
    """The workload's own inputs; all (dialogue, head) pairs of the oracle."""
    torch = torch_cuda()
    from paper_2408_00539_amd import ops
    w = W.make_workload(index)
    T = w.segs.total
    announce("fwd every element workload", index, T)
    o = _nan(torch, (T, w.hq, w.d), torch.bfloat16)
    lse = _nan(torch, (w.hq, T), torch.float32)
    ops.fwd(dev_bf16(w.q), dev_bf16(w.k), dev_bf16(w.v), _segs_dev(w.segs), w.scale,
            out=(o, lse))
    torch.cuda.synchronize()
    ro, rl = oracle.fwd(f64(w.q), f64(w.k), f64(w.v), *_args(w.segs), w.scale,
                        workers=WORKERS)
    compare("O (all elements)", host_f64(o), ro)
    compare("LSE (all elements)", host_f64(lse), rl)


@pytest.mark.timeout(900)
def test_bwd_every_element_vs_oracle():
    """Workload 4's own inputs, every element of dQ, dK, dV."""
    torch = torch_cuda()
    from paper_2408_00539_amd import ops
    w = W.make_workload(4)
    T = w.segs.total
    segs = _segs_dev(w.segs)
    Q, K, V, DO = dev_bf16(w.q), dev_bf16(w.k), dev_bf16(w.v), dev_bf16(w.do)
    o, lse = ops.fwd(Q, K, V, segs, w.scale)
    announce("bwd every element workload 4")
    dq = _nan(torch, (T, w.hq, w.d), torch.float32)
    dk = _nan(torch, (T, w.hkv, w.d), torch.float32)
    dv = _nan(torch, (T, w.hkv, w.d), torch.float32)
    ops.bwd(Q, K, V, o, lse, DO, segs, w.scale, out=(dq, dk, dv))
    torch.cuda.synchronize()
    gq, gk, gv = host_f64(dq), host_f64(dk), host_f64(dv)
    del dq, dk, dv, Q, K, V, DO, o, lse
    rq, rk, rv = oracle.bwd(f64(w.q), f64(w.k), f64(w.v), f64(w.do), *_args(w.segs),
                            w.scale, workers=WORKERS)
    compare("dQ (all elements)", gq, rq)
    compare("dK (all elements)", gk, rk)
    compare("dV (all elements)", gv, rv)
