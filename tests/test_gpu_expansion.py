"""GPU parity of ISM's single pass against the prefix-mask sample expansion
(Sec. 1; Eq. 3 against Eq. 5 on the rows both masks share).

The same dialogues run through ism_attn_fwd / ism_attn_bwd twice: once as ISM
dialogues, once expanded into the samples a prefix-mask model trains on. Each
run is compared with the oracle; the rows of Q_k and A_k (and, for a loss on
answer rows only, the gradients summed over a token's copies) must agree
between the two runs.
"""

import numpy as np
import pytest

import oracle
from paper_2408_00539_amd import workloads as W
from tests._gpu import announce, compare, dev_bf16, f64, host_f64, torch_cuda

pytestmark = pytest.mark.gpu


def _bits(rng, *shape):
    return W.to_bf16_bits(rng.standard_normal(shape, dtype=np.float32))


def _layout():
    return W.segments_from_lengths([W.alternating([40, 70, 33, 65, 1, 129]),
                                    W.alternating([64, 64, 100, 3])])


def _shared_rows(segs, exp, src):
    """Expanded rows of Q_k and A_k of every sample (and their originals)."""
    rows = []
    for kk in range(exp.batch):
        s, e = int(exp.cu_seqlens[kk]), int(exp.cu_seqlens[kk + 1])
        last = int(src[int(exp.cu_segs[2 * kk + 1]) - 1])
        g = int(np.searchsorted(segs.cu_segs, last, side="right")) - 1
        rows.append(np.arange(s + int(segs.cu_segs[g]) - int(src[s]), e))
    rows = np.concatenate(rows)
    return rows, src[rows]


def _answer_rows(segs):
    ans = np.zeros(segs.total, dtype=bool)
    for g in range(segs.num_segs):
        if not segs.seg_is_query[g]:
            ans[segs.cu_segs[g]:segs.cu_segs[g + 1]] = True
    return ans


@pytest.mark.parametrize("d,hq,hkv", [(64, 4, 2), (128, 8, 2)])
def test_forward_shared_rows(d, hq, hkv):
    torch = torch_cuda()
    from paper_2408_00539_amd import ops
    rng = np.random.default_rng(d + hq)
    segs = _layout()
    exp, src = W.prefix_expansion(segs)
    T = segs.total
    q, k, v = _bits(rng, T, hq, d), _bits(rng, T, hkv, d), _bits(rng, T, hkv, d)
    scale = 1 / np.sqrt(d)
    out = {}
    for name, sg, ix in (("ism", segs, np.arange(T)), ("prefix", exp, src)):
        announce("fwd", name, d, hq, hkv)
        dsg = ops.Segments.from_host(sg.cu_seqlens, sg.cu_segs, sg.seg_is_query)
        o, lse = ops.fwd(dev_bf16(q[ix]), dev_bf16(k[ix]), dev_bf16(v[ix]), dsg,
                         scale)
        torch.cuda.synchronize()
        o, lse = host_f64(o), host_f64(lse)
        ro, rl = oracle.fwd(f64(q[ix]), f64(k[ix]), f64(v[ix]), sg.cu_seqlens,
                            sg.cu_segs, sg.seg_is_query, scale)
        compare(f"O {name}", o, ro)
        compare(f"LSE {name}", lse, rl)
        out[name] = (o, lse)
    er, orig = _shared_rows(segs, exp, src)
    compare("O shared rows", out["prefix"][0][er], out["ism"][0][orig])
    compare("LSE shared rows", out["prefix"][1][:, er], out["ism"][1][:, orig])


@pytest.mark.parametrize("d,hq,hkv", [(64, 4, 2), (128, 4, 4)])
def test_answer_loss_gradients(d, hq, hkv):
    torch = torch_cuda()
    from paper_2408_00539_amd import ops
    rng = np.random.default_rng(3 * d + hq)
    segs = _layout()
    exp, src = W.prefix_expansion(segs)
    T = segs.total
    q, k, v = _bits(rng, T, hq, d), _bits(rng, T, hkv, d), _bits(rng, T, hkv, d)
    do = _bits(rng, T, hq, d)
    do[~_answer_rows(segs)] = 0
    edo = np.zeros((len(src), hq, d), np.uint16)
    for kk in range(exp.batch):
        a, e = int(exp.cu_segs[2 * kk + 1]), int(exp.cu_seqlens[kk + 1])
        edo[a:e] = do[src[a:e]]
    scale = 1 / np.sqrt(d)
    grads = {}
    for name, sg, ix, g_do in (("ism", segs, np.arange(T), do),
                               ("prefix", exp, src, edo)):
        announce("bwd", name, d, hq, hkv)
        dsg = ops.Segments.from_host(sg.cu_seqlens, sg.cu_segs, sg.seg_is_query)
        Q, K, V = dev_bf16(q[ix]), dev_bf16(k[ix]), dev_bf16(v[ix])
        o, lse = ops.fwd(Q, K, V, dsg, scale)
        dq, dk, dv = ops.bwd(Q, K, V, o, lse, dev_bf16(g_do), dsg, scale, True)
        torch.cuda.synchronize()
        dq, dk, dv = host_f64(dq), host_f64(dk), host_f64(dv)
        rq, rk, rv = oracle.bwd(f64(q[ix]), f64(k[ix]), f64(v[ix]), f64(g_do),
                                sg.cu_seqlens, sg.cu_segs, sg.seg_is_query, scale)
        compare(f"dQ {name}", dq, rq)
        compare(f"dK {name}", dk, rk)
        compare(f"dV {name}", dv, rv)
        grads[name] = (dq, dk, dv)
    for i, n in enumerate(("dQ", "dK", "dV")):
        summed = np.zeros_like(grads["ism"][i])
        np.add.at(summed, src, grads["prefix"][i])
        compare(f"{n} expansion summed vs ism", summed, grads["ism"][i])
