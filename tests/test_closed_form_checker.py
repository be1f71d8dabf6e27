"""The full-size Q = 0 checks can see a one-key (or one-row) error.

For the layouts of the full-size workloads, an output that is right up to the
device's rounding passes the checks of tests/_closed_form.py, and the same
output fails once the EXPECTED arrays are perturbed by one key at the rows
where such an error is hardest to see (the longest rows) or by one row at
the keys seen by the most rows. The perturbation is planted in the expected
values on the CPU, never in a kernel.
"""

import numpy as np
import pytest

import oracle
from paper_2408_00539_amd import workloads as W
from tests._closed_form import DV_TOL, LSE_TOL, O_ABS, O_REL, bf16_round, close


def _args(segs):
    return segs.cu_seqlens, segs.cu_segs, segs.seg_is_query


@pytest.mark.parametrize("index", [1, 2, 4])
def test_forward_checks_catch_one_key(index):
    segs = W.make_segments(index, index)
    T = segs.total
    rng = np.random.default_rng(index)
    v = rng.standard_normal((T, 1, 128)).astype(np.float32).astype(np.float64)
    o_ref, lse_ref = oracle.uniform_fwd(v, *_args(segs))
    o_dev = bf16_round(o_ref[:, 0])
    lse_dev = lse_ref.astype(np.float32).astype(np.float64)
    close("O", o_dev, o_ref[:, 0], O_REL, O_ABS)
    assert np.max(np.abs(lse_dev - lse_ref)) <= LSE_TOL

    L = oracle.lim(*_args(segs))
    cu = segs.cu_seqlens
    sb = cu[oracle.seq_index(cu, T)]
    n = L - sb + 1
    # the longest rows, and a few more spread over the batch
    rows = [int(np.argmax(n))] + [int(j) for j in rng.choice(np.nonzero(n > 64)[0], 8)]
    for j in rows:
        s = int(sb[j])
        for extra in (+1, -1):
            hi = int(L[j]) + extra
            e = int(cu[np.searchsorted(cu, j, side="right")])
            if hi < s or hi >= e:
                continue
            o_bad = o_ref[:, 0].copy()
            o_bad[j] = v[s:hi + 1, 0].mean(axis=0)
            with pytest.raises(AssertionError):
                close("O planted", o_dev, o_bad, O_REL, O_ABS)
            lse_bad = lse_ref.copy()
            lse_bad[j] = np.log(hi - s + 1)
            assert np.max(np.abs(lse_dev - lse_bad)) > LSE_TOL


def test_backward_dv_check_catches_one_row():
    segs = W.make_segments(4, 4)
    T = segs.total
    rng = np.random.default_rng(4)
    k = rng.standard_normal((T, 1, 8))
    v = rng.standard_normal((T, 1, 8))
    L = oracle.lim(*_args(segs))
    cu = segs.cu_seqlens
    n = L - cu[oracle.seq_index(cu, T)] + 1
    p = bf16_round(1.0 / n)
    _, _, dv_ref = oracle.uniform_bwd(k, v, 1, 0.088, *_args(segs), row_weight=p)
    dv_dev = dv_ref.astype(np.float32).astype(np.float64)
    close("dV", dv_dev, dv_ref, 0.0, DV_TOL)
    se = oracle.seer(*_args(segs))
    # a key's first seeing row dropped (or one earlier row added) moves its
    # dV by that row's weight; the smallest such weight is the hardest case
    i = int(np.argmin(p[se]))
    assert p[se[i]] > 2 * DV_TOL
    dv_bad = dv_ref.copy()
    dv_bad[i] -= p[se[i]]
    with pytest.raises(AssertionError):
        close("dV planted", dv_dev, dv_bad, 0.0, DV_TOL)
    if se[i] > cu[np.searchsorted(cu, i, side="right") - 1]:
        dv_bad = dv_ref.copy()
        dv_bad[i] += p[se[i] - 1]
        with pytest.raises(AssertionError):
            close("dV planted", dv_dev, dv_bad, 0.0, DV_TOL)
