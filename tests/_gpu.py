"""Helpers of the GPU parity tests (no oracle arithmetic here)."""

import os
import sys

import numpy as np
import pytest

# tolerance of the parity bar: bf16 inputs, fp32 accumulation, compared with
# the fp64 oracle on the same bf16 values
MAX_ABS = 2e-2
MEAN_ABS = 2e-3


def torch_cuda():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def dev_bf16(bits):
    """uint16 bf16 bit patterns (numpy) -> bf16 tensor on cuda:0."""
    torch = torch_cuda()
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.view(torch.bfloat16).to("cuda")


def host_f64(t):
    """GPU tensor (bf16 / fp32) -> float64 numpy."""
    return t.detach().float().cpu().numpy().astype(np.float64)


def f64(bits):
    from paper_2408_00539_amd.workloads import bf16_bits_to_f32
    return bf16_bits_to_f32(bits).astype(np.float64)


def compare(name, got, ref, max_abs=MAX_ABS, mean_abs=MEAN_ABS, where=None):
    """Assert the parity bar on the finite entries of ref (oracle)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (name, got.shape, ref.shape)
    m = np.isfinite(ref) if where is None else where
    assert m.any(), f"{name}: nothing compared"
    err = np.abs(got[m] - ref[m])
    assert np.all(np.isfinite(got[m])), f"{name}: non-finite GPU values"
    mx, mn = float(err.max()), float(err.mean())
    msg = f"{name}: max abs {mx:.3e} (bar {max_abs}), mean abs {mn:.3e} (bar {mean_abs})"
    # also reported: the largest |ref| and, for the bf16 output O, the error
    # in units of the bf16 spacing (2^(e - 7) for |x| in [2^e, 2^(e+1))): the
    # largest error against the spacing at the tensor's largest |ref|, and the
    # median error against the spacing at each element's own |ref|
    r = np.abs(ref[m])
    rmax = float(r.max())
    extra = f"; max |ref| {rmax:.3e}"
    if name.startswith("O") and rmax > 0:
        spacing = lambda x: np.exp2(np.floor(np.log2(x)) - 7)
        per_elem = err / spacing(np.maximum(r, 2.0 ** -40))
        extra += (f", max err {mx / float(spacing(rmax)):.2f} bf16 ulps at that scale,"
                  f" median {float(np.median(per_elem)):.2f} ulps per element")
    print(msg + extra)
    sys.stdout.flush()
    assert mx <= max_abs and mn <= mean_abs, msg
    return mx, mn


def announce(*parts):
    """Print (and flush) what the next GPU step runs."""
    print("[gpu-case]", *parts, flush=True)
