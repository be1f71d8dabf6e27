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
    # also reported: the largest |ref|, and the error in units of the bf16
    # spacing at each reference value (2^(e - 7) for |ref| in [2^e, 2^(e+1)),
    # references below 1e-6 counted at 1e-6)
    r = np.abs(ref[m])
    ulp = np.exp2(np.floor(np.log2(np.maximum(r, 1e-6))) - 7)
    print(f"{msg}; max |ref| {float(r.max()):.3e}, max err {float((err / ulp).max()):.2f} bf16 ulps")
    sys.stdout.flush()
    assert mx <= max_abs and mn <= mean_abs, msg
    return mx, mn


def announce(*parts):
    """Print (and flush) what the next GPU step runs."""
    print("[gpu-case]", *parts, flush=True)
