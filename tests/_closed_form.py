"""Checks of device outputs against the oracle's closed forms at Q = 0.

With Q = 0 every visible score is 0, so each row's softmax is uniform over
its visible keys: the outputs are fixed by how many keys a row sees and
which ones (Eq. 5). The tolerances here are tight enough that one key too
many or too few on the longest rows of the full-size layouts fails (the
CPU test test_closed_form_checker.py plants such an error in the expected
arrays and checks that it is caught).
"""

import sys

import numpy as np

from paper_2408_00539_amd.workloads import bf16_bits_to_f32, to_bf16_bits

# LSE = ln(n) in fp32: the device adds exact ones, so only the fp32 rounding
# of the logarithm remains (~1e-6 at ln(16384)); one key more or less moves
# it by ln((n + 1) / n) >= 6.1e-5 for n <= 16384
LSE_TOL = 1e-5
# O = mean of V in bf16: round to nearest even leaves <= 2^-9 relative; the
# fp32 sums add ~1e-6 absolute. One key more or less moves a row by
# |v_i - O| / n, ~5e-5 at n = 16384 against a bar of ~3.5e-5 there.
O_REL, O_ABS = 2.0 ** -8, 4e-6
# dV = sum of bf16 weights ~ 1 / n over the rows that see a key, fp32
# accumulation: ~1e-5 at worst; one row more or less moves it by
# >= bf16(1 / 8192) = 1.22e-4 on the 8192-token dialogues
DV_TOL = 3e-5


def bf16_round(x):
    """Nearest bf16 value (round to nearest even) of float64 x, as float64."""
    x = np.asarray(x, dtype=np.float64)
    return bf16_bits_to_f32(to_bf16_bits(x.astype(np.float32))).astype(np.float64)


def close(name, got, ref, rel, abs_):
    """Assert |got - ref| <= rel |ref| + abs_ for every element (got must be
    finite everywhere, so an unwritten NaN-filled output fails)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (name, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{name}: non-finite values (unwritten or bad rows)"
    bar = rel * np.abs(ref) + abs_
    err = np.abs(got - ref)
    ratio = err / bar
    worst = np.unravel_index(int(np.argmax(ratio)), ratio.shape)
    msg = (f"{name}: worst error / bar {float(ratio[worst]):.3f} at {tuple(int(i) for i in worst)} "
           f"(err {float(err[worst]):.3e}, bar {float(bar[worst]):.3e})")
    print(msg)
    sys.stdout.flush()
    assert np.all(err <= bar), msg
    return float(ratio[worst])
