"""Pins of the constants the parity bounds are built from (CPU only).

The bound on the effect of rounding P to bf16 uses bf16's unit roundoff, and
the out bound beside it uses half a bf16 ulp at |ref|.  Both are checked here
against torch's own float32 -> bfloat16 conversion (round to nearest even), so
that a constant off by a factor of two fails.
"""

import numpy as np
import torch

from helpers import BF16_UNIT_ROUNDOFF, bf16_half_ulp


def _round_bf16(x):
    return torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()


def test_unit_roundoff_is_the_largest_relative_error_of_one_rounding():
    rng = np.random.default_rng(5)
    x = (rng.uniform(1.0, 2.0, 1 << 20) * 2.0 ** rng.integers(-60, 60, 1 << 20)).astype(np.float32)
    rel = np.abs(_round_bf16(x) - x.astype(np.float64)) / np.abs(x.astype(np.float64))
    assert rel.max() <= BF16_UNIT_ROUNDOFF
    assert rel.max() > 0.99 * BF16_UNIT_ROUNDOFF    # attained: a smaller constant would fail
    # just above 1 the error is exactly the unit roundoff (ties go to even: down to 1)
    tie = np.array([1.0 + 2.0 ** -8], dtype=np.float32)
    assert _round_bf16(tie)[0] == 1.0


def test_half_ulp_bounds_the_absolute_error_of_one_rounding():
    rng = np.random.default_rng(6)
    x = (rng.standard_normal(1 << 20) * 2.0 ** rng.integers(-20, 20, 1 << 20)).astype(np.float32)
    err = np.abs(_round_bf16(x) - x.astype(np.float64))
    hu = bf16_half_ulp(x)
    assert np.all(err <= hu)
    assert (err / hu).max() > 0.99
    assert bf16_half_ulp(np.array([4.5]))[0] == 2.0 ** -6    # ulp on [4, 8) is 2^-5
