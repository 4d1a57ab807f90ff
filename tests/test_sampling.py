"""The parity helpers' rounding bound, checked on the CPU against torch's own
round-to-nearest-even conversion to bf16."""
from __future__ import annotations

import numpy as np
import pytest
import torch

from sampling import assert_parity, bf16_half_ulp


def _bf16(x: np.ndarray) -> np.ndarray:
    return torch.from_numpy(x).to(torch.bfloat16).double().numpy()


def test_half_ulp_bounds_bf16_rounding_at_every_magnitude():
    rng = np.random.default_rng(0)
    x = rng.standard_normal(200_000) * np.exp2(rng.integers(-20, 20, 200_000))
    # fp32 values, as the kernels round them: torch takes fp64 to bf16 through
    # fp32, which would round twice
    x = x.astype(np.float32).astype(np.float64)
    err = np.abs(_bf16(x) - x)
    assert np.all(err <= bf16_half_ulp(x))
    # and it is tight: halfway between two neighbouring bf16 values (8 significant
    # bits) the rounding moves a value by exactly the bound
    lo = _bf16(x)
    mid = lo + np.sign(x) * 2 * bf16_half_ulp(lo) / 2
    np.testing.assert_array_equal(np.abs(_bf16(mid) - mid), bf16_half_ulp(lo))


@pytest.mark.parametrize("x,h", [(1.0, 2.0 ** -8), (1.99, 2.0 ** -8), (2.0, 2.0 ** -7),
                                 (-8.024514, 2.0 ** -5), (0.3, 2.0 ** -10), (0.0, 0.0)])
def test_half_ulp_values(x, h):
    assert bf16_half_ulp(np.array([x]))[0] == h


def test_output_rounding_alone_can_pass_the_max_abs_bound():
    # an exact Delta output of -8.0245 (a one-key window: v_i + Delta) stored in
    # bf16 is -8.0 at best, 0.0245 away
    ref = np.concatenate([[-8.024514], np.full(99, 0.5)])
    got = _bf16(ref)
    with pytest.raises(AssertionError):
        assert_parity(got, ref)
    assert_parity(got, ref, slack=bf16_half_ulp(ref))
    # the slack forgives the output's rounding, not an error of the computation
    off = np.zeros_like(ref)
    off[1] = 0.025
    with pytest.raises(AssertionError):
        assert_parity(got + off, ref, slack=bf16_half_ulp(ref))
