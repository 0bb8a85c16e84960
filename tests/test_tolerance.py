"""The parity tolerance is neither vacuous nor stricter than fp16 output allows."""
import numpy as np
import pytest

from parity_util import assert_close, ulp


def test_ulp_of_fp16_grid():
    assert ulp(1.5) == 2.0 ** -10
    assert ulp(4.0958) == 2.0 ** -8
    assert ulp(0.01) == 2.0 ** -17
    assert ulp(3.0, "bf16") == 2.0 ** -6


def test_correctly_rounded_output_always_passes():
    rng = np.random.default_rng(1)
    r = rng.standard_normal(200000) * 2.5
    g = r.astype(np.float16).astype(np.float64)
    assert_close(g, r, "f16", "rounded")


def test_two_millis_off_below_four_fails():
    r = np.array([0.5, 1.0, 3.9, -2.0])
    g = r.copy()
    g[2] += 2.1e-3
    with pytest.raises(AssertionError):
        assert_close(g, r, "f16", "planted")


def test_one_percent_relative_error_fails_everywhere():
    rng = np.random.default_rng(2)
    r = rng.standard_normal(1000) * 5
    g = r * 1.011
    with pytest.raises(AssertionError):
        assert_close(g, r, "f16", "planted")
