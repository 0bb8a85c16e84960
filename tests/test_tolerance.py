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
    assert_close(g, r, "f16", "rounded", dev=np.zeros_like(r))


def test_a_full_ulp_above_four_fails():
    """At |r| >= 4 the bound is half an fp16 spacing plus what the weights'
    rounding can add (dev), not a whole spacing."""
    r = np.array([4.1, -5.3, 6.0, 0.2])
    g = r.copy()
    g[1] -= 2.0 ** -8 * 0.9          # 3.5e-3: under one spacing, over half of one
    with pytest.raises(AssertionError):
        assert_close(g, r, "f16", "planted", dev=np.zeros_like(r))
    # a row whose weights spread over values 1 apart may move by 2^-11 * 1.125 * dev more
    ok = r.copy()
    ok[1] -= 2.0 ** -9 + 2.0 ** -11 * 0.5
    assert_close(ok, r, "f16", "dev term", dev=np.full_like(r, 1.0))


def test_weight_rounding_term_matches_its_derivation():
    """A softmax whose every weight is rounded to fp16 stays inside the bound."""
    rng = np.random.default_rng(3)
    for _ in range(20):
        s = rng.standard_normal(300) * 3
        v = rng.standard_normal((300, 8)) * 4
        p = np.exp(s - s.max())
        w = p / p.sum()
        r = w @ v
        dev = w @ np.abs(v - r)
        pr = p.astype(np.float16).astype(np.float64)
        g = ((pr @ v) / pr.sum()).astype(np.float16).astype(np.float64)
        assert_close(g, r, "f16", "rounded weights", dev=dev)


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


def test_accumulation_allowance_grows_past_4096_keys():
    from parity_util import accumulation_allowance
    # 16 keys per MFMA step, half an fp32 ulp (2^-24) per step
    assert accumulation_allowance() == accumulation_allowance(4096) == 2.0 ** -16
    assert accumulation_allowance(77) == 2.0 ** -16
    assert accumulation_allowance(1 << 20) == (1 << 20) / 16 * 2.0 ** -24
    assert accumulation_allowance(26_843_648) > 0.09
