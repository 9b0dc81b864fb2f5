"""The value-comparison rules the GPU tests apply (tests/_parity.py), checked
on the CPU: an fp32 sum of exact products passes them, a planted error
fails them, and the plain relative figures are what their definitions say."""
import numpy as np
import pytest

from _parity import U_ACC, assert_values, value_figures


def _fp32_dot(rng, rows, n):
    x = rng.standard_normal((rows, n)).astype(np.float32)
    y = rng.standard_normal((rows, n)).astype(np.float32)
    p = x.astype(np.float64) * y.astype(np.float64)
    got = np.cumsum(p.astype(np.float32), axis=1, dtype=np.float32)[:, -1]
    return got, p.sum(axis=1), np.abs(p).sum(axis=1)


def test_fp32_sum_passes_and_plain_figures():
    """Sequential fp32 sums of 819 N(0,1) products against fp64: every rule
    holds at 1e-4; the elementwise plain figure over |r| >= 1e-3 max|r|
    may exceed 1e-4 only on badly conditioned entries, which the asserted
    subset (kappa <= 0.1 tol / u) leaves out."""
    rng = np.random.default_rng(1)
    got, acc, mag = _fp32_dot(rng, 20000, 819)
    f = assert_values(got, acc, mag, "f32")
    d = np.abs(got - acc)
    assert f["normwise_rel"] == pytest.approx(d.max() / np.abs(acc).max())
    big = np.abs(acc) >= 1e-3 * np.abs(acc).max()
    assert f["n_big"] == int(big.sum())
    assert f["plain_rel_big"] == pytest.approx((d[big] / np.abs(acc[big])).max())
    wc = big & (mag / np.abs(acc) <= 0.1 * 1e-4 / U_ACC)
    assert f["n_wc"] == int(wc.sum()) and f["n_wc"] > 0.8 * len(acc)


def test_planted_errors_fail():
    rng = np.random.default_rng(2)
    got, acc, mag = _fp32_dot(rng, 2000, 64)
    i = int(np.argmax(np.abs(acc)))
    bad = got.copy()
    bad[i] += 3e-4 * abs(acc[i]) + 3e-4 * mag[i]  # mag-relative and plain error both above 1e-4
    with pytest.raises(AssertionError):
        assert_values(bad, acc, mag, "f32")
    zero = got.copy()
    acc2, mag2 = acc.copy(), mag.copy()
    acc2[0] = mag2[0] = 0.0
    zero[0] = 1e-30  # a value where every product is zero must be exactly zero
    with pytest.raises(AssertionError):
        assert_values(zero, acc2, mag2, "f32")


def test_bf16_output_rounding_within_bf16_tolerance():
    """W written as bf16 (round to nearest even from fp32 sums) stays within
    the bf16 tolerance on every figure: the rounding adds at most 2^-9
    relative to each value."""
    rng = np.random.default_rng(3)
    got, acc, mag = _fp32_dot(rng, 5000, 256)
    b = got.astype(np.float32).view(np.uint32)
    b = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16 << 16).astype(np.uint32).view(np.float32)
    f = value_figures(b, acc, mag, 1e-2)
    assert f["plain_rel_wc"] <= 2.0 ** -8 and f["mag_rel"] <= 2.0 ** -8
    assert_values(b, acc, mag, "bf16")
