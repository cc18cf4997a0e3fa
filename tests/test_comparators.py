"""Pins for the comparators that decide every GPU parity verdict.

``oracle.normalized_error`` judges FP16 results (max |C_gpu - C_ref| / D with
D = sum_k |a||b|), ``gpu_util.assert_parity`` applies it (and bit-exactness for
the integer paths), and ``gpu_util.ulp_of`` / ``assert_scaled`` judge the
scaled outputs. A slip in any of them would let a wrong GPU result pass, so
each is checked here on inputs whose verdict is known by hand: errors worked
out exactly, values exactly at and just past the tolerance, NaN and infinity,
zero error scales, and ulp spacings against numpy's ``spacing`` (a library
routine) at format boundaries. CPU only: the tensors are host tensors.
"""
import numpy as np
import pytest
import torch

import oracle
from tests.gpu_util import F16_TOL, assert_parity, assert_scaled, ulp_of

# ------------------------------------------------------------ normalized_error


def test_normalized_error_hand_computed():
    ref = np.array([[1.0, 2.0], [-3.0, 0.5]])
    D = np.array([[4.0, 8.0], [16.0, 2.0]])
    # errors 0.5 / 4, 0, 1 / 16, 0.25 / 2: the max is 0.125 (two elements tie)
    gpu = np.array([[1.5, 2.0], [-2.0, 0.25]], np.float32)
    assert oracle.normalized_error(gpu, ref, D) == 0.125
    # the sign of the difference does not matter
    assert oracle.normalized_error(np.array([[0.5, 2.0], [-3.0, 0.5]], np.float32), ref, D) == 0.125
    # the maximum, not the first or the mean: one bad element among good ones
    big = np.zeros((64, 64)), np.ones((64, 64))
    g = np.zeros((64, 64), np.float32)
    g[37, 5] = 0.75
    assert oracle.normalized_error(g, *big) == 0.75
    assert oracle.normalized_error(np.zeros((64, 64), np.float32), *big) == 0.0


def test_normalized_error_at_the_tolerance():
    ref = np.array([1.0, -1.0])
    D = np.array([1024.0, 2048.0])
    at = np.array([1.0 + F16_TOL * 1024.0, -1.0], np.float64)  # exactly 1e-3 of D (1.024 is not a
    err = oracle.normalized_error(at, ref, D)                   # binary32 value: compare in binary64)
    assert abs(err - F16_TOL) < 1e-15
    over = np.array([1.0, -1.0 - 1.01 * F16_TOL * 2048.0])
    assert oracle.normalized_error(over, ref, D) > F16_TOL
    with pytest.raises(AssertionError):
        assert_parity("f16", over.astype(np.float32), ref, D)
    ok = np.array([1.0 + 0.5 * F16_TOL * 1024.0, -1.0], np.float32)
    assert assert_parity("f16", ok, ref, D) <= F16_TOL


@pytest.mark.parametrize("bad", [np.nan, np.inf, -np.inf])
def test_normalized_error_non_finite_is_infinite(bad):
    ref = np.zeros(4)
    D = np.ones(4)
    g = np.zeros(4, np.float32)
    g[2] = bad
    assert oracle.normalized_error(g, ref, D) == np.inf
    with pytest.raises(AssertionError):
        assert_parity("f16", g, ref, D)


def test_normalized_error_zero_scale():
    ref = np.array([0.0, 0.0, 2.0])
    D = np.array([0.0, 0.0, 4.0])
    # D = 0: the exact value is 0; any nonzero result is an infinite error
    assert oracle.normalized_error(np.array([0.0, 1e-30, 2.0], np.float32), ref, D) == np.inf
    # +0 and -0 are both exact
    assert oracle.normalized_error(np.array([-0.0, 0.0, 2.0], np.float32), ref, D) == 0.0
    # all D = 0 and all results zero: error 0
    assert oracle.normalized_error(np.zeros(3, np.float32), np.zeros(3), np.zeros(3)) == 0.0
    # the finite elements still count when some D are zero
    assert oracle.normalized_error(np.array([0.0, 0.0, 2.5], np.float32), ref, D) == 0.125


def test_assert_parity_integers_are_bit_exact():
    ref = np.arange(-50, 50, dtype=np.int64).reshape(10, 10) * 1000003
    assert assert_parity("s8", ref.astype(np.int32), ref, None) == 0.0
    off = ref.astype(np.int32)
    off[7, 3] += 1
    with pytest.raises(AssertionError):
        assert_parity("s4", off, ref, None)
    with pytest.raises(AssertionError):  # FP32 output where INT32 is due
        assert_parity("s8", ref.astype(np.float32), ref, None)
    big = np.array([[2 ** 31]], np.int64)  # an oracle value outside int32 is refused
    with pytest.raises(AssertionError):
        assert_parity("s8", np.array([[0]], np.int32), big, None)


# ------------------------------------------------------------------- ulp_of


def _boundary_values(dtype):
    fi = np.finfo(dtype)
    xs = [1.0, 1.5, 2.0, 3.0, 0.75, float(fi.tiny), float(fi.tiny) * 3]
    for k in (-3, 0, 1, 4, 10):
        p = np.asarray(2.0 ** k, dtype)
        xs += [float(p), float(np.nextafter(p, dtype(0))), float(np.nextafter(p, dtype(np.inf)))]
    return np.array(xs)


@pytest.mark.parametrize("out,dtype", [("f32", np.float32), ("f16", np.float16)])
def test_ulp_of_matches_numpy_spacing(out, dtype):
    xs = _boundary_values(dtype)
    want = np.abs(np.spacing(xs.astype(dtype)).astype(np.float64))
    np.testing.assert_array_equal(ulp_of(xs, out), want)
    np.testing.assert_array_equal(ulp_of(-xs, out), want)  # sign does not matter
    # the largest finite value (numpy's spacing overflows there): 2^(emax - fraction bits)
    fi = np.finfo(dtype)
    assert ulp_of(np.array([float(fi.max)]), out)[0] == 2.0 ** (fi.maxexp - 1 - fi.nmant)
    # subnormal range: the fixed spacing of the smallest normal's binade
    sub = float(np.finfo(dtype).tiny) / 8
    assert ulp_of(np.array([sub, 0.0]), out).tolist() == [float(np.finfo(dtype).smallest_subnormal)] * 2


def test_ulp_of_binary64_values_just_below_a_power_of_two():
    """Exact values are binary64: one just below 2^k is still in the binade
    below (a rounded log2 would put it in the next one)."""
    for k in (2, 5, 20):
        x = np.nextafter(2.0 ** k, 0.0)
        assert ulp_of(np.array([x]), "f32")[0] == 2.0 ** (k - 1 - 23)
        assert ulp_of(np.array([x]), "f16")[0] == 2.0 ** (k - 1 - 10)
        assert ulp_of(np.array([x]), "bf16")[0] == 2.0 ** (k - 1 - 7)


def test_ulp_of_bfloat16():
    """bfloat16: 7 stored fraction bits, smallest normal 2^-126."""
    x = np.array([1.0, 1.99, 2.0, 3.0e38, 2.0 ** -126, 2.0 ** -130])
    want = [2.0 ** -7, 2.0 ** -7, 2.0 ** -6, 2.0 ** (127 - 7), 2.0 ** -133, 2.0 ** -133]
    assert ulp_of(x, "bf16").tolist() == want


# ------------------------------------------------------------- assert_scaled


@pytest.mark.parametrize("out,tdt,n_ulp", [("f32", torch.float32, 3), ("f16", torch.float16, 1),
                                           ("bf16", torch.bfloat16, 1)])
def test_assert_scaled_accepts_the_bound_and_rejects_past_it(out, tdt, n_ulp):
    exact = np.array([1.0, -3.0, 1000.0, 2.0 ** -5, 0.375])
    u = ulp_of(exact, out)
    assert_scaled(torch.tensor(exact, dtype=tdt), exact, None, out)  # exact values pass
    # n_ulp away from the exact value passes (the values are on the format's grid)
    at = exact + n_ulp * u
    assert_scaled(torch.tensor(at, dtype=tdt), exact, None, out)
    # one more ulp fails, on any single element
    for i in range(len(exact)):
        past = exact.copy()
        past[i] += (n_ulp + 1) * u[i]
        with pytest.raises(AssertionError):
            assert_scaled(torch.tensor(past, dtype=tdt), exact, None, out)


@pytest.mark.parametrize("bad", [np.nan, np.inf])
def test_assert_scaled_rejects_non_finite(bad):
    exact = np.array([1.0, 2.0])
    with pytest.raises(AssertionError):
        assert_scaled(torch.tensor([1.0, bad], dtype=torch.float32), exact, None, "f32")


def test_assert_scaled_fp16_inputs_add_the_sum_bound():
    """FP16 inputs: the tolerance grows by 1e-3 of the (scaled) error scale D."""
    exact = np.array([10.0])
    D = np.array([100.0])
    within = torch.tensor([10.0 + 0.09], dtype=torch.float32)   # 0.09 < 1e-3 * 100 + ulps
    assert_scaled(within, exact, D, "f32")
    with pytest.raises(AssertionError):
        assert_scaled(torch.tensor([10.0 + 0.2], dtype=torch.float32), exact, D, "f32")
    with pytest.raises(AssertionError):  # without D the same value is far off
        assert_scaled(within, exact, None, "f32")
