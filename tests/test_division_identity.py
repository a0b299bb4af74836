"""The HIP kernels compute the binary32 quotient x / lambda as
fl32(fl64(x * fl64(1 / lambda))) instead of an IEEE binary32 divide.

Why this is exact: with q = x / lambda, |fl64 result - q| <= q * 2^-52, while
an odd 25-bit midpoint M between binary32 neighbours satisfies
|q - M| >= q * 2^-50 (x has a 24-bit significand, M * lambda needs >= 25
bits, so x != M * lambda and their difference is at least one unit of the
finer exponent).  So both round to the same binary32 value whenever q is a
normal number.  These tests check that claim against numpy's IEEE binary32
division, including inputs built to land next to rounding midpoints."""
import numpy as np


def _via_reciprocal(x, lam):
    return (x.astype(np.float64) * (1.0 / lam.astype(np.float64))).astype(np.float32)


def test_random_pairs():
    rng = np.random.default_rng(0)
    n = 2_000_000
    x = (np.rint(rng.uniform(0, 4096, n) * 64) / 64 * rng.integers(1, 4097, n)).astype(np.float32)
    lam = rng.uniform(0.01, 500.0, n).astype(np.float32)
    np.testing.assert_array_equal(x / lam, _via_reciprocal(x, lam))
    # wide dynamic range
    x = np.exp2(rng.uniform(-40, 40, n)).astype(np.float32)
    lam = np.exp2(rng.uniform(-40, 40, n)).astype(np.float32)
    np.testing.assert_array_equal(x / lam, _via_reciprocal(x, lam))


def test_near_midpoints():
    rng = np.random.default_rng(1)
    n = 1_000_000
    # M = odd 25-bit integer * 2^-25 in [0.5, 1): a midpoint of binary32 values
    m = (rng.integers(2**23, 2**24, n) * 2 + 1).astype(np.float64) * 2.0**-25
    lam = rng.uniform(0.5, 300.0, n).astype(np.float32)
    base = (m * lam.astype(np.float64)).astype(np.float32)
    for k in (-2, -1, 0, 1, 2):
        x = np.nextafter(base, np.float32(np.inf) if k > 0 else np.float32(0), dtype=np.float32) if k else base
        if abs(k) == 2:
            x = np.nextafter(x, np.float32(np.inf) if k > 0 else np.float32(0), dtype=np.float32)
        np.testing.assert_array_equal(x / lam, _via_reciprocal(x, lam))


def test_exact_quotients_and_zero():
    lam = np.array([1, 2, 3, 4, 5, 7, 10, 12, 16, 20], np.float32)
    x = lam * np.float32(0.75)
    np.testing.assert_array_equal(x / lam, _via_reciprocal(x, lam))
    z = np.zeros_like(lam)
    np.testing.assert_array_equal(z / lam, _via_reciprocal(z, lam))
