"""Pins of the oracle's truncating quantiser (Ozaki-II-TZ: Eq. (scale) with
truncation toward zero in place of round to nearest, Table variants), for
both modulus sets.  Expected values from Python Fractions (int() of a
Fraction truncates toward zero), big integers and CPython's correctly
rounded conversions."""
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle
import workloads


def _signed(hi, lo):
    v = ((hi & ((1 << 64) - 1)) << 64) | lo
    return v - (1 << 128) if v >> 127 else v


def _py_round(X, e):
    if X == 0:
        return 0.0
    if e >= 0:
        try:
            return float(X * 2 ** e)
        except OverflowError:
            return math.copysign(math.inf, X)
    return X / 2 ** (-e)


def test_tz_scalar_vs_fraction():
    rng = np.random.default_rng(3)
    cases = [(2.5, 0), (-2.5, 0), (2.7, 0), (-2.7, 0), (0.999999, 0), (-0.999999, 0), (3.0, 0),
             (-3.0, 0), (0.5, 0), (-0.5, 0), (1e-310, 1070), (-1e-310, 1070), (5e-324, 1100),
             (1.5, 51), (-(2.0 ** 52) - 0.5, 0), (0.0, 10), (-0.0, 10)]
    for _ in range(3000):
        x = float(rng.standard_normal() * math.exp(rng.standard_normal() * 8))
        cases.append((x, int(rng.integers(-10, 50))))
    for x, sigma in cases:
        exact = Fraction(x) * Fraction(2) ** sigma
        if abs(exact) >= 2 ** 62:
            continue
        z = oracle.quantise(x, sigma, oracle.TZ)
        assert z == int(exact), (x, sigma)
        # toward zero: never larger in magnitude, less than one away
        assert abs(z) <= abs(exact) and abs(exact - z) < 1
        assert z == 0 or (z > 0) == (x > 0)
        # RN and TZ agree on integers and differ by at most one elsewhere
        r = oracle.quantise(x, sigma)
        assert abs(r - z) <= 1
        if exact.denominator == 1:
            assert r == z


def test_tz_nonfinite_row_quantises_to_zero():
    assert oracle.quantise(1.0, -(2 ** 31), oracle.TZ) == 0


def _python_pipeline(A, B, set):
    m, k = A.shape
    n = B.shape[1]
    t = oracle.scale_bits(k, set)
    sig = [t - math.frexp(float(np.max(np.abs(A[i]))))[1] for i in range(m)]
    tau = [t - math.frexp(float(np.max(np.abs(B[:, j]))))[1] for j in range(n)]
    Aq = [[int(Fraction(float(A[i, l])) * Fraction(2) ** sig[i]) for l in range(k)] for i in range(m)]
    Bq = [[int(Fraction(float(B[l, j])) * Fraction(2) ** tau[j]) for l in range(k)] for j in range(n)]
    X = [[sum(Aq[i][l] * Bq[j][l] for l in range(k)) for j in range(n)] for i in range(m)]
    C = np.array([[_py_round(X[i][j], -sig[i] - tau[j]) for j in range(n)] for i in range(m)])
    return sig, tau, Aq, Bq, X, C


@pytest.mark.parametrize("set", [0, 1])
@pytest.mark.parametrize("shape,s,seed", [((5, 7, 9), 0.5, 1), ((4, 6, 64), 2.0, 3), ((6, 5, 130), 4.0, 5),
                                          ((3, 4, 1), 1.0, 4)])
def test_tz_dgemm_matches_bigint_brute_force(shape, s, seed, set):
    m, n, k = shape
    A = workloads.random_matrix(m, k, s, seed)
    B = workloads.random_matrix(k, n, s, seed + 100)
    res = oracle.dgemm(A, B, set=set, quant=oracle.TZ)
    sig, tau, Aq, Bq, X, C = _python_pipeline(A, B, set)
    assert list(res.sigma) == sig and list(res.tau) == tau
    assert res.ZA.tolist() == Aq and res.ZB.tolist() == Bq
    for i in range(m):
        for j in range(n):
            assert _signed(int(res.Xhi[i, j]), int(res.Xlo[i, j])) == X[i][j]
    assert np.array_equal(res.C.view(np.uint64), C.view(np.uint64))


def test_tz_error_bound_vs_exact_product():
    """With truncation each quantised operand errs by less than one unit of
    its scale (twice the RN bound):
    |C - AB| <= 2^{-tau} sum|a| + 2^{-sigma} sum|b| + k 2^{-sigma-tau} + u|C|."""
    for (m, n, k, s, seed) in [(6, 5, 40, 0.5, 1), (4, 4, 200, 1.0, 2), (5, 3, 64, 2.0, 3)]:
        A = workloads.random_matrix(m, k, s, seed)
        B = workloads.random_matrix(k, n, s, seed + 1)
        res = oracle.dgemm(A, B, quant=oracle.TZ)
        for i in range(m):
            for j in range(n):
                exact = sum(Fraction(float(A[i, l])) * Fraction(float(B[l, j])) for l in range(k))
                si, tj = int(res.sigma[i]), int(res.tau[j])
                bound = (Fraction(2) ** (-tj) * sum(abs(Fraction(float(A[i, l]))) for l in range(k))
                         + Fraction(2) ** (-si) * sum(abs(Fraction(float(B[l, j]))) for l in range(k))
                         + k * Fraction(2) ** (-si - tj)
                         + Fraction(abs(float(res.C[i, j]))) * Fraction(1, 2 ** 53))
                assert abs(Fraction(float(res.C[i, j])) - exact) <= bound


def test_tz_integer_inputs_are_exact():
    rng = np.random.default_rng(12)
    A = rng.integers(-1000, 1000, size=(7, 9)).astype(np.float64)
    B = rng.integers(-1000, 1000, size=(9, 8)).astype(np.float64)
    for set in (0, 1):
        res = oracle.dgemm(A, B, quant=oracle.TZ, set=set)
        assert np.array_equal(res.C, (A.astype(np.int64) @ B.astype(np.int64)).astype(np.float64))


def test_tz_differs_from_rn_on_generic_data():
    """The variants are not the same computation: on generic data some
    quantised entries differ (by exactly one) and so do some outputs."""
    A = workloads.random_matrix(8, 50, 1.0, 21)
    B = workloads.random_matrix(50, 8, 1.0, 22)
    rn = oracle.dgemm(A, B)
    tz = oracle.dgemm(A, B, quant=oracle.TZ)
    d = rn.ZA - tz.ZA
    assert np.all(np.abs(d) <= 1) and np.any(d != 0)
    assert np.all(np.abs(tz.ZA) <= np.abs(A * 2.0 ** rn.sigma[:, None]))
    assert not np.array_equal(rn.C, tz.C)
