"""Pins of the oracle's accurate mode (Sec. 2, Eq. (alpha): one extra
low-precision GEMM bounds the input magnitudes, alpha = 3r + 1 products).

The paper fixes what the mode must achieve -- every entry of A'B' inside
[-M/2, M/2) (Eq. (moduli)) with scales chosen from a magnitude bound -- but
not the bound's encoding; the reading pinned here is: digits
ceil(16 |x| 2^-e) in {0..16}, their exact product U, the largest total
shift L_ij with 2^L U_ij <= 2^8 (M/2 - 1), split into column shifts
u_j = floor(min_i L_ij / 2) and row shifts s_i = min_j (L_ij - u_j), both
capped at 58.  Expected values come from Python integers and Fractions, the
published modulus list (tests/golden/modulus_set.json), numpy's integer
matmul, closed forms on saturating inputs, and brute force on tiny shapes.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
CAP = 58


def _mods(set):
    if set == 0:
        with open(os.path.join(GOLDEN, "modulus_set.json")) as f:
            return json.load(f)["moduli"]
    with open(os.path.join(GOLDEN, "modulus_set_a.json")) as f:
        return json.load(f)["moduli"]


def _limit(set):
    """2^8 (M/2 - 1) from the published moduli."""
    return (math.prod(_mods(set)) // 2 - 1) << 8


def _frexp_e(v):
    v = [abs(float(x)) for x in v]
    return math.frexp(max(v))[1] if max(v) > 0 else 0


def _digit(x, e):
    return math.ceil(abs(Fraction(float(x))) * 16 / Fraction(2) ** e)


def test_alpha_is_one_more_than_fast_mode():
    with open(os.path.join(GOLDEN, "modulus_set.json")) as f:
        g = json.load(f)
    assert g["alpha_accurate_mode"] == 3 * g["r"] + 1


def test_mag_digit_vs_fraction():
    rng = np.random.default_rng(11)
    for _ in range(3000):
        e = int(rng.integers(-1070, 1020))
        x = math.ldexp(float(rng.random()), e) * (1 if rng.random() < 0.5 else -1)
        if rng.random() < 0.1:  # largest magnitude below 2^e
            x = math.copysign(math.ldexp(1 - 2.0 ** -53, e), x)
        if rng.random() < 0.05:  # exact multiples of 2^{e-4}
            x = math.ldexp(int(rng.integers(0, 16)), e - 4)
        if rng.random() < 0.05:  # scaled value below the normal range
            x = math.ldexp(1.0, int(rng.integers(-1074, -1000))) * (1 if rng.random() < 0.5 else -1)
            e = int(rng.integers(-20, 1020))
        d = oracle.mag_digit(x, e)
        assert d == _digit(x, e) and 0 <= d <= 16
        assert (d == 0) == (x == 0)
        assert abs(Fraction(x)) <= d * Fraction(2) ** (e - 4) < abs(Fraction(x)) + Fraction(2) ** (e - 4)


def test_mag_digit_far_below_the_maximum():
    for x, e in [(5e-324, 1000), (-5e-324, 4), (2.0 ** -1000, 80), (2.0 ** -1022, 60)]:
        assert oracle.mag_digit(x, e) == _digit(x, e) == 1


def test_mag_digits_vectors_and_flags():
    A = workloads.random_matrix(7, 33, 2.0, 5)
    A[3] = 0.0
    A[5, 2] = np.nan
    eA = oracle.frexp_exponents(A, 0)
    assert eA[5] == oracle.NONFINITE and eA[3] == 0
    for i in (0, 1, 2, 4, 6):
        assert eA[i] == _frexp_e(A[i])
    D = oracle.mag_digits(A, 0, eA)
    assert not D[3].any() and not D[5].any()
    for i in (0, 1, 2, 4, 6):
        assert D[i].tolist() == [_digit(x, int(eA[i])) for x in A[i]]
        assert D[i].max() >= 8  # the largest magnitude is at least 2^{e-1}
    B = workloads.random_matrix(33, 6, 0.5, 6)
    eB = oracle.frexp_exponents(B, 1)
    DB = oracle.mag_digits(B, 1, eB)
    for j in range(6):
        assert eB[j] == _frexp_e(B[:, j])
        assert DB[j].tolist() == [_digit(x, int(eB[j])) for x in B[:, j]]


def test_bound_gemm_vs_numpy():
    rng = np.random.default_rng(3)
    DA = rng.integers(0, 17, size=(9, 301)).astype(np.uint8)
    DB = rng.integers(0, 17, size=(7, 301)).astype(np.uint8)
    U = oracle.bound_gemm(DA, DB)
    assert np.array_equal(U, DA.astype(np.int64) @ DB.astype(np.int64).T)
    # the FP64 matmul route of large products agrees with the C loops
    DA = np.full((40, 5000), 16, np.uint8)
    DA[1::2] = rng.integers(0, 17, size=(20, 5000))
    DB = rng.integers(0, 17, size=(30, 5000)).astype(np.uint8)
    assert np.array_equal(oracle.bound_gemm(DA, DB, loops=True), oracle.bound_gemm(DA, DB, loops=False))


@pytest.mark.parametrize("set", [0, 1])
def test_acc_total_is_the_largest_safe_shift(set):
    T = _limit(set)
    us = [1, 2, 3, 255, 256, 257, 1 << 20, (1 << 24) - 1, 1 << 24, 256 * 65536, (1 << 31) - 1]
    us += [int(u) for u in np.random.default_rng(set).integers(1, 1 << 31, 200)]
    for U in us:
        L = oracle.acc_total(U, set)
        assert (U << L) <= T < (U << (L + 1)), (U, L)
    assert oracle.acc_total(0, set) >= 1000


@pytest.mark.parametrize("set", [0, 1])
@pytest.mark.parametrize("k", [1, 3, 64, 300, 1024, 4099])
def test_saturating_inputs_fill_the_range_exactly(set, k):
    """Every element just below 2^e (digit 16 everywhere, RN rounds each
    scaled value up to 2^s): A'B' = k 2^{s+u} must lie inside [-M/2, M/2)
    -- the oracle's CRT result equals the exact product -- and one more bit
    on either side would leave it: the shifts use the whole range."""
    m, n = 3, 4
    top = 1 - 2.0 ** -53
    A = np.full((m, k), top) * np.array([[1.0], [-4.0], [0.5]])
    B = np.full((k, n), top) * np.array([[2.0, -1.0, 8.0, -0.25]])
    res = oracle.dgemm(A, B, set=set, accurate=True, check_exact=True)
    _, _, U, s, u = oracle.accurate_exponents(A, B, set)
    assert (U == 256 * k).all()
    half = math.prod(_mods(set)) // 2
    tight = 0
    for i in range(m):
        for j in range(n):
            X = int(res.ZA[i].astype(object) @ res.ZB[j].astype(object))
            assert -half <= X < half
            # RN takes (1 - 2^-53) 2^s up to 2^s for s <= 52 (a tie to even
            # at 52); from 53 on the scaled value is already an integer
            a = 1 << int(s[i]) if s[i] <= 52 else (1 << int(s[i])) - (1 << int(s[i] - 53))
            b = 1 << int(u[j]) if u[j] <= 52 else (1 << int(u[j])) - (1 << int(u[j] - 53))
            assert abs(X) == k * a * b
            if s[i] < CAP and u[j] < CAP:
                assert k << int(s[i] + u[j] + 1) > half - 1
                tight += 1
    assert tight == m * n or k < 64  # small k: the cap of 58 binds first
    assert s.min() >= oracle.scale_bits(k, set) and u.min() >= oracle.scale_bits(k, set)


def _py_shifts(A, B, set):
    """Brute force of the reading with Python integers."""
    m, k = A.shape
    n = B.shape[1]
    T = _limit(set)
    eA = [_frexp_e(A[i]) for i in range(m)]
    eB = [_frexp_e(B[:, j]) for j in range(n)]
    DA = [[_digit(A[i, l], eA[i]) for l in range(k)] for i in range(m)]
    DB = [[_digit(B[l, j], eB[j]) for l in range(k)] for j in range(n)]
    BIG = 10 ** 6

    def total(U):
        if U == 0:
            return BIG
        L = 0
        while (U << (L + 1)) <= T:
            L += 1
        return L

    Ls = [[total(sum(DA[i][l] * DB[j][l] for l in range(k))) for j in range(n)] for i in range(m)]
    u = [min(CAP, min(Ls[i][j] for i in range(m)) // 2) for j in range(n)]
    s = [min(CAP, min(Ls[i][j] - u[j] for j in range(n))) for i in range(m)]
    return [s[i] - eA[i] for i in range(m)], [u[j] - eB[j] for j in range(n)]


def _py_round(X, e):
    """Correctly rounded X 2^e (Python's int/int division is)."""
    return float(X * 2 ** e) if e >= 0 else X / (1 << -e)


@pytest.mark.parametrize("set", [0, 1])
@pytest.mark.parametrize("shape,s,seed", [((5, 7, 9), 0.5, 1), ((4, 3, 65), 2.0, 2), ((3, 4, 1), 1.0, 3),
                                          ((6, 2, 200), 4.0, 4)])
def test_accurate_dgemm_matches_brute_force(set, shape, s, seed):
    m, n, k = shape
    A = workloads.random_matrix(m, k, s, seed)
    B = workloads.random_matrix(k, n, s, seed + 50)
    A[0, 0] = 0.0
    res = oracle.dgemm(A, B, set=set, accurate=True)
    sig, tau = _py_shifts(A, B, set)
    assert list(res.sigma) == sig and list(res.tau) == tau
    Aq = [[round(Fraction(float(A[i, l])) * Fraction(2) ** sig[i]) for l in range(k)] for i in range(m)]
    Bq = [[round(Fraction(float(B[l, j])) * Fraction(2) ** tau[j]) for l in range(k)] for j in range(n)]
    assert res.ZA.tolist() == Aq and res.ZB.tolist() == Bq
    C = np.array([[_py_round(sum(Aq[i][l] * Bq[j][l] for l in range(k)), -sig[i] - tau[j])
                   for j in range(n)] for i in range(m)])
    assert np.array_equal(res.C.view(np.uint64), C.view(np.uint64))


@pytest.mark.parametrize("set", [0, 1])
def test_accurate_error_bound_and_gain(set):
    """The a-priori bound of Eq. (scale) with the accurate shifts holds, and
    on normal data the accurate mode is several times more accurate than the
    fast rule (each side gains about log2(256 k / U) / 2 bits)."""
    m, n, k = 6, 5, 1024
    A = workloads.random_matrix(m, k, 1.0, 7 + set)
    B = workloads.random_matrix(k, n, 1.0, 17 + set)
    acc = oracle.dgemm(A, B, set=set, accurate=True)
    fast = oracle.dgemm(A, B, set=set)
    err_acc = err_fast = 0.0
    for i in range(m):
        for j in range(n):
            exact = sum(Fraction(float(A[i, l])) * Fraction(float(B[l, j])) for l in range(k))
            si, tj = int(acc.sigma[i]), int(acc.tau[j])
            bound = (Fraction(2) ** (-tj - 1) * sum(abs(Fraction(float(A[i, l]))) for l in range(k))
                     + Fraction(2) ** (-si - 1) * sum(abs(Fraction(float(B[l, j]))) for l in range(k))
                     + k * Fraction(2) ** (-si - tj - 2)
                     + Fraction(abs(float(acc.C[i, j]))) * Fraction(1, 2 ** 53))
            e = abs(Fraction(float(acc.C[i, j])) - exact)
            assert e <= bound
            err_acc = max(err_acc, float(e))
            err_fast = max(err_fast, float(abs(Fraction(float(fast.C[i, j])) - exact)))
    assert (acc.sigma >= fast.sigma).all() and (acc.tau >= fast.tau).all()
    assert err_acc <= err_fast / 4


@pytest.mark.parametrize("set", [0, 1])
def test_nonfinite_and_zero_vectors_leave_the_other_shifts_alone(set):
    A = workloads.random_matrix(6, 40, 2.0, 8)
    B = workloads.random_matrix(40, 5, 2.0, 9)
    sig0, tau0, _, _, _ = oracle.accurate_exponents(A, B, set)
    A2 = np.vstack([A, np.zeros((1, 40)), A[:1]])
    A2[-1, 3] = np.inf
    B2 = np.hstack([B, B[:, :1]])
    B2[7, -1] = np.nan
    sig, tau, U, s, u = oracle.accurate_exponents(A2, B2, set)
    assert np.array_equal(sig[:6], sig0) and np.array_equal(tau[:5], tau0)
    assert sig[-1] == oracle.NONFINITE and tau[-1] == oracle.NONFINITE
    assert s[6] == CAP and sig[6] == CAP  # zero row: e = 0, no constraint
    assert not U[6].any() and not U[-1].any() and not U[:, -1].any()
    res = oracle.dgemm(A2, B2, set=set, accurate=True)
    assert not res.C[6, :5].any()
    assert np.isnan(res.C[:, -1]).all() and not np.isfinite(res.C[-1]).any()
    assert np.array_equal(res.C[:6, :5], oracle.dgemm(A, B, set=set, accurate=True).C)
