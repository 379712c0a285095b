"""Pins of the oracle's all-byte modulus set (candidate A of Sec. 5.1) on the
INT8 route: every centred residue is itself the int8 operand, one product per
modulus.

Expected values come from the paper's printed numbers (``tests/golden``),
Python big integers and Fractions, CPython's correctly rounded conversions,
closed forms, and brute force on tiny inputs; none retypes the oracle.
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
SET_A = 1


def _golden():
    with open(os.path.join(GOLDEN, "modulus_set_a.json")) as f:
        return json.load(f)


def _centred(x, m):
    r = x % m
    return r - m if 2 * r >= m else r


def _signed(hi, lo):
    v = ((hi & ((1 << 64) - 1)) << 64) | lo
    return v - (1 << 128) if v >> 127 else v


def test_set_a_matches_paper():
    g = _golden()
    mods = oracle.moduli(SET_A)
    assert mods == g["moduli"]
    assert len(mods) == g["r_int8"] == oracle.num_moduli(SET_A)
    assert len(mods) + 1 == g["alpha_int8"]          # one int8 product per modulus, + 1
    assert 3 * 12 + 1 == g["alpha_fp8_published"]
    for a in range(len(mods)):
        assert mods[a] <= 256
        for b in range(a + 1, len(mods)):
            assert math.gcd(mods[a], mods[b]) == 1
    P = oracle.product_of_moduli(SET_A)
    assert P == math.prod(mods)
    assert round(math.log2(P), 1) == g["log2_P_printed"]
    # the published set is untouched by the set parameter
    assert oracle.moduli(0) == oracle.moduli()
    assert oracle.product_of_moduli(0) == oracle.product_of_moduli()


def test_set_a_garner_constants_are_inverses():
    mods = oracle.moduli(SET_A)
    w = oracle.garner_constants(SET_A)
    for j in range(1, len(mods)):
        assert (w[j] * math.prod(mods[:j])) % mods[j] == 1
        assert 0 < w[j] < mods[j]


def test_set_a_residues_exhaustive_16bit():
    """App. A items (ii) and (v): the centred residue in [-m/2, m/2), the even
    endpoint -128 of m = 256 included, on every 16-bit integer."""
    g = _golden()
    z = np.arange(-(1 << 15), 1 << 15, dtype=np.int64)[None, :]
    res = oracle.residues(z, SET_A)
    assert res.shape == (15, 1, 1 << 16)
    for i, m in enumerate(oracle.moduli(SET_A)):
        r = res[i, 0].astype(np.int64)
        assert np.all((z[0] - r) % m == 0)
        assert np.all(2 * r >= -m) and np.all(2 * r < m)
        assert np.all(r >= -128) and np.all(r <= 127)   # an int8 operand as it stands
    r256 = res[0, 0].astype(np.int64)
    assert r256.min() == g["even_endpoint_m256"] and r256.max() == 127
    assert int(r256[(1 << 15) + 128]) == -128 and int(r256[(1 << 15) - 128]) == -128


def test_set_a_residues_stratified_64bit():
    rng = np.random.default_rng(17)
    vals = [0, 1, -1, 128, -128, 255, (1 << 52), -(1 << 52), (1 << 62) - 1, -(1 << 62), -(1 << 63), (1 << 63) - 1]
    for b in range(1, 63):
        vals += [int(v) for v in rng.integers(-(1 << b), 1 << b, size=20)]
    z = np.array(vals, dtype=np.int64)[None, :]
    res = oracle.residues(z, SET_A)
    for i, m in enumerate(oracle.moduli(SET_A)):
        assert [int(r) for r in res[i, 0]] == [_centred(v, m) for v in vals]


def test_set_a_planes_are_the_residues():
    Z = np.array([[0, 128, -128, 255, -255, 256, 1 << 51, -(1 << 51) + 3, 12345]], dtype=np.int64)
    P = oracle.planes(Z, 128, set=SET_A)
    assert P.shape == (15, 1, 128) and P.dtype == np.int8
    assert not P[:, :, Z.shape[1]:].any()
    for i, m in enumerate(oracle.moduli(SET_A)):
        assert [int(x) for x in P[i, 0, :Z.shape[1]]] == [_centred(int(v), m) for v in Z[0]]


@pytest.mark.parametrize("k", [1, 2, 3, 64, 1024, 4096, 7937, 8192, 16384, 29773, 1 << 22])
def test_set_a_scale_bits_is_the_largest_safe_t(k):
    P = oracle.product_of_moduli(SET_A)
    t = oracle.scale_bits(k, SET_A)
    mu = k * 4 ** t
    assert mu < P // 2
    assert k * 4 ** (t + 1) >= P // 2
    mods = oracle.moduli(SET_A)
    for X in (mu, -mu):
        c = np.array([[[_centred(X, m)]] for m in mods], dtype=np.int32)
        hi, lo = oracle.garner(c, SET_A)
        assert _signed(int(hi[0, 0]), int(lo[0, 0])) == X


def test_set_a_scale_bits_closed_form():
    # log2(P/2) = 116.8..., so t = floor((116.8... - log2 k) / 2) with the
    # strict inequality; at k = 8192 that is 51, three bits above the published set's 48
    P = oracle.product_of_moduli(SET_A)
    for k in (64, 1024, 8192):
        t = 0
        while k * 4 ** (t + 1) < P // 2:
            t += 1
        assert oracle.scale_bits(k, SET_A) == t
    assert oracle.scale_bits(8192, SET_A) == 51 and oracle.scale_bits(8192) == 48


def test_set_a_garner_crt_round_trip():
    mods = oracle.moduli(SET_A)
    P = math.prod(mods)
    rng = np.random.default_rng(25)
    Xs = [0, 1, -1, -(P // 2), P // 2 - 1, P // 4, -(P // 4) - 1, 1 << 116, -(1 << 116)]
    for _ in range(300):
        x = 0
        for _ in range(2):
            x = (x << 62) | int(rng.integers(0, 1 << 62))
        Xs.append(x % P - P // 2)
    Xs = [x for x in Xs if -(P // 2) <= x < P // 2]
    C = np.array([[[_centred(x, m) for x in Xs]] for m in mods], dtype=np.int32)
    hi, lo = oracle.garner(C, SET_A)
    assert [_signed(int(h), int(l)) for h, l in zip(hi[0], lo[0])] == Xs


def _py_round(X, e):
    if X == 0:
        return 0.0
    if e >= 0:
        try:
            return float(X * 2 ** e)
        except OverflowError:
            return math.copysign(math.inf, X)
    return X / 2 ** (-e)


def test_round_scaled_above_113_bits():
    """Set A's products reach 117 bits: wider than binary128's significand,
    the rounding must still be a single correct one (CPython's int/int
    division and int->float conversion are)."""
    rng = np.random.default_rng(33)
    cases = []
    for b in range(110, 118):
        base = 1 << (b - 1)
        # ties and near-ties at the double rounding position, sticky bits
        # far below binary128's last place
        cases += [(base + (1 << (b - 54)), 0), (base + (1 << (b - 54)) + 1, 0),
                  (base + (3 << (b - 55)), -3), (base + (1 << (b - 54)) - 1, 7),
                  (-(base + (1 << (b - 54)) + 1), -1100), (base + 1, -1074 - b + 40)]
    for _ in range(3000):
        bits = int(rng.integers(100, 118))
        X = (int(rng.integers(0, 1 << 62)) << 62 | int(rng.integers(0, 1 << 62))) % (1 << bits)
        if rng.random() < 0.5:
            X = -X
        cases.append((X, int(rng.integers(-1300, 900))))
    for X, e in cases:
        got = oracle.round_scaled(X, e)
        want = _py_round(X, e)
        assert got == want and math.copysign(1, got) == math.copysign(1, want), (X, e, got, want)


def test_set_a_residue_gemm_brute_force():
    rng = np.random.default_rng(41)
    m, n, k = 5, 4, 300
    mods = oracle.moduli(SET_A)
    ZA = rng.integers(-(1 << 50), 1 << 50, size=(m, k))
    ZB = rng.integers(-(1 << 50), 1 << 50, size=(n, k))
    # extreme residues: every operand -128 on m = 256 (the largest int8 product)
    ZA[0, :] = -128
    ZB[0, :] = -128
    rA = oracle.residues(ZA, SET_A)
    rB = oracle.residues(ZB, SET_A)
    C = oracle.residue_gemm(rA, rB, SET_A)
    assert C.shape == (15, m, n)
    for q, mod in enumerate(mods):
        for i in range(m):
            for j in range(n):
                X = sum(int(a) * int(b) for a, b in zip(ZA[i], ZB[j]))
                assert int(C[q, i, j]) == _centred(X, mod)


def _python_pipeline(A, B):
    m, k = A.shape
    n = B.shape[1]
    t = oracle.scale_bits(k, SET_A)
    sig = [t - math.frexp(float(np.max(np.abs(A[i]))))[1] for i in range(m)]
    tau = [t - math.frexp(float(np.max(np.abs(B[:, j]))))[1] for j in range(n)]
    Aq = [[round(Fraction(float(A[i, l])) * Fraction(2) ** sig[i]) for l in range(k)] for i in range(m)]
    Bq = [[round(Fraction(float(B[l, j])) * Fraction(2) ** tau[j]) for l in range(k)] for j in range(n)]
    X = [[sum(Aq[i][l] * Bq[j][l] for l in range(k)) for j in range(n)] for i in range(m)]
    C = np.array([[_py_round(X[i][j], -sig[i] - tau[j]) for j in range(n)] for i in range(m)])
    return sig, tau, Aq, Bq, X, C


@pytest.mark.parametrize("shape,s,seed", [((5, 7, 9), 0.5, 1), ((4, 6, 64), 2.0, 3), ((6, 5, 130), 4.0, 5),
                                          ((3, 4, 1), 1.0, 4)])
def test_set_a_dgemm_matches_bigint_brute_force(shape, s, seed):
    m, n, k = shape
    A = workloads.random_matrix(m, k, s, seed)
    B = workloads.random_matrix(k, n, s, seed + 100)
    res = oracle.dgemm(A, B, set=SET_A)
    sig, tau, Aq, Bq, X, C = _python_pipeline(A, B)
    assert list(res.sigma) == sig and list(res.tau) == tau
    assert res.ZA.tolist() == Aq and res.ZB.tolist() == Bq
    for i in range(m):
        for j in range(n):
            assert _signed(int(res.Xhi[i, j]), int(res.Xlo[i, j])) == X[i][j]
    assert np.array_equal(res.C.view(np.uint64), C.view(np.uint64))
    assert res.planesA.shape[0] == 15 and res.planesA.dtype == np.int8


def test_set_a_is_at_least_as_accurate_as_published_set():
    """Three more scale bits per operand at this k: the summed error against
    the exact product is no larger than the published set's."""
    A = workloads.random_matrix(6, 200, 2.0, 11)
    B = workloads.random_matrix(200, 5, 2.0, 12)
    ra = oracle.dgemm(A, B, set=SET_A).C
    rs = oracle.dgemm(A, B).C
    ea = es = Fraction(0)
    for i in range(6):
        for j in range(5):
            exact = sum(Fraction(float(A[i, l])) * Fraction(float(B[l, j])) for l in range(200))
            ea += abs(Fraction(float(ra[i, j])) - exact)
            es += abs(Fraction(float(rs[i, j])) - exact)
    assert ea <= es


def test_rounding_at_boundaries_matches_python():
    """Values at and next to FP64 rounding boundaries at every magnitude,
    unscaled and scaled onto the subnormal and overflow thresholds, round as
    CPython's correctly rounded conversions do."""
    mods = oracle.moduli(1)
    Xs = workloads.boundary_values(oracle.product_of_moduli(1), math.prod(int(m) for m in mods[:7]))
    C = np.array([[[_centred(x, m) for x in Xs]] for m in mods], dtype=np.int32)
    hi, lo = oracle.garner(C, 1)
    ea = np.zeros(1, np.int32)
    for target in (None, -1022, -1023, -1030, -1075, 1023, 1024):
        es = [0 if target is None else target - (abs(x).bit_length() - 1) for x in Xs]
        eb = np.array([-e for e in es], dtype=np.int32)
        got = oracle.reconstruct(hi, lo, ea, eb)[0]
        want = np.array([_py_round(x, e) for x, e in zip(Xs, es)])
        assert np.array_equal(got.view(np.uint64), want.view(np.uint64)), target
