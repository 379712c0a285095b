"""Pins of the CPU oracle against what the paper and the mathematics fix.

Nothing here retypes the oracle's formulas: every expected value comes from
the paper's printed numbers (``tests/golden``), from an independent library
routine (Python big integers and Fractions, CPython's correctly rounded
int/int division, torch's e4m3 conversion), from closed forms, or from brute
force on tiny inputs.
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


def golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# --------------------------------------------------------------- modulus set
def test_modulus_set_matches_paper():
    g = golden("modulus_set.json")
    mods = oracle.moduli()
    assert mods == g["moduli"]
    for a in range(len(mods)):
        for b in range(a + 1, len(mods)):
            assert math.gcd(mods[a], mods[b]) == 1
    M = oracle.product_of_moduli()
    assert M == math.prod(mods)
    assert round(math.log2(M), 1) == g["log2_M_printed"]
    assert [oracle.planes_of(i) for i in range(12)] == [2] * 6 + [3] * 6
    assert sum(oracle.planes_of(i) for i in range(12)) == g["p_store"]
    assert 3 * len(mods) == g["p_mma"]
    r = g["r"]
    assert r * (r - 1) // 2 + 2 * r == g["n_gamma"]
    for s in g["squares_sqrt"]:
        assert s * s in mods


def test_garner_constants_are_inverses():
    mods = oracle.moduli()
    w = oracle.garner_constants()
    for j in range(1, 12):
        assert (w[j] * math.prod(mods[:j])) % mods[j] == 1
        assert 0 < w[j] < mods[j]


# --------------------------------------------------------------- scale bits
@pytest.mark.parametrize("k", [1, 2, 3, 63, 64, 65, 255, 256, 1024, 4096, 7937, 8192, 29773, 1 << 22])
def test_scale_bits_is_the_largest_safe_t(k):
    """Eq. (moduli): |c'| <= k 2^{2t} must stay inside [-M/2, M/2).  The worst
    case A' = B' = 2^t (all ones at full scale) must round-trip through the
    residues, and t + 1 must not be safe any more."""
    M = oracle.product_of_moduli()
    t = oracle.scale_bits(k)
    mu = k * 4 ** t
    assert mu < M // 2 and -mu >= -(M // 2)
    assert k * 4 ** (t + 1) >= M // 2
    # the extreme product survives the CRT round trip through the oracle
    mods = oracle.moduli()
    for X in (mu, -mu):
        c = np.array([[[_centred(X, m)]] for m in mods], dtype=np.int32)
        hi, lo = oracle.garner(c)
        assert _signed(int(hi[0, 0]), int(lo[0, 0])) == X


def _centred(x, m):
    r = x % m
    return r - m if 2 * r >= m else r


def _signed(hi, lo):
    v = ((hi & ((1 << 64) - 1)) << 64) | lo
    return v - (1 << 128) if v >> 127 else v


def test_scale_bits_known_values():
    # values of t(k) for the workload shapes
    assert [oracle.scale_bits(k) for k in (64, 1024, 4096, 7937, 8192)] == [52, 50, 49, 48, 48]
    assert oracle.scale_bits(0) == -1


# --------------------------------------------------------------- residues
def test_worked_example_residue():
    g = golden("worked_example_byte_planes.json")
    x, m = g["x"], g["modulus"]
    assert x == int(g["x_hex"], 16)
    # the printed byte planes and constants are what they claim to be
    assert list(x.to_bytes(4, "little")) == g["byte_planes"]
    assert [pow(2, 8 * j, m) for j in range(4)] == g["constants"]
    lo, hi = g["constants_low_limb"], g["constants_high_limb"]
    assert [a + 256 * b for a, b in zip(lo, hi)] == g["constants"]
    b = g["byte_planes"]
    assert sum(p * q for p, q in zip(b, lo)) == g["dot_low"]
    assert sum(p * q for p, q in zip(b, hi)) == g["dot_high"]
    assert g["dot_low"] + 256 * g["dot_high"] == g["recombined"]
    # the oracle's centred residue reproduces the printed residue
    assert oracle.centred_mod(x, m) == g["residue"]
    assert oracle.centred_mod(g["recombined"], m) == g["residue"]


def test_byte_plane_constant_bounds():
    g = golden("byte_plane_constants.json")
    mods = oracle.moduli()
    consts = [[pow(2, 8 * j, m) for j in range(8)] for m in mods]
    assert max(max(c) for c in consts) == g["max_constant"]
    assert max(max(x >> 8 for x in c) for c in consts) <= g["max_high_limb"]
    assert 8 * 255 * 255 == g["dot_bound_lhs"] < 2 ** g["dot_bound_rhs_log2"]
    a, b = g["identical_high_limb_vectors"]
    assert [x >> 8 for x in consts[mods.index(a)]] == [x >> 8 for x in consts[mods.index(b)]]


def test_residues_exhaustive_16bit():
    """Signed residue equivalence, exhaustive over 16-bit z, including the
    even-modulus boundary -m/2 (validation criteria of Sec. 7)."""
    z = np.arange(-(1 << 15), 1 << 15, dtype=np.int64)[None, :]
    res = oracle.residues(z)
    for i, m in enumerate(oracle.moduli()):
        r = res[i, 0].astype(np.int64)
        assert np.all((z[0] - r) % m == 0)
        assert np.all(2 * r >= -m) and np.all(2 * r < m)
    # m = 1024: -512 included, +512 excluded
    assert oracle.centred_mod(512, 1024) == -512
    assert oracle.centred_mod(-512, 1024) == -512
    assert oracle.centred_mod(511, 1024) == 511
    assert oracle.centred_mod(544, 1089) == 544
    assert oracle.centred_mod(545, 1089) == -544


def test_residues_stratified_64bit():
    rng = np.random.default_rng(7)
    vals = [0, 1, -1, (1 << 52), -(1 << 52), (1 << 55), -(1 << 55), (1 << 62) - 1, -(1 << 62)]
    for b in range(1, 63):
        vals += [int(v) for v in rng.integers(-(1 << b), 1 << b, size=20)]
    z = np.array(vals, dtype=np.int64)[None, :]
    res = oracle.residues(z)
    for i, m in enumerate(oracle.moduli()):
        for zz, rr in zip(vals, res[i, 0]):
            rr = int(rr)
            assert (zz - rr) % m == 0 and -m <= 2 * rr < m


# --------------------------------------------------------------- limbs
def _e4m3_exact(values):
    import torch
    t = torch.tensor(values, dtype=torch.float32)
    back = t.to(torch.float8_e4m3fn).to(torch.float32)
    return (back == t).tolist()


def test_e4m3_membership_against_torch():
    vals = list(range(-460, 461))
    ref = _e4m3_exact(vals)
    mine = [oracle.in_e4m3(v) for v in vals]
    # torch's e4m3fn saturates at 448 as well; all integers > 448 are excluded
    assert mine == [r and abs(v) <= 448 for v, r in zip(vals, ref)]
    g = golden("lemma1_carry_layout.json")
    assert [v for v in range(-24, 25) if not oracle.in_e4m3(v)] == g["canonical_sums_not_in_e4m3"]


def test_lemma1_layout_exhaustive():
    g = golden("lemma1_carry_layout.json")
    mods = oracle.moduli()
    for m in g["nonsquare_moduli"]:
        i = mods.index(m)
        lo = -(m // 2)
        ds = list(range(lo, lo + m))
        L = [oracle.limbs(i, d) for d in ds]
        flat = sorted({x for l in L for x in l})
        ok = dict(zip(flat, _e4m3_exact(flat)))
        carried = 0
        for d, (d0, d1, s) in zip(ds, L):
            assert d0 + 16 * d1 == d
            assert s == d0 + d1
            assert ok[d0] and ok[d1] and ok[s]
            assert abs(d0) <= g["max_abs_d0"] and abs(d1) <= g["max_abs_d1"] and abs(s) <= g["max_abs_sum"]
            canon0 = ((d + 8) % 16) - 8
            if d0 != canon0:
                carried += 1
        if m == 511:
            assert carried == g["carried_residues_at_511"]
    assert g["max_abs_sum"] ** 2 == g["max_pair_product"]
    assert (1 << 24) // g["max_pair_product"] == g["exact_fp32_depth"]


def test_lemma1_bound_is_sharp():
    """All residues of m = 513 admit the layout; m = 514 has one that does not."""
    g = golden("lemma1_carry_layout.json")

    def layout_ok(m):
        lo = -(m // 2)
        for d in range(lo, lo + m):
            d0, d1, s = oracle.split16(d)
            if not (d0 + 16 * d1 == d and all(_e4m3_exact([d0, d1, s]))):
                return False
        return True

    assert layout_ok(g["sharp_bound_passes"])
    assert not layout_ok(g["sharp_bound_fails"])


def test_square_digits():
    g = golden("modulus_set.json")
    mods = oracle.moduli()
    for i, s in enumerate(g["squares_sqrt"]):
        m = s * s
        assert mods[i] == m
        lo = -(m // 2)
        for d in range(lo, lo + m):
            d0, d1 = oracle.limbs(i, d)
            assert d0 + s * d1 == d
            assert -s <= 2 * d0 < s                      # balanced base-s digit
            assert abs(d0) <= g["square_digit_max_abs"] and abs(d1) <= g["square_digit_max_abs"]
        # 16 s + 16 covers half the range; tight at s = 33
        assert 16 * s + 16 >= (m - 1) // 2
    s = g["square_span_tight_at"]
    assert 16 * s + 16 == (s * s - 1) // 2


@pytest.mark.parametrize("i", range(12))
def test_limb_epilogue_all_pairs(i):
    """Square epilogue {1, s, s} and Eq. (karcarry) over all m^2 ordered
    pairs: the limb combination is the product of the residues mod m."""
    m = oracle.moduli()[i]
    tab = oracle.limb_product_table(i).astype(np.int64)
    d = np.arange(m, dtype=np.int64) - m // 2
    prod = d[:, None] * d[None, :]
    assert np.all((tab - prod) % m == 0)
    assert np.all(2 * tab >= -m) and np.all(2 * tab < m)


def test_karatsuba_identity_exact_integers():
    """Eq. (karcarry) is an integer identity, not only a congruence."""
    g = golden("lemma1_carry_layout.json")["karatsuba_coefficients"]
    i = oracle.moduli().index(511)
    for d in range(-255, 256, 7):
        for e in range(-255, 256, 11):
            a = oracle.limbs(i, d)
            b = oracle.limbs(i, e)
            v = g["d0e0"] * a[0] * b[0] + g["sum"] * a[2] * b[2] + g["d1e1"] * a[1] * b[1]
            assert v == d * e


# --------------------------------------------------------------- quantiser
def test_quantise_round_half_even():
    cases = [(2.5, 0, 2), (3.5, 0, 4), (-2.5, 0, -2), (-3.5, 0, -4), (0.5, 0, 0), (-0.5, 0, 0),
             (1.5, 0, 2), (0.75, 1, 2), (0.25, 1, 0), (5e-324, 1074, 1), (5e-324, 1073, 0)]
    for x, s, want in cases:
        assert oracle.quantise(x, s) == want


def test_quantise_random_vs_fraction():
    rng = np.random.default_rng(11)
    for _ in range(3000):
        x = float(rng.standard_normal() * 2.0 ** int(rng.integers(-60, 60)))
        s = int(rng.integers(-80, 100))
        q = Fraction(x) * Fraction(2) ** s
        if abs(q) >= 2 ** 60:
            continue
        assert oracle.quantise(x, s) == round(q)   # Fraction.__round__ is half-even


# --------------------------------------------------------------- exponents
def test_exponents_frexp_definition():
    rng = np.random.default_rng(3)
    A = workloads.random_matrix(20, 37, 2.0, 5)
    A[3] = 0.0
    A[4, 5] = 5e-324
    A[4, :5] = 0.0
    A[4, 6:] = 0.0
    A[5, 2] = np.nan
    A[6, 9] = -np.inf
    A[7, :] = rng.standard_normal(37) * 1e-310   # subnormal row
    t = oracle.scale_bits(37)
    sig = oracle.exponents(A, 0, t)
    for r in range(20):
        row = A[r]
        if not np.all(np.isfinite(row)):
            assert sig[r] == oracle.NONFINITE
            continue
        mx = float(np.max(np.abs(row)))
        e = math.frexp(mx)[1]
        assert sig[r] == t - e
        if mx > 0:
            assert 2.0 ** (e - 1) <= mx < 2.0 ** e
    assert sig[3] == t                      # zero row: frexp(0) exponent is 0
    # columns of B use the same rule on the transposed view
    tau = oracle.exponents(A.T.copy(), 1, oracle.scale_bits(20))
    sig2 = oracle.exponents(A.copy(), 0, oracle.scale_bits(20))
    assert np.array_equal(tau, sig2)


# --------------------------------------------------------------- Garner
def test_garner_crt_round_trip():
    mods = oracle.moduli()
    M = math.prod(mods)
    rng = np.random.default_rng(5)
    Xs = [0, 1, -1, -(M // 2), M // 2 - 1, M // 4, -(M // 4) - 1]
    Xs += [int(rng.integers(0, 1 << 62)) * (1 << 49) + int(rng.integers(0, 1 << 49)) - M // 2 for _ in range(200)]
    Xs = [x for x in Xs if -(M // 2) <= x < M // 2]

    C = np.array([[[_centred(x, m) for x in Xs]] for m in mods], dtype=np.int32)
    hi, lo = oracle.garner(C)
    got = [_signed(int(h), int(l)) for h, l in zip(hi[0], lo[0])]
    assert got == Xs


# --------------------------------------------------------------- rounding
def _py_round(X, e):
    """CPython's int -> float conversions are correctly rounded (ties to even,
    subnormals included); int / int true division likewise."""
    if X == 0:
        return 0.0
    if e >= 0:
        try:
            return float(X * 2 ** e)
        except OverflowError:
            return math.copysign(math.inf, X)
    return X / 2 ** (-e)


def test_round_scaled_matches_python():
    rng = np.random.default_rng(9)
    cases = [(1, 0), (3, -1), (-3, -1), ((1 << 53) + 1, 0), ((1 << 53) + 3, 0), ((1 << 54) + 2, 0),
             ((1 << 111) - 1, -1200), (-(1 << 111), 900), (1, -1074), (1, -1075), (3, -1076),
             (1, -1076), ((1 << 53) - 1, 971), ((1 << 53) - 1, 972), ((1 << 54) - 1, 970)]
    for _ in range(4000):
        bits = int(rng.integers(1, 112))
        X = int(rng.integers(0, 1 << 62)) * (1 << 50) + int(rng.integers(0, 1 << 50))
        X = X % (1 << bits)
        if rng.random() < 0.5:
            X = -X
        e = int(rng.integers(-1250, 1000))
        cases.append((X, e))
    # exact ties at the rounding position
    for b in range(54, 112, 3):
        cases.append(((1 << b) + (1 << (b - 53)), 0))
        cases.append(((1 << b) + (3 << (b - 54)), -5))
    for X, e in cases:
        got = oracle.round_scaled(X, e)
        want = _py_round(X, e)
        assert got == want and math.copysign(1, got) == math.copysign(1, want), (X, e, got, want)


# --------------------------------------------------------------- end to end
def _python_pipeline(A, B):
    """Independent brute force with Python integers and Fractions: the
    quantiser of Eq. (scale) by exact rational rounding, the exact product,
    and the correctly rounded rescale."""
    m, k = A.shape
    n = B.shape[1]
    t = oracle.scale_bits(k)
    sig = [t - math.frexp(float(np.max(np.abs(A[i]))))[1] for i in range(m)]
    tau = [t - math.frexp(float(np.max(np.abs(B[:, j]))))[1] for j in range(n)]
    Aq = [[round(Fraction(float(A[i, l])) * Fraction(2) ** sig[i]) for l in range(k)] for i in range(m)]
    Bq = [[round(Fraction(float(B[l, j])) * Fraction(2) ** tau[j]) for l in range(k)] for j in range(n)]
    X = [[sum(Aq[i][l] * Bq[j][l] for l in range(k)) for j in range(n)] for i in range(m)]
    C = np.array([[_py_round(X[i][j], -sig[i] - tau[j]) for j in range(n)] for i in range(m)])
    return sig, tau, Aq, Bq, X, C


@pytest.mark.parametrize("shape,s,seed", [((5, 7, 9), 0.5, 1), ((8, 3, 33), 1.0, 2), ((4, 6, 64), 2.0, 3),
                                          ((3, 4, 1), 1.0, 4), ((6, 5, 130), 4.0, 5)])
def test_dgemm_matches_bigint_brute_force(shape, s, seed):
    m, n, k = shape
    A = workloads.random_matrix(m, k, s, seed)
    B = workloads.random_matrix(k, n, s, seed + 100)
    res = oracle.dgemm(A, B)
    sig, tau, Aq, Bq, X, C = _python_pipeline(A, B)
    assert list(res.sigma) == sig and list(res.tau) == tau
    assert res.ZA.tolist() == Aq and res.ZB.tolist() == Bq
    for i in range(m):
        for j in range(n):
            assert _signed(int(res.Xhi[i, j]), int(res.Xlo[i, j])) == X[i][j]
    assert np.array_equal(res.C.view(np.uint64), C.view(np.uint64))
    # the per-modulus products are the residues of the exact product
    for q, mod in enumerate(oracle.moduli()):
        for i in range(m):
            for j in range(n):
                r = int(res.Cres[q, i, j])
                assert (X[i][j] - r) % mod == 0 and -mod <= 2 * r < mod


def test_dgemm_error_bound_vs_exact_product():
    """A-priori bound derived from Eq. (scale) with round to nearest:
    |C - AB| <= 2^{-tau-1} sum|a| + 2^{-sigma-1} sum|b| + k 2^{-sigma-tau-2} + u|C|."""
    for (m, n, k, s, seed) in [(6, 5, 40, 0.5, 1), (4, 4, 200, 1.0, 2), (5, 3, 64, 2.0, 3)]:
        A = workloads.random_matrix(m, k, s, seed)
        B = workloads.random_matrix(k, n, s, seed + 1)
        res = oracle.dgemm(A, B)
        for i in range(m):
            for j in range(n):
                exact = sum(Fraction(float(A[i, l])) * Fraction(float(B[l, j])) for l in range(k))
                si, tj = int(res.sigma[i]), int(res.tau[j])
                bound = (Fraction(2) ** (-tj - 1) * sum(abs(Fraction(float(A[i, l]))) for l in range(k))
                         + Fraction(2) ** (-si - 1) * sum(abs(Fraction(float(B[l, j]))) for l in range(k))
                         + k * Fraction(2) ** (-si - tj - 2)
                         + Fraction(abs(float(res.C[i, j]))) * Fraction(1, 2 ** 53))
                assert abs(Fraction(float(res.C[i, j])) - exact) <= bound


def test_dgemm_special_cases():
    rng = np.random.default_rng(2)
    # small integers are exact at t bits: C is the exact integer product
    A = rng.integers(-1000, 1000, size=(7, 50)).astype(np.float64)
    B = rng.integers(-1000, 1000, size=(50, 9)).astype(np.float64)
    res = oracle.dgemm(A, B)
    assert np.array_equal(res.C, (A.astype(np.int64) @ B.astype(np.int64)).astype(np.float64))
    # B = I: C_ij = 2^{-sigma_i} rint(2^{sigma_i} a_ij)
    A = workloads.random_matrix(6, 12, 2.0, 4)
    res = oracle.dgemm(A, np.eye(12))
    want = np.array([[Fraction(round(Fraction(float(A[i, j])) * Fraction(2) ** int(res.sigma[i])))
                      * Fraction(2) ** -int(res.sigma[i]) for j in range(12)] for i in range(6)], dtype=float)
    assert np.array_equal(res.C, want)
    # k = 1: one rounding of a'b'
    A = workloads.random_matrix(4, 1, 1.0, 8)
    B = workloads.random_matrix(1, 5, 1.0, 9)
    res = oracle.dgemm(A, B)
    for i in range(4):
        for j in range(5):
            X = int(res.ZA[i, 0]) * int(res.ZB[j, 0])
            assert res.C[i, j] == _py_round(X, -int(res.sigma[i]) - int(res.tau[j]))
    # zero matrices give +0.0
    res = oracle.dgemm(np.zeros((3, 4)), np.zeros((4, 2)))
    assert np.all(res.C == 0) and not np.any(np.signbit(res.C))


def _py_dot(a_row, b_col) -> float:
    """The index-order FP64 dot product in plain Python floats (IEEE binary64
    products and sums, each rounded; no fused multiply-add)."""
    s = 0.0
    for x, y in zip(a_row, b_col):
        s = s + float(x) * float(y)
    return s


def _same(x: float, y: float) -> bool:
    return (math.isnan(x) and math.isnan(y)) or (x == y and math.copysign(1, x) == math.copysign(1, y))


def _nonfinite_inputs():
    A = workloads.random_matrix(7, 8, 1.0, 1)
    B = workloads.random_matrix(8, 6, 1.0, 2)
    A[1, 3] = np.nan                       # NaN row
    A[2, 0] = np.inf                       # +Inf row; B[0, 4] = 0 below gives Inf * 0
    A[3, 2], A[3, 5] = np.inf, -np.inf     # Inf - Inf
    A[4, :2] = 1e308                       # finite terms overflow to +Inf ...
    A[4, 7] = -np.inf                      # ... then meet -Inf: NaN in this order
    B[6, 2] = np.inf                       # +Inf column
    B[0, 4] = 0.0
    B[:2, 5] = 1.0                         # column 5 drives row 4's overflow
    B[7, 5] = 2.0
    return A, B


def test_dgemm_nonfinite_rows_reissued_natively():
    """Alg. 1's last step (range check, native FP64 re-issue): every output
    of a row of A or column of B holding a NaN or infinity equals the
    index-order dot product in plain Python floats; every other output is the
    emulated value (the same as without the re-issue, and finite)."""
    A, B = _nonfinite_inputs()
    res = oracle.dgemm(A, B, check_exact=True)
    emu = oracle.dgemm(A, B, fallback=False).C
    flagged_rows = {1, 2, 3, 4}
    flagged_cols = {2}
    kinds = set()
    for i in range(A.shape[0]):
        for j in range(B.shape[1]):
            if i in flagged_rows or j in flagged_cols:
                want = _py_dot(A[i], B[:, j])
                assert _same(res.C[i, j], want), (i, j, res.C[i, j], want)
                assert not math.isfinite(want)
                kinds.add("nan" if math.isnan(want) else "inf")
                assert math.isnan(emu[i, j])          # the stage-wise reconstruction's NaN
            else:
                assert res.C[i, j] == emu[i, j] and math.isfinite(res.C[i, j])
    assert kinds == {"nan", "inf"}
    assert math.isnan(res.C[2, 4]) and math.isnan(res.C[3, 0]) and math.isnan(res.C[4, 5])
    assert res.C[2, 0] == _py_dot(A[2], B[:, 0]) and math.isinf(res.C[2, 0])
    # a flagged row quantises to zero planes
    assert not res.planesA[:, 1].any()


def test_dgemm_sub_nonfinite_rows_reissued_natively():
    A, B = _nonfinite_inputs()
    C0 = workloads.random_matrix(7, 6, 1.0, 3)
    C0[0, 2] = np.inf
    res = oracle.dgemm(A, B, C_in=C0)
    emu = oracle.dgemm(A, B, C_in=C0, fallback=False).C
    for i in range(7):
        for j in range(6):
            if i in (1, 2, 3, 4) or j == 2:
                assert _same(res.C[i, j], float(C0[i, j]) - _py_dot(A[i], B[:, j])), (i, j)
            else:
                assert res.C[i, j] == emu[i, j]


def test_dgemm_subtract_is_two_roundings():
    A = workloads.random_matrix(4, 16, 1.0, 3)
    B = workloads.random_matrix(16, 5, 1.0, 4)
    C0 = workloads.random_matrix(4, 5, 1.0, 5)
    plain = oracle.dgemm(A, B).C
    sub = oracle.dgemm(A, B, C_in=C0).C
    assert np.array_equal(sub, C0 - plain)


def test_planes_layout_and_padding():
    A = workloads.random_matrix(3, 70, 1.0, 6)
    res = oracle.dgemm(A, workloads.random_matrix(70, 2, 1.0, 7))
    P = res.planesA
    assert P.shape == (30, 3, 128)
    assert not P[:, :, 70:].any()   # zero padding up to the 128-byte plane row
    mods = oracle.moduli()
    for i, m in enumerate(mods):
        q = oracle.plane_base(i)
        base = 33 if i == 0 else (32 if i == 1 else int(round(math.sqrt(m))))
        for v in range(3):
            for l in range(70):
                d = _centred(int(res.ZA[v, l]), m)
                if i < 6:
                    assert int(P[q, v, l]) + base * int(P[q + 1, v, l]) == d
                else:
                    assert int(P[q, v, l]) + 16 * int(P[q + 1, v, l]) == d
                    assert int(P[q + 2, v, l]) == int(P[q, v, l]) + int(P[q + 1, v, l])


def test_workload_generator_is_deterministic():
    a1, b1, _ = workloads.make_inputs("tiny")
    a2, b2, _ = workloads.make_inputs("tiny")
    assert np.array_equal(a1, a2) and np.array_equal(b1, b2)
    assert a1.shape == (64, 64) and b1.shape == (64, 64)


def test_rounding_at_boundaries_matches_python():
    """Values at and next to FP64 rounding boundaries at every magnitude,
    unscaled and scaled onto the subnormal and overflow thresholds, round as
    CPython's correctly rounded conversions do."""
    mods = oracle.moduli()
    Xs = workloads.boundary_values(oracle.product_of_moduli(), math.prod(int(m) for m in mods[:6]))
    C = np.array([[[_centred(x, m) for x in Xs]] for m in mods], dtype=np.int32)
    hi, lo = oracle.garner(C)
    ea = np.zeros(1, np.int32)
    for target in (None, -1022, -1023, -1030, -1075, 1023, 1024):
        es = [0 if target is None else target - (abs(x).bit_length() - 1) for x in Xs]
        eb = np.array([-e for e in es], dtype=np.int32)
        got = oracle.reconstruct(hi, lo, ea, eb)[0]
        want = np.array([_py_round(x, e) for x, e in zip(Xs, es)])
        assert np.array_equal(got.view(np.uint64), want.view(np.uint64)), target
