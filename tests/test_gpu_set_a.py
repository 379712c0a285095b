"""Parity of the HIP path with the CPU oracle for the all-byte modulus set
(Sec. 5.1, candidate A) on the int8 route, stage by stage and end to end.

Planes (int8 residues), per-modulus products and exponents must match bit
for bit, the FP64 output to 0 ulp (any NaN matches any NaN).  Shapes span
several output tiles of both shapes, several 128-byte k stages and ragged tails;
k values reach both residue paths of the deconstruction (scale bits above
and at most 51) and the int32 segment reduction of the product (k beyond
65536)."""
import math

import numpy as np
import pytest

import oracle
import paper_2609_09095_amd as oz
import workloads
from gpu_util import (device_layout, assert_bits_equal, assert_int_equal, gpu_deconstruct, gpu_dgemm, int8_bytes,
                      log, require_gpu, to_dev)

pytestmark = pytest.mark.gpu
SET = oz.A15      # the device library's number for the all-byte set
OSET = 1          # the oracle's


@pytest.fixture(scope="module", autouse=True)
def gpu():
    require_gpu()


def _oracle_side(X, side):
    k = X.shape[1] if side == 0 else X.shape[0]
    t = oracle.scale_bits(k, OSET)
    e = oracle.exponents(X, side, t)
    Z = oracle.quantise_vectors(X, side, e)
    return e, oracle.planes(Z, set=OSET)


def _edge_matrix(rows, k, seed):
    rng = np.random.default_rng(seed)
    X = workloads.random_matrix(rows, k, 1.0, seed)
    X[0] = 0.0
    X[1] = rng.standard_normal(k) * 1e-310
    X[2] = 0.0
    X[2, k // 2] = 5e-324
    X[3, 3 % k] = np.nan
    X[4, 1 % k] = -np.inf
    X[5] = rng.standard_normal(k) * 1e300
    X[5, 0] = 1.7e308
    X[6] = np.round(rng.standard_normal(k) * 1000)
    X[7] = rng.standard_normal(k)
    X[7, 0] = 1e6
    X[8] = (rng.integers(-64, 64, size=k) + 0.5) * 2.0 ** -50
    X[8, 0] = 1.0
    X[9] = -0.0
    X[10] = rng.standard_normal(k) * 2.0 ** -1020
    return X


# ------------------------------------------------------------ deconstruction
@pytest.mark.parametrize("shape,s,seed", [((64, 64), 0.5, 1), ((5, 70), 1.0, 2), ((130, 129), 2.0, 3),
                                          ((1, 1), 1.0, 4), ((33, 1000), 0.5, 5), ((9, 8192), 1.0, 6),
                                          ((3, 9000), 4.0, 7), ((17, 4096), 1.0, 8), ((9, 1800), 2.0, 9),
                                          ((5, 7000), 0.5, 10)])
@pytest.mark.parametrize("side", [0, 1])
def test_deconstruct_matches_oracle(shape, s, seed, side):
    X = workloads.random_matrix(shape[0], shape[1], s, seed)
    if side == 1:
        X = np.ascontiguousarray(X.T)
    k = X.shape[1] if side == 0 else X.shape[0]
    log(f"[A15] deconstruct side={side} shape={X.shape} t={oracle.scale_bits(k, OSET)}")
    planes, exps = gpu_deconstruct(X, side, SET)
    e, P = _oracle_side(X, side)
    assert planes.shape[1] == 15
    assert_int_equal(exps.cpu().numpy(), e, "exponents")
    assert_int_equal(planes.cpu().numpy(), device_layout(int8_bytes(P)), "planes")


@pytest.mark.parametrize("side", [0, 1])
@pytest.mark.parametrize("k", [1, 63, 200, 8000])
def test_deconstruct_edge_values(side, k):
    log(f"[A15] deconstruct edge values side={side} k={k}")
    X = _edge_matrix(12, k, 10 + k)
    if side == 1:
        X = np.ascontiguousarray(X.T)
    planes, exps = gpu_deconstruct(X, side, SET)
    e, P = _oracle_side(X, side)
    assert_int_equal(exps.cpu().numpy(), e, "exponents")
    assert_int_equal(planes.cpu().numpy(), device_layout(int8_bytes(P)), "planes")
    assert exps.cpu().numpy()[3] == oz.EXP_NONFINITE and exps.cpu().numpy()[4] == oz.EXP_NONFINITE


@pytest.mark.parametrize("k", [8192, 4096, 1024, 64])
def test_deconstruct_boundary_residues(k):
    """Rows whose scaled integers sit on every residue boundary: multiples of
    each modulus plus and minus half of it (the -128 endpoint of 256, the
    +-(m-1)/2 ends of the odd moduli, quotients next to a half integer), at
    the top of the scale range; a second set of rows reaches |y| just below
    2^t.  t = 51, 52, 53 and 55: each residue route (the nearest quotient
    with ylo from the magic sum or split off, and the corrected quotient)."""
    t = oracle.scale_bits(k, OSET)
    log(f"[A15] deconstruct boundary residues k={k} t={t}")
    rng = np.random.default_rng(5)
    X = np.zeros((4 * 15, k))
    for i, m in enumerate(oracle.moduli(OSET)):
        q = rng.integers(-(1 << (t - 9)), 1 << (t - 9), size=k)
        X[2 * i] = (q * m + m // 2).astype(np.float64)
        X[2 * i + 1] = (q * m - m // 2).astype(np.float64)
        X[2 * i, 0] = X[2 * i + 1, 0] = 2.0 ** (t - 1)   # sets the scale to 2^0
        top = (1 << t) // m
        q = rng.integers(top - 1024, top, size=k) * rng.choice([-1, 1], size=k)
        X[30 + 2 * i] = (q * m + m // 2).astype(np.float64)
        X[30 + 2 * i + 1] = (q * m - m // 2).astype(np.float64)
        X[30 + 2 * i, 0] = X[30 + 2 * i + 1, 0] = float((1 << t) - 1)   # scale 2^0, |y| < 2^t
    # past 2^53 the integers round to doubles: keep every one below 2^t
    lim = np.nextafter(2.0 ** t, 0.0)
    X = np.clip(X, -lim, lim)
    assert np.all(np.abs(X) < 2.0 ** t)
    planes, exps = gpu_deconstruct(X, 0, SET)
    e, P = _oracle_side(X, 0)
    assert_int_equal(exps.cpu().numpy(), e, "exponents")
    assert_int_equal(planes.cpu().numpy(), device_layout(int8_bytes(P)), "planes")


# ------------------------------------------------------------ residue products
def _quantised(m, n, k, seed):
    A = workloads.random_matrix(m, k, 1.0, seed)
    B = workloads.random_matrix(k, n, 1.0, seed + 50)
    t = oracle.scale_bits(k, OSET)
    ZA = oracle.quantise_vectors(A, 0, oracle.exponents(A, 0, t))
    ZB = oracle.quantise_vectors(B, 1, oracle.exponents(B, 1, t))
    return ZA, ZB


def _gemm_check(ZA, ZB):
    import torch
    m, k = ZA.shape
    n = ZB.shape[0]
    PA = device_layout(int8_bytes(oracle.planes(ZA, set=OSET)))
    PB = device_layout(int8_bytes(oracle.planes(ZB, set=OSET)))
    C = oz.ozaki25_residue_gemm(m, n, k, to_dev(PA), to_dev(PB), set=SET)
    torch.cuda.synchronize()
    want = oracle.residue_gemm(oracle.residues(ZA, OSET), oracle.residues(ZB, OSET), OSET)
    assert_int_equal(C.cpu().numpy(), want, "per-modulus products")


@pytest.mark.parametrize("m,n,k,seed", [(64, 64, 64, 1), (1, 1, 1, 2), (130, 200, 129, 3),
                                        (257, 129, 700, 4), (5, 300, 64, 5), (128, 128, 1, 6),
                                        (300, 520, 384, 7)])
def test_residue_gemm_matches_oracle(m, n, k, seed):
    log(f"[A15] residue gemm m={m} n={n} k={k}")
    _gemm_check(*_quantised(m, n, k, seed))


def test_residue_gemm_full_range_residues():
    log("[A15] residue gemm with uniform residues")
    rng = np.random.default_rng(78)
    m, n, k = 96, 160, 320
    ZA = rng.integers(-(1 << 62), 1 << 62, size=(m, k), dtype=np.int64)
    ZB = rng.integers(-(1 << 62), 1 << 62, size=(n, k), dtype=np.int64)
    _gemm_check(ZA, ZB)


@pytest.mark.parametrize("k", [65536, 65664, 140000])
def test_residue_gemm_long_extreme_rows(k):
    """Every residue of every row -128 mod 256 (the largest int8 product,
    2^14 per term, same sign): the int32 sums grow linearly and would
    overflow past k = 131071 without the segment reduction."""
    log(f"[A15] residue gemm, extreme constant rows, k={k}")
    rng = np.random.default_rng(k)
    m, n = 24, 40
    za = rng.integers(-(1 << 40), 1 << 40, size=(m, 1), dtype=np.int64) * 256 - 128
    zb = rng.integers(-(1 << 40), 1 << 40, size=(n, 1), dtype=np.int64) * 256 - 128
    _gemm_check(np.repeat(za, k, axis=1), np.repeat(zb, k, axis=1))


def test_residue_gemm_k_zero_writes_zeros():
    import torch
    C = torch.full((15, 3, 4), 7, dtype=torch.int32, device="cuda")
    dummy = torch.zeros(16, dtype=torch.uint8, device="cuda")
    oz.ozaki25_residue_gemm(3, 4, 0, dummy, dummy, C, set=SET)
    torch.cuda.synchronize()
    assert not C.cpu().numpy().any()


# ------------------------------------------------------------ reconstruction
def _centred(x, m):
    r = x % m
    return r - m if 2 * r >= m else r


def _random_X(rng, count):
    M = oracle.product_of_moduli(OSET)
    h = M // 2
    xs = [0, 1, -1, -h, h - 1, h - 2, -h + 1, (1 << 53) + 1, -(1 << 53) - 1, (1 << 116) + 3,
          -(1 << 116) - 5, (1 << 113) + 1, -(1 << 114) + 7]
    while len(xs) < count:
        b = int(rng.integers(0, 118))
        x = (int(rng.integers(0, 1 << 62)) << 62) | int(rng.integers(0, 1 << 62))
        x %= (1 << b) if b else 1
        x = -x if rng.random() < 0.5 else x
        if -h <= x < h:
            xs.append(x)
    return xs[:count]


@pytest.mark.parametrize("subtract", [False, True])
def test_reconstruct_matches_oracle(subtract):
    log(f"[A15] reconstruct subtract={subtract}")
    import torch
    rng = np.random.default_rng(32)
    m, n = 37, 300
    mods = oracle.moduli(OSET)
    Xs = _random_X(rng, m * n)
    Cres = np.array([[_centred(x, mm) for x in Xs] for mm in mods], dtype=np.int32).reshape(15, m, n)
    ea = rng.integers(-1100, 1200, size=m).astype(np.int32)
    eb = rng.integers(-1100, 1200, size=n).astype(np.int32)
    ea[0] = oz.EXP_NONFINITE
    eb[5] = oz.EXP_NONFINITE
    ea[1], eb[1] = 1074 + 60, 0
    ea[2], eb[2] = -1000, 0
    ea[3], eb[3] = 1074 + 118, 0      # the whole magnitude below the rounding point
    C0 = workloads.random_matrix(m, n, 1.0, 8) if subtract else None
    Cd = to_dev(C0) if subtract else torch.empty((m, n), dtype=torch.float64, device="cuda")
    oz.ozaki25_reconstruct(to_dev(Cres), to_dev(ea), to_dev(eb), Cd, subtract=subtract, set=SET)
    torch.cuda.synchronize()
    hi, lo = oracle.garner(Cres, OSET)
    want = oracle.reconstruct(hi, lo, ea, eb, C0)
    assert_bits_equal(Cd.cpu().numpy(), want, "reconstructed C")


def test_reconstruct_exact_ties():
    log("[A15] reconstruct ties up to 116 bits")
    import torch
    mods = oracle.moduli(OSET)
    Xs = []
    for b in range(54, 117):
        for odd in (0, 1):
            x = (1 << b) + (odd << (b - 52)) + (1 << (b - 53))
            Xs += [x, -x, x + 1, -x - 1]
    n = len(Xs)
    Cres = np.array([[_centred(x, mm) for x in Xs] for mm in mods], dtype=np.int32).reshape(15, 1, n)
    ea = np.zeros(1, np.int32)
    eb = np.zeros(n, np.int32)
    Cd = oz.ozaki25_reconstruct(to_dev(Cres), to_dev(ea), to_dev(eb), set=SET)
    torch.cuda.synchronize()
    hi, lo = oracle.garner(Cres, OSET)
    assert_bits_equal(Cd.cpu().numpy(), oracle.reconstruct(hi, lo, ea, eb), "ties")
    assert_bits_equal(Cd.cpu().numpy()[0], np.array([float(x) for x in Xs]), "ties vs CPython")


def test_reconstruct_near_rounding_boundaries():
    """Values at and next to rounding boundaries at every magnitude, near
    small multiples of the high half's weight and at the range ends, unscaled
    and scaled to land on the subnormal and overflow thresholds: bit for bit
    with the oracle, and unscaled with CPython's correctly rounded int to
    float conversion."""
    log("[A15] reconstruct near rounding boundaries")
    import torch
    mods = oracle.moduli(OSET)
    M = oracle.product_of_moduli(OSET)
    Xs = workloads.boundary_values(M, _high_weight(mods))
    n = len(Xs)
    Cres = np.array([[_centred(x, mm) for x in Xs] for mm in mods], dtype=np.int32).reshape(15, 1, n)
    hi, lo = oracle.garner(Cres, OSET)
    ea = np.zeros(1, np.int32)
    eb = np.zeros(n, np.int32)
    Cd = oz.ozaki25_reconstruct(to_dev(Cres), to_dev(ea), to_dev(eb), set=SET)
    torch.cuda.synchronize()
    assert_bits_equal(Cd.cpu().numpy(), oracle.reconstruct(hi, lo, ea, eb), "unscaled")
    assert_bits_equal(Cd.cpu().numpy()[0], np.array([float(x) for x in Xs]), "unscaled vs CPython")
    # sigma_i + tau_j = -e puts each result at exponent bitlen(X) - 1 + e
    for target in (-1022, -1023, -1030, -1075, 1023, 1024):
        eb = np.array([-(target - (abs(x).bit_length() - 1)) for x in Xs], dtype=np.int32)
        Cd = oz.ozaki25_reconstruct(to_dev(Cres), to_dev(ea), to_dev(eb), set=SET)
        torch.cuda.synchronize()
        assert_bits_equal(Cd.cpu().numpy(), oracle.reconstruct(hi, lo, ea, eb), f"result exponent {target}")


def _high_weight(mods):
    """Product of the moduli below the reconstruction's high half."""
    split = 6 if len(mods) == 12 else 7
    return math.prod(int(m) for m in mods[:split])


# ------------------------------------------------------------ end to end
@pytest.mark.parametrize("m,n,k,s,seed", [(64, 64, 64, 0.5, 1), (1, 1, 1, 1.0, 2), (3, 5, 7, 1.0, 3),
                                          (130, 129, 65, 2.0, 4), (257, 1, 300, 1.0, 5),
                                          (1, 300, 257, 1.0, 6), (200, 190, 1000, 4.0, 7),
                                          (70, 260, 8192, 1.0, 8), (300, 272, 200, 1.0, 9),
                                          (70, 528, 130, 2.0, 10), (300, 112, 150, 1.0, 11)])
def test_dgemm_matches_oracle(m, n, k, s, seed):
    log(f"[A15] dgemm m={m} n={n} k={k} s={s}")
    A = workloads.random_matrix(m, k, s, seed)
    B = workloads.random_matrix(k, n, s, seed + 1)
    C = gpu_dgemm(A, B, set=SET)
    r = oracle.dgemm(A, B, want_planes=False, set=OSET)
    assert_bits_equal(C.cpu().numpy(), r.C, "C")


def test_dgemm_edge_values():
    log("[A15] dgemm with zero, subnormal, NaN, infinite and huge rows/columns")
    A = _edge_matrix(12, 40, 3)
    B = np.ascontiguousarray(_edge_matrix(12, 40, 4).T)
    C = gpu_dgemm(A, B, set=SET)
    r = oracle.dgemm(A, B, want_planes=False, set=OSET)
    assert_bits_equal(C.cpu().numpy(), r.C, "C")
    got = C.cpu().numpy()
    assert np.all(np.isnan(got[3])) and np.all(np.isnan(got[:, 3]))
    assert not np.any(np.isfinite(got[4])) and not np.any(np.isfinite(got[:, 4]))


def test_dgemm_integer_inputs_are_exact():
    log("[A15] dgemm small integers")
    rng = np.random.default_rng(13)
    A = rng.integers(-1000, 1000, size=(70, 90)).astype(np.float64)
    B = rng.integers(-1000, 1000, size=(90, 80)).astype(np.float64)
    C = gpu_dgemm(A, B, set=SET)
    assert np.array_equal(C.cpu().numpy(), (A.astype(np.int64) @ B.astype(np.int64)).astype(np.float64))


def test_dgemm_sub_matches_oracle():
    log("[A15] dgemm_sub 100x120x333")
    A = workloads.random_matrix(100, 333, 1.0, 43)
    B = workloads.random_matrix(333, 120, 1.0, 44)
    C0 = workloads.random_matrix(100, 120, 1.0, 45)
    C = gpu_dgemm(A, B, C0, set=SET)
    r = oracle.dgemm(A, B, C_in=C0, want_planes=False, set=OSET)
    assert_bits_equal(C.cpu().numpy(), r.C, "C - AB")


def test_dgemm_k_zero():
    import torch
    A = torch.empty((3, 0), dtype=torch.float64, device="cuda")
    B = torch.empty((0, 4), dtype=torch.float64, device="cuda")
    C = torch.full((3, 4), 5.0, dtype=torch.float64, device="cuda")
    oz.ozaki25_dgemm(A, B, C, set=SET)
    torch.cuda.synchronize()
    assert np.all(C.cpu().numpy() == 0) and not np.any(np.signbit(C.cpu().numpy()))


def test_dgemm_strided_operands_and_workspace():
    log("[A15] dgemm_ex with leading dimensions and a caller workspace")
    import torch
    m, n, k = 77, 66, 150
    A = workloads.random_matrix(m, k, 1.0, 52)
    B = workloads.random_matrix(k, n, 1.0, 53)
    Ab = torch.zeros((m, k + 9), dtype=torch.float64, device="cuda")
    Bb = torch.zeros((k, n + 3), dtype=torch.float64, device="cuda")
    Cb = torch.full((m, n + 5), 3.0, dtype=torch.float64, device="cuda")
    Ab[:, :k] = to_dev(A)
    Bb[:, :n] = to_dev(B)
    ws = torch.empty(oz.ozaki25_dgemm_workspace_size(m, n, k, SET), dtype=torch.uint8, device="cuda")
    oz.ozaki25_dgemm_ex(Ab[:, :k], Bb[:, :n], Cb[:, :n], workspace=ws, set=SET)
    torch.cuda.synchronize()
    r = oracle.dgemm(A, B, want_planes=False, set=OSET)
    assert_bits_equal(Cb[:, :n].cpu().numpy(), r.C, "C")
    assert np.all(Cb[:, n:].cpu().numpy() == 3.0)


@pytest.mark.parametrize("m,n,k,seed", [(40, 300, 8576, 91), (24, 40, 70000, 92), (256, 256, 8192, 93)])
def test_dgemm_split_k_matches_oracle(m, n, k, seed):
    """Split k range for few output tiles (int8 kernel, partial residue
    bytes summed mod m)."""
    log(f"[A15] dgemm split-k m={m} n={n} k={k}")
    A = workloads.random_matrix(m, k, 1.0, seed)
    B = workloads.random_matrix(k, n, 1.0, seed + 1)
    C = gpu_dgemm(A, B, set=SET)
    r = oracle.dgemm(A, B, want_planes=False, set=OSET)
    assert_bits_equal(C.cpu().numpy(), r.C, "C")


@pytest.mark.parametrize("m,n,k,seed", [(300, 128, 700, 94), (300, 129, 700, 95), (513, 96, 2000, 96)])
def test_dgemm_narrow_tiles_match_oracle(m, n, k, seed):
    log(f"[A15] dgemm narrow m={m} n={n} k={k}")
    A = workloads.random_matrix(m, k, 1.0, seed)
    B = workloads.random_matrix(k, n, 1.0, seed + 1)
    C = gpu_dgemm(A, B, set=SET)
    r = oracle.dgemm(A, B, want_planes=False, set=OSET)
    assert_bits_equal(C.cpu().numpy(), r.C, "C")
