"""Parity of the HIP path with the CPU oracle, stage by stage and end to end.

Integer stages (exponents, planes, per-modulus products) must match bit for
bit; the FP64 output must match to 0 ulp (any NaN matches any NaN).  Sizes
here let the oracle finish in seconds while spanning several 128 x 128 output
tiles, several 64-byte k stages and ragged tails on every dimension."""
import math

import numpy as np
import pytest

import oracle
import paper_2609_09095_amd as oz
import workloads
from gpu_util import (device_layout, assert_bits_equal, assert_int_equal, e4m3_bytes, gpu_deconstruct, gpu_dgemm,
                      log, require_gpu, to_dev)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    require_gpu()


def _oracle_side(X, side):
    k = X.shape[1] if side == 0 else X.shape[0]
    t = oracle.scale_bits(k)
    e = oracle.exponents(X, side, t)
    Z = oracle.quantise_vectors(X, side, e)
    return e, oracle.planes(Z)


# ------------------------------------------------------------ deconstruction
@pytest.mark.parametrize("shape,s,seed", [((64, 64), 0.5, 1), ((5, 70), 1.0, 2), ((130, 129), 2.0, 3),
                                          ((1, 1), 1.0, 4), ((33, 1000), 0.5, 5), ((300, 17), 4.0, 6)])
@pytest.mark.parametrize("side", [0, 1])
def test_deconstruct_matches_oracle(shape, s, seed, side):
    log(f"deconstruct side={side} shape={shape} s={s} seed={seed}")
    X = workloads.random_matrix(shape[0], shape[1], s, seed)
    planes, exps = gpu_deconstruct(X, side)
    e, P = _oracle_side(X, side)
    assert_int_equal(exps.cpu().numpy(), e, "exponents")
    assert_int_equal(planes.cpu().numpy(), device_layout(e4m3_bytes(P)), "planes")


@pytest.mark.parametrize("k", [1024, 128, 64, 16])
def test_deconstruct_boundary_residues(k):
    """Rows whose scaled integers are multiples of each modulus plus and
    minus half of it (the ends of the centred range, quotients next to a
    half integer), and a second set reaching |y| just below 2^t, for
    t = 50, 51, 52 and 53: the nearest quotient route and the corrected one."""
    t = oracle.scale_bits(k)
    log(f"deconstruct boundary residues k={k} t={t}")
    rng = np.random.default_rng(7)
    mods = oracle.moduli()
    X = np.zeros((4 * len(mods), k))
    for i, m in enumerate(mods):
        q = rng.integers(-(1 << (t - 12)), 1 << (t - 12), size=k)
        X[2 * i] = (q * m + m // 2).astype(np.float64)
        X[2 * i + 1] = (q * m - m // 2).astype(np.float64)
        X[2 * i, 0] = X[2 * i + 1, 0] = 2.0 ** (t - 1)   # sets the scale to 2^0
        top = (1 << t) // m
        q = rng.integers(top - 1024, top, size=k) * rng.choice([-1, 1], size=k)
        r = 2 * len(mods) + 2 * i
        X[r] = (q * m + m // 2).astype(np.float64)
        X[r + 1] = (q * m - m // 2).astype(np.float64)
        X[r, 0] = X[r + 1, 0] = float((1 << t) - 1)   # scale 2^0, |y| < 2^t
    assert np.all(np.abs(X) < 2.0 ** t)
    for side in (0, 1):
        Xs = X if side == 0 else np.ascontiguousarray(X.T)
        planes, exps = gpu_deconstruct(Xs, side)
        e, P = _oracle_side(Xs, side)
        assert_int_equal(exps.cpu().numpy(), e, "exponents")
        assert_int_equal(planes.cpu().numpy(), device_layout(e4m3_bytes(P)), "planes")


def _edge_matrix(rows, k, seed):
    rng = np.random.default_rng(seed)
    X = workloads.random_matrix(rows, k, 1.0, seed)
    X[0] = 0.0                                          # zero row
    X[1] = rng.standard_normal(k) * 1e-310              # subnormal row
    X[2] = 0.0
    X[2, k // 2] = 5e-324                               # one smallest subnormal
    X[3, 3 % k] = np.nan                                # NaN row
    X[4, 1 % k] = -np.inf                               # infinite row
    X[5] = rng.standard_normal(k) * 1e300               # huge row
    X[5, 0] = 1.7e308
    X[6] = np.round(rng.standard_normal(k) * 1000)      # small integers (exact)
    X[7] = rng.standard_normal(k)
    X[7, 0] = 1e6                                       # one dominant entry
    X[8] = (rng.integers(-64, 64, size=k) + 0.5) * 2.0 ** -50   # ties after scaling
    X[8, 0] = 1.0
    X[9] = -0.0
    X[10] = rng.standard_normal(k) * 2.0 ** -1020       # normal/subnormal boundary
    return X


@pytest.mark.parametrize("side", [0, 1])
@pytest.mark.parametrize("k", [1, 63, 200])
def test_deconstruct_edge_values(side, k):
    log(f"deconstruct edge values side={side} k={k}")
    X = _edge_matrix(12, k, 10 + k)
    if side == 1:
        X = np.ascontiguousarray(X.T)
    planes, exps = gpu_deconstruct(X, side)
    e, P = _oracle_side(X, side)
    assert_int_equal(exps.cpu().numpy(), e, "exponents")
    assert_int_equal(planes.cpu().numpy(), device_layout(e4m3_bytes(P)), "planes")
    assert exps.cpu().numpy()[3] == oz.EXP_NONFINITE and exps.cpu().numpy()[4] == oz.EXP_NONFINITE


def test_deconstruct_leading_dimension():
    log("deconstruct with padded leading dimension")
    import torch
    X = workloads.random_matrix(40, 100, 1.0, 21)
    big = torch.zeros((40, 131), dtype=torch.float64, device="cuda")
    big[:, :100] = to_dev(X)
    planes, exps = oz.ozaki25_deconstruct(0, big[:, :100])
    torch.cuda.synchronize()
    e, P = _oracle_side(X, 0)
    assert_int_equal(exps.cpu().numpy(), e, "exponents")
    assert_int_equal(planes.cpu().numpy(), device_layout(e4m3_bytes(P)), "planes")


# ------------------------------------------------------------ residue products
@pytest.mark.parametrize("m,n,k,seed", [(64, 64, 64, 1), (1, 1, 1, 2), (130, 200, 129, 3),
                                        (257, 129, 700, 4), (5, 300, 64, 5), (128, 128, 1, 6)])
def test_residue_gemm_matches_oracle(m, n, k, seed):
    log(f"residue gemm m={m} n={n} k={k}")
    import torch
    A = workloads.random_matrix(m, k, 1.0, seed)
    B = workloads.random_matrix(k, n, 1.0, seed + 50)
    t = oracle.scale_bits(k)
    ZA = oracle.quantise_vectors(A, 0, oracle.exponents(A, 0, t))
    ZB = oracle.quantise_vectors(B, 1, oracle.exponents(B, 1, t))
    PA, PB = oracle.planes(ZA), oracle.planes(ZB)
    C = oz.ozaki25_residue_gemm(m, n, k, to_dev(device_layout(e4m3_bytes(PA))), to_dev(device_layout(e4m3_bytes(PB))))
    torch.cuda.synchronize()
    want = oracle.residue_gemm(oracle.residues(ZA), oracle.residues(ZB))
    assert_int_equal(C.cpu().numpy(), want, "per-modulus products")


def test_residue_gemm_full_range_residues():
    """Uniform residues over the whole int64 range of the quantised values."""
    log("residue gemm with uniform residues")
    import torch
    rng = np.random.default_rng(77)
    m, n, k = 96, 160, 320
    ZA = rng.integers(-(1 << 62), 1 << 62, size=(m, k), dtype=np.int64)
    ZB = rng.integers(-(1 << 62), 1 << 62, size=(n, k), dtype=np.int64)
    C = oz.ozaki25_residue_gemm(m, n, k, to_dev(device_layout(e4m3_bytes(oracle.planes(ZA)))),
                                to_dev(device_layout(e4m3_bytes(oracle.planes(ZB)))))
    torch.cuda.synchronize()
    want = oracle.residue_gemm(oracle.residues(ZA), oracle.residues(ZB))
    assert_int_equal(C.cpu().numpy(), want, "per-modulus products")


@pytest.mark.parametrize("k", [16384, 16512, 20000, 33000])
def test_residue_gemm_long_constant_rows(k):
    """Rows of A and columns of B that repeat one value: every term of a
    limb product has the same sign and size, so the FP32 accumulator sums
    grow linearly in k -- up to 22^2 * 16384 between reductions -- and the
    products cross one, two or three accumulation segments."""
    log(f"residue gemm, constant rows, k={k}")
    import torch
    rng = np.random.default_rng(k)
    m, n = 40, 72
    za = rng.integers(-(1 << 50), 1 << 50, size=(m, 1), dtype=np.int64)
    zb = rng.integers(-(1 << 50), 1 << 50, size=(n, 1), dtype=np.int64)
    ZA, ZB = np.repeat(za, k, axis=1), np.repeat(zb, k, axis=1)
    C = oz.ozaki25_residue_gemm(m, n, k, to_dev(device_layout(e4m3_bytes(oracle.planes(ZA)))),
                                to_dev(device_layout(e4m3_bytes(oracle.planes(ZB)))))
    torch.cuda.synchronize()
    want = oracle.residue_gemm(oracle.residues(ZA), oracle.residues(ZB))
    assert_int_equal(C.cpu().numpy(), want, "per-modulus products")


def test_residue_gemm_k_zero_writes_zeros():
    import torch
    C = torch.full((12, 3, 4), 7, dtype=torch.int32, device="cuda")
    dummy = torch.zeros(16, dtype=torch.uint8, device="cuda")
    oz.ozaki25_residue_gemm(3, 4, 0, dummy, dummy, C)
    torch.cuda.synchronize()
    assert not C.cpu().numpy().any()


# ------------------------------------------------------------ reconstruction
def _centred(x, m):
    r = x % m
    return r - m if 2 * r >= m else r


def _random_X(rng, count):
    M = oracle.product_of_moduli()
    # both ends of [-M/2, M/2), including the 544 values at each end where a
    # balanced mixed-radix form and the lift part ways
    h = M // 2
    xs = [0, 1, -1, -h, h - 1, (1 << 53) + 1, -(1 << 53) - 1, (1 << 54) + 2,
          h - 2, h - 543, h - 544, h - 545, h - 546, h - 300,
          -h + 1, -h + 543, -h + 544, -h + 545, -h + 300]
    while len(xs) < count:
        b = int(rng.integers(0, 112))
        x = int(rng.integers(0, 1 << 62)) * (1 << 50) + int(rng.integers(0, 1 << 50))
        x %= (1 << b) if b else 1
        xs.append(-x if rng.random() < 0.5 else x)
    return xs[:count]


@pytest.mark.parametrize("subtract", [False, True])
def test_reconstruct_matches_oracle(subtract):
    log(f"reconstruct subtract={subtract}")
    import torch
    rng = np.random.default_rng(31)
    m, n = 37, 300
    mods = oracle.moduli()
    Xs = _random_X(rng, m * n)
    Cres = np.array([[_centred(x, mm) for x in Xs] for mm in mods], dtype=np.int32).reshape(12, m, n)
    # exponents spanning normal, subnormal, underflow and overflow results
    ea = rng.integers(-1100, 1200, size=m).astype(np.int32)
    eb = rng.integers(-1100, 1200, size=n).astype(np.int32)
    ea[0] = oz.EXP_NONFINITE
    eb[5] = oz.EXP_NONFINITE
    ea[1], eb[1] = 1074 + 60, 0       # deep subnormal / underflow
    ea[2], eb[2] = -1000, 0           # overflow for large X
    C0 = workloads.random_matrix(m, n, 1.0, 8) if subtract else None
    Cd = to_dev(C0) if subtract else torch.empty((m, n), dtype=torch.float64, device="cuda")
    oz.ozaki25_reconstruct(to_dev(Cres), to_dev(ea), to_dev(eb), Cd, subtract=subtract)
    torch.cuda.synchronize()
    hi, lo = oracle.garner(Cres)
    want = oracle.reconstruct(hi, lo, ea, eb, C0)
    assert_bits_equal(Cd.cpu().numpy(), want, "reconstructed C")


def test_reconstruct_exact_ties():
    """X with an exact half-ulp remainder at 53 bits rounds to even."""
    log("reconstruct ties")
    import torch
    mods = oracle.moduli()
    Xs = []
    for b in range(54, 111):
        for odd in (0, 1):
            Xs.append((1 << b) + (odd << (b - 52)) + (1 << (b - 53)))
            Xs.append(-((1 << b) + (odd << (b - 52)) + (1 << (b - 53))))
    n = len(Xs)
    Cres = np.array([[_centred(x, mm) for x in Xs] for mm in mods], dtype=np.int32).reshape(12, 1, n)
    ea = np.zeros(1, np.int32)
    eb = np.zeros(n, np.int32)
    Cd = oz.ozaki25_reconstruct(to_dev(Cres), to_dev(ea), to_dev(eb))
    torch.cuda.synchronize()
    hi, lo = oracle.garner(Cres)
    assert_bits_equal(Cd.cpu().numpy(), oracle.reconstruct(hi, lo, ea, eb), "ties")
    assert_bits_equal(Cd.cpu().numpy()[0], np.array([float(x) for x in Xs]), "ties vs CPython")


def test_reconstruct_near_rounding_boundaries():
    """Values at and next to rounding boundaries at every magnitude, near
    small multiples of the high half's weight and at the range ends, unscaled
    and scaled to land on the subnormal and overflow thresholds: bit for bit
    with the oracle, and unscaled with CPython's correctly rounded int to
    float conversion."""
    log("reconstruct near rounding boundaries")
    import torch
    mods = oracle.moduli()
    M = oracle.product_of_moduli()
    Xs = workloads.boundary_values(M, _high_weight(mods))
    n = len(Xs)
    Cres = np.array([[_centred(x, mm) for x in Xs] for mm in mods], dtype=np.int32).reshape(12, 1, n)
    hi, lo = oracle.garner(Cres)
    ea = np.zeros(1, np.int32)
    eb = np.zeros(n, np.int32)
    Cd = oz.ozaki25_reconstruct(to_dev(Cres), to_dev(ea), to_dev(eb))
    torch.cuda.synchronize()
    assert_bits_equal(Cd.cpu().numpy(), oracle.reconstruct(hi, lo, ea, eb), "unscaled")
    assert_bits_equal(Cd.cpu().numpy()[0], np.array([float(x) for x in Xs]), "unscaled vs CPython")
    # sigma_i + tau_j = -e puts each result at exponent bitlen(X) - 1 + e
    for target in (-1022, -1023, -1030, -1075, 1023, 1024):
        eb = np.array([-(target - (abs(x).bit_length() - 1)) for x in Xs], dtype=np.int32)
        Cd = oz.ozaki25_reconstruct(to_dev(Cres), to_dev(ea), to_dev(eb))
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
                                          (300, 264, 200, 1.0, 8), (70, 520, 130, 2.0, 9),
                                          (300, 96, 150, 1.0, 10)])
def test_dgemm_matches_oracle(m, n, k, s, seed):
    log(f"dgemm m={m} n={n} k={k} s={s}")
    A = workloads.random_matrix(m, k, s, seed)
    B = workloads.random_matrix(k, n, s, seed + 1)
    C = gpu_dgemm(A, B)
    r = oracle.dgemm(A, B, want_planes=False)
    assert_bits_equal(C.cpu().numpy(), r.C, "C")


def test_dgemm_tiny_workload():
    log("dgemm tiny workload 64^3")
    A, B, _ = workloads.make_inputs("tiny")
    C = gpu_dgemm(A, B)
    r = oracle.dgemm(A, B)
    assert_bits_equal(C.cpu().numpy(), r.C, "C")
    planesA, expsA = gpu_deconstruct(A, 0)
    planesB, expsB = gpu_deconstruct(B, 1)
    assert_int_equal(expsA.cpu().numpy(), r.sigma, "sigma")
    assert_int_equal(expsB.cpu().numpy(), r.tau, "tau")
    assert_int_equal(planesA.cpu().numpy(), device_layout(e4m3_bytes(r.planesA)), "planes A")
    assert_int_equal(planesB.cpu().numpy(), device_layout(e4m3_bytes(r.planesB)), "planes B")


def test_dgemm_reach_workload():
    """256 x 256 x 8192: the long-k single-tile-reach case, all outputs."""
    log("dgemm reach workload 256x256x8192")
    import torch
    A, B, _ = workloads.make_inputs("reach")
    C = gpu_dgemm(A, B)
    r = oracle.dgemm(A, B)
    assert_bits_equal(C.cpu().numpy(), r.C, "C")
    planesA, expsA = gpu_deconstruct(A, 0)
    planesB, expsB = gpu_deconstruct(B, 1)
    assert_int_equal(expsA.cpu().numpy(), r.sigma, "sigma")
    assert_int_equal(expsB.cpu().numpy(), r.tau, "tau")
    assert_int_equal(planesA.cpu().numpy(), device_layout(e4m3_bytes(r.planesA)), "planes A")
    assert_int_equal(planesB.cpu().numpy(), device_layout(e4m3_bytes(r.planesB)), "planes B")
    Cres = oz.ozaki25_residue_gemm(256, 256, 8192, planesA, planesB)
    torch.cuda.synchronize()
    assert_int_equal(Cres.cpu().numpy(), r.Cres, "per-modulus products")


def test_dgemm_edge_values():
    log("dgemm with zero, subnormal, NaN, infinite and huge rows/columns")
    A = _edge_matrix(12, 40, 3)
    B = np.ascontiguousarray(_edge_matrix(12, 40, 4).T)
    C = gpu_dgemm(A, B)
    r = oracle.dgemm(A, B, want_planes=False)
    assert_bits_equal(C.cpu().numpy(), r.C, "C")
    got = C.cpu().numpy()
    # rows 3, 4 of A and columns 3, 4 of B hold a NaN / an infinity: those
    # outputs are re-issued natively (never finite); the rest are emulated
    assert np.all(np.isnan(got[3])) and np.all(np.isnan(got[:, 3]))
    assert not np.any(np.isfinite(got[4])) and not np.any(np.isfinite(got[:, 4]))
    assert not np.any(np.isnan(got[np.ix_([0, 1, 2, 5, 6, 7], [0, 1, 2, 5, 6, 7])]))


def test_dgemm_integer_inputs_are_exact():
    log("dgemm small integers")
    rng = np.random.default_rng(12)
    A = rng.integers(-1000, 1000, size=(70, 90)).astype(np.float64)
    B = rng.integers(-1000, 1000, size=(90, 80)).astype(np.float64)
    C = gpu_dgemm(A, B)
    assert np.array_equal(C.cpu().numpy(), (A.astype(np.int64) @ B.astype(np.int64)).astype(np.float64))


def test_dgemm_sub_matches_oracle():
    log("dgemm_sub 100x120x333")
    A = workloads.random_matrix(100, 333, 1.0, 40)
    B = workloads.random_matrix(333, 120, 1.0, 41)
    C0 = workloads.random_matrix(100, 120, 1.0, 42)
    C = gpu_dgemm(A, B, C0)
    r = oracle.dgemm(A, B, C_in=C0, want_planes=False)
    assert_bits_equal(C.cpu().numpy(), r.C, "C - AB")


def test_dgemm_k_zero():
    import torch
    A = torch.empty((3, 0), dtype=torch.float64, device="cuda")
    B = torch.empty((0, 4), dtype=torch.float64, device="cuda")
    C = torch.full((3, 4), 5.0, dtype=torch.float64, device="cuda")
    oz.ozaki25_dgemm(A, B, C)
    torch.cuda.synchronize()
    assert np.all(C.cpu().numpy() == 0) and not np.any(np.signbit(C.cpu().numpy()))
    C.fill_(5.0)
    oz.ozaki25_dgemm_sub(A, B, C)
    torch.cuda.synchronize()
    assert np.all(C.cpu().numpy() == 5.0)


def test_dgemm_strided_operands_and_workspace():
    log("dgemm_ex with leading dimensions and a caller workspace")
    import torch
    m, n, k = 77, 66, 150
    A = workloads.random_matrix(m, k, 1.0, 50)
    B = workloads.random_matrix(k, n, 1.0, 51)
    Ab = torch.zeros((m, k + 9), dtype=torch.float64, device="cuda")
    Bb = torch.zeros((k, n + 3), dtype=torch.float64, device="cuda")
    Cb = torch.full((m, n + 5), 3.0, dtype=torch.float64, device="cuda")
    Ab[:, :k] = to_dev(A)
    Bb[:, :n] = to_dev(B)
    ws = torch.empty(oz.ozaki25_dgemm_workspace_size(m, n, k), dtype=torch.uint8, device="cuda")
    oz.ozaki25_dgemm_ex(Ab[:, :k], Bb[:, :n], Cb[:, :n], workspace=ws)
    torch.cuda.synchronize()
    r = oracle.dgemm(A, B, want_planes=False)
    assert_bits_equal(Cb[:, :n].cpu().numpy(), r.C, "C")
    assert np.all(Cb[:, n:].cpu().numpy() == 3.0)


def test_dgemm_is_deterministic():
    log("dgemm repeat bitwise")
    import torch
    A = to_dev(workloads.random_matrix(300, 500, 1.0, 60))
    B = to_dev(workloads.random_matrix(500, 260, 1.0, 61))
    C1 = oz.ozaki25_dgemm(A, B)
    C2 = oz.ozaki25_dgemm(A, B)
    torch.cuda.synchronize()
    assert torch.equal(C1.view(torch.int64), C2.view(torch.int64))


def test_dgemm_stage_events():
    log("dgemm_ex stage events")
    import torch
    A = to_dev(workloads.random_matrix(256, 1024, 1.0, 70))
    B = to_dev(workloads.random_matrix(1024, 256, 1.0, 71))
    C = torch.empty((256, 256), dtype=torch.float64, device="cuda")
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(oz.NUM_STAGE_EVENTS)]
    for e in evs:
        e.record()
    oz.ozaki25_dgemm_ex(A, B, C, stage_events=evs)
    torch.cuda.synchronize()
    times = [evs[i].elapsed_time(evs[i + 1]) for i in range(oz.NUM_STAGE_EVENTS - 1)]
    assert all(t >= 0 for t in times) and sum(times) > 0
    assert math.isfinite(sum(times))


@pytest.mark.parametrize("m,n,k,seed", [(40, 300, 8576, 81), (24, 40, 70000, 82), (256, 256, 1024, 83)])
def test_dgemm_split_k_matches_oracle(m, n, k, seed):
    """Few output tiles: the fused path splits the k range across blocks
    (uneven stage ranges) and sums the partial products mod m."""
    log(f"dgemm split-k m={m} n={n} k={k}")
    A = workloads.random_matrix(m, k, 1.0, seed)
    B = workloads.random_matrix(k, n, 1.0, seed + 1)
    C = gpu_dgemm(A, B)
    r = oracle.dgemm(A, B, want_planes=False)
    assert_bits_equal(C.cpu().numpy(), r.C, "C")


@pytest.mark.parametrize("m,n,k,seed", [(300, 128, 700, 84), (300, 129, 700, 85), (513, 96, 2000, 86),
                                        (260, 1, 129, 87)])
def test_dgemm_narrow_tiles_match_oracle(m, n, k, seed):
    """At most 128 columns use the 512 x 128 tile (n = 129 the 256 x 256 one)."""
    log(f"dgemm narrow m={m} n={n} k={k}")
    A = workloads.random_matrix(m, k, 1.0, seed)
    B = workloads.random_matrix(k, n, 1.0, seed + 1)
    C = gpu_dgemm(A, B)
    r = oracle.dgemm(A, B, want_planes=False)
    assert_bits_equal(C.cpu().numpy(), r.C, "C")
    import torch
    planesA, _ = gpu_deconstruct(A, 0)
    planesB, _ = gpu_deconstruct(B, 1)
    Cres = oz.ozaki25_residue_gemm(m, n, k, planesA, planesB)
    torch.cuda.synchronize()
    assert_int_equal(Cres.cpu().numpy(), r.Cres, "per-modulus products")
