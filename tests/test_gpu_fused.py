"""Storage mode F for A (at most 128 columns, at least 1024 rows, both
modulus sets): ozaki25_dgemm_ex converts A inside the product kernel instead
of storing its planes.  Every output is compared with the oracle bit for bit
(any NaN matching any NaN): ragged rows, columns and k, one column, k past
the segments after which the sums are reduced (65536 k for the all-byte
set's int32 sums, 16384 k for the published set's square digit sums), C -=
AB, the truncating quantiser, rows and columns with non-finite values
(native re-issue), a wide exponent range, and zero, subnormal, huge and
tie rows."""
import numpy as np
import pytest

import oracle
import paper_2609_09095_amd as oz
import workloads
from gpu_util import assert_bits_equal, log, require_gpu, sample_indices, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    require_gpu()


SETS = [pytest.param(oz.S12, id="S12"), pytest.param(oz.A15, id="A15")]


def _run(A, B, set, C0=None, quant=oz.RN):
    import torch
    m, k = A.shape
    n = B.shape[1]
    ws = torch.empty(oz.ozaki25_dgemm_workspace_size(m, n, k, set), dtype=torch.uint8, device="cuda")
    C = to_dev(C0) if C0 is not None else torch.empty((m, n), dtype=torch.float64, device="cuda")
    oz.ozaki25_dgemm_ex(to_dev(A), to_dev(B), C, subtract=C0 is not None, workspace=ws, set=set,
                        quantiser=quant)
    torch.cuda.synchronize()
    return C.cpu().numpy()


@pytest.mark.parametrize("set", SETS)
@pytest.mark.parametrize("m,n,k,s,seed", [(1024, 128, 64, 1.0, 1), (1300, 70, 1000, 1.0, 2),
                                          (2049, 1, 257, 2.0, 3), (4096, 128, 4096, 1.0, 4),
                                          (1500, 100, 130, 4.0, 5), (1030, 128, 8, 0.5, 6)])
def test_fused_matches_oracle(set, m, n, k, s, seed):
    log(f"fused set={set} m={m} n={n} k={k} s={s}")
    A = workloads.random_matrix(m, k, s, seed)
    B = workloads.random_matrix(k, n, s, seed + 100)
    assert_bits_equal(_run(A, B, set), oracle.dgemm(A, B, set=set, want_planes=False).C, "C")


@pytest.mark.parametrize("set", SETS)
def test_fused_k_sweep(set):
    """k around the points where the all-byte kernel's main loop (both
    look-ahead stages whole) hands over to its guarded steps, and where the
    last stage turns partial or lies past k: each multiple of 64 from 256
    to 576 and its two neighbours."""
    m, n = 1024, 3
    ks = sorted({kk + d for kk in range(256, 577, 64) for d in (-1, 0, 1)})
    for i, k in enumerate(ks):
        A = workloads.random_matrix(m, k, 1.0, 300 + i)
        B = workloads.random_matrix(k, n, 1.0, 400 + i)
        log(f"fused set={set} k={k}")
        assert_bits_equal(_run(A, B, set), oracle.dgemm(A, B, set=set, want_planes=False).C, f"C (k={k})")


@pytest.mark.parametrize("set", SETS)
def test_fused_subtract_tz_and_nonfinite(set):
    m, n, k = 1100, 90, 300
    A = workloads.random_matrix(m, k, 1.0, 11)
    B = workloads.random_matrix(k, n, 1.0, 12)
    C0 = workloads.random_matrix(m, n, 1.0, 13)
    A[5, 7] = np.nan
    A[1090, 0] = -np.inf
    B[3, 40] = np.inf
    log(f"fused set={set} C -= AB with non-finite rows and columns")
    assert_bits_equal(_run(A, B, set, C0), oracle.dgemm(A, B, C_in=C0, set=set, want_planes=False).C,
                      "C -= AB")
    log(f"fused set={set} truncating quantiser")
    A[5, 7], A[1090, 0], B[3, 40] = 1.0, 2.0, 3.0
    assert_bits_equal(_run(A, B, set, quant=oz.TZ),
                      oracle.dgemm(A, B, set=set, want_planes=False, quant=oracle.TZ).C, "C (TZ)")


@pytest.mark.parametrize("set", SETS)
def test_fused_long_k_segments(set):
    """k = 70000 crosses the segments after which the sums are reduced mod
    m (65536 k for the all-byte set, 16384 k for the published set's square
    digit sums)."""
    m, n, k = 1024, 3, 70000
    A = workloads.random_matrix(m, k, 1.0, 21)
    B = workloads.random_matrix(k, n, 1.0, 22)
    rows = sample_indices(m, 64, 23)
    log(f"fused set={set} k={k}")
    got = _run(A, B, set)[rows]
    want = oracle.dgemm(A, B, rows=rows, set=set, want_planes=False).C
    assert_bits_equal(got, want, "C (sampled rows)")


@pytest.mark.parametrize("set", SETS)
@pytest.mark.parametrize("quant", [pytest.param(oz.RN, id="RN"), pytest.param(oz.TZ, id="TZ")])
def test_fused_edge_rows(set, quant):
    """Zero, subnormal, huge, tie, boundary and non-finite rows of A and
    columns of B, converted inside the product kernel with their own row
    scales (k = 600: whole stages, then a partial one)."""
    m, n, k = 1040, 24, 600
    A = workloads.edge_rows(workloads.random_matrix(m, k, 1.0, 61), 62)
    B = np.ascontiguousarray(workloads.edge_rows(workloads.random_matrix(n, k, 1.0, 63), 64).T)
    log(f"fused set={set} edge rows and columns, quantiser {quant}")
    want = oracle.dgemm(A, B, set=set, want_planes=False, quant=oracle.TZ if quant == oz.TZ else oracle.RN).C
    got = _run(A, B, set, quant=quant)
    assert_bits_equal(got, want, "C")
    # row 3 of A and column 3 of B hold a NaN: re-issued natively
    assert np.all(np.isnan(got[3])) and np.all(np.isnan(got[:, 3]))


def test_fused_published_constant_vectors():
    """Published set: constant rows of A and columns of B, so that every
    term of a sum has the same residue product and the FP32 sums grow
    without cancellation between reductions (their largest magnitudes for
    those residues), beside random rows and columns."""
    m, n, k = 1024, 8, 2048
    A = workloads.random_matrix(m, k, 1.0, 32)
    B = workloads.random_matrix(k, n, 1.0, 33)
    A[:16, :] = np.ldexp(1.0, -3) * (1 - 2.0 ** -40)
    A[16:32, :] = -1.0
    A[32:48, :] = 3.0 * (1 + 2.0 ** -30)
    B[:, :2] = 7.0 * (1 - 2.0 ** -45)
    B[:, 2] = -3.0
    log("fused S12 constant rows and columns")
    assert_bits_equal(_run(A, B, oz.S12), oracle.dgemm(A, B, set=0, want_planes=False).C, "C")
