"""Alg. 1's last step on the GPU: outputs whose row of A or column of B holds
a NaN or an infinity are re-issued on the native FP64 path (the index-order
dot product, rounded products then sums, no FMA) by the GEMM entry points
that see A and B, and compared with the oracle's re-issue bit for bit (any
NaN matches any NaN; infinities by sign).  The stage API's reconstruction
and the stored-planes entry point, which do not see A and B, keep NaN
there.  Cases: Inf * 0, Inf - Inf, a finite overflow that only the index
order turns into NaN, k spanning several K stages, both sets, C = AB and
C -= AB, and the allocation-free entry point."""
import numpy as np
import pytest

import oracle
import paper_2609_09095_amd as oz
import workloads
from gpu_util import assert_bits_equal, log, require_gpu, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    require_gpu()


def _inputs(m, n, k, seed):
    A = workloads.random_matrix(m, k, 1.0, seed)
    B = workloads.random_matrix(k, n, 1.0, seed + 1)
    A[1, 3] = np.nan
    A[2, 0] = np.inf
    A[3, 2], A[3, k - 1] = np.inf, -np.inf   # with B[2, 0] = B[k-1, 0] = 1: Inf - Inf
    A[4, :2] = 1e308
    A[4, k - 1] = -np.inf
    B[k - 2, 2] = np.inf
    B[0, 4] = 0.0
    B[:2, 5] = 1.0
    B[k - 1, 5] = 2.0
    B[5, n - 1] = np.nan
    B[2, 0] = B[k - 1, 0] = 1.0
    return A, B


def _assert_inf_signs(got, want, what):
    gi, wi = np.isinf(got), np.isinf(want)
    assert np.array_equal(gi, wi), f"{what}: infinity pattern differs"
    assert np.array_equal(np.signbit(got[gi]), np.signbit(want[wi])), f"{what}: infinity signs differ"


@pytest.mark.parametrize("set", [oz.S12, oz.A15])
@pytest.mark.parametrize("m,n,k,seed", [(9, 8, 8, 1), (300, 270, 1000, 2), (40, 520, 257, 3)])
def test_dgemm_reissues_nonfinite_rows_and_columns(set, m, n, k, seed):
    log(f"native re-issue set={set} m={m} n={n} k={k}")
    A, B = _inputs(m, n, k, seed)
    got = oz.ozaki25_dgemm(to_dev(A), to_dev(B), set=set).cpu().numpy()
    want = oracle.dgemm(A, B, set=set, want_planes=False).C
    assert_bits_equal(got, want, "C")
    _assert_inf_signs(got, want, "C")
    assert np.isnan(got[4, 5]) and np.isnan(got[2, 4]) and np.isnan(got[3, 0])
    assert np.isinf(got[2, 0])
    flagged = np.zeros((m, n), bool)
    flagged[[1, 2, 3, 4]] = True
    flagged[:, [2, n - 1]] = True
    assert not np.any(np.isfinite(got[flagged])) and np.all(np.isfinite(got[~flagged]))


@pytest.mark.parametrize("set", [oz.S12, oz.A15])
def test_dgemm_sub_and_noalloc_reissue(set):
    import torch
    m, n, k = 130, 70, 300
    A, B = _inputs(m, n, k, 7)
    C0 = workloads.random_matrix(m, n, 1.0, 9)
    C0[0, 2] = np.inf
    want = oracle.dgemm(A, B, C_in=C0, set=set, want_planes=False).C
    C = to_dev(C0)
    oz.ozaki25_dgemm_sub(to_dev(A), to_dev(B), C, set=set)
    got = C.cpu().numpy()
    assert_bits_equal(got, want, "C -= AB")
    _assert_inf_signs(got, want, "C -= AB")
    C = torch.empty((m, n), dtype=torch.float64, device="cuda")
    oz.ozaki25_dgemm_noalloc(to_dev(A), to_dev(B), C, set=set)
    want = oracle.dgemm(A, B, set=set, want_planes=False).C
    got = C.cpu().numpy()
    assert_bits_equal(got, want, "noalloc C")
    _assert_inf_signs(got, want, "noalloc C")


@pytest.mark.parametrize("set", [oz.S12, oz.A15])
def test_stage_api_and_stored_planes_keep_nan(set):
    import torch
    m, n, k = 9, 8, 8
    A, B = _inputs(m, n, k, 11)
    want = oracle.dgemm(A, B, set=set, want_planes=False, fallback=False).C
    pa, ea = oz.ozaki25_deconstruct(0, to_dev(A), set=set)
    pb, eb = oz.ozaki25_deconstruct(1, to_dev(B), set=set)
    Cres = oz.ozaki25_residue_gemm(m, n, k, pa, pb, set=set)
    got = oz.ozaki25_reconstruct(Cres, ea, eb, set=set).cpu().numpy()
    assert_bits_equal(got, want, "stage-wise C")
    got = oz.ozaki25_dgemm_planes(k, pa, ea, pb, eb, set=set).cpu().numpy()
    torch.cuda.synchronize()
    assert_bits_equal(got, want, "stored-planes C")
    assert np.all(np.isnan(got[[1, 2, 3, 4]])) and np.all(np.isnan(got[:, [2, n - 1]]))
