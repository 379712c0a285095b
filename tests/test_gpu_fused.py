"""Storage mode F for A (the all-byte set, at most 128 columns, at least 1024
rows): ozaki25_dgemm_ex converts A inside the product kernel instead of
storing its planes.  Every output is compared with the oracle bit for bit
(any NaN matching any NaN): ragged rows, columns and k, one column, k past
the 65536-long segments of the int32 sums, C -= AB, the truncating
quantiser, rows and columns with non-finite values (native re-issue), and
a wide exponent range."""
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


def _run(A, B, C0=None, quant=oz.RN):
    import torch
    m, k = A.shape
    n = B.shape[1]
    ws = torch.empty(oz.ozaki25_dgemm_workspace_size(m, n, k, oz.A15), dtype=torch.uint8, device="cuda")
    C = to_dev(C0) if C0 is not None else torch.empty((m, n), dtype=torch.float64, device="cuda")
    oz.ozaki25_dgemm_ex(to_dev(A), to_dev(B), C, subtract=C0 is not None, workspace=ws, set=oz.A15,
                        quantiser=quant)
    torch.cuda.synchronize()
    return C.cpu().numpy()


@pytest.mark.parametrize("m,n,k,s,seed", [(1024, 128, 64, 1.0, 1), (1300, 70, 1000, 1.0, 2),
                                          (2049, 1, 257, 2.0, 3), (4096, 128, 4096, 1.0, 4),
                                          (1500, 100, 130, 4.0, 5)])
def test_fused_matches_oracle(m, n, k, s, seed):
    log(f"fused A15 m={m} n={n} k={k} s={s}")
    A = workloads.random_matrix(m, k, s, seed)
    B = workloads.random_matrix(k, n, s, seed + 100)
    assert_bits_equal(_run(A, B), oracle.dgemm(A, B, set=1, want_planes=False).C, "C")


def test_fused_subtract_tz_and_nonfinite():
    m, n, k = 1100, 90, 300
    A = workloads.random_matrix(m, k, 1.0, 11)
    B = workloads.random_matrix(k, n, 1.0, 12)
    C0 = workloads.random_matrix(m, n, 1.0, 13)
    A[5, 7] = np.nan
    A[1090, 0] = -np.inf
    B[3, 40] = np.inf
    log("fused A15 C -= AB with non-finite rows and columns")
    assert_bits_equal(_run(A, B, C0), oracle.dgemm(A, B, C_in=C0, set=1, want_planes=False).C, "C -= AB")
    log("fused A15 truncating quantiser")
    A[5, 7], A[1090, 0], B[3, 40] = 1.0, 2.0, 3.0
    assert_bits_equal(_run(A, B, quant=oz.TZ),
                      oracle.dgemm(A, B, set=1, want_planes=False, quant=oracle.TZ).C, "C (TZ)")


def test_fused_long_k_segments():
    """k = 70000 crosses the 65536-long segment after which the int32 sums
    are reduced mod m."""
    m, n, k = 1024, 3, 70000
    A = workloads.random_matrix(m, k, 1.0, 21)
    B = workloads.random_matrix(k, n, 1.0, 22)
    rows = sample_indices(m, 64, 23)
    got = _run(A, B)[rows]
    want = oracle.dgemm(A, B, rows=rows, set=1, want_planes=False).C
    assert_bits_equal(got, want, "C (sampled rows)")
