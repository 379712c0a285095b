"""Accurate mode (Sec. 2, Eq. (alpha)) on the GPU against the oracle.

The exponents (sigma of every row of A, tau of every column of B) must
equal the oracle's exactly -- they come from the magnitude digits, the int8
bound product (split-k included), its per-output totals and the row and
column minima -- and every output of ozaki25_dgemm_accurate must equal the
oracle's accurate-mode result bit for bit (any NaN matching any NaN): both
modulus sets, ragged shapes, wide exponent ranges, saturating inputs that
put the bound at its edge, zero and non-finite rows and columns, C -= AB,
the truncating quantiser and the all-byte set's fused path for A.  At the
8192^3 square size the exponents are compared in full and sampled outputs
against the oracle."""
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


def _exps(A, B, set):
    import torch
    ea, eb = oz.ozaki25_accurate_exponents(to_dev(A), to_dev(B), set=set)
    torch.cuda.synchronize()
    return ea.cpu().numpy(), eb.cpu().numpy()


def _dgemm(A, B, set, C0=None, quant=oz.RN, events=False):
    import torch
    m, k = A.shape
    n = B.shape[1]
    ws = torch.empty(oz.ozaki25_dgemm_accurate_workspace_size(m, n, k, set), dtype=torch.uint8,
                     device="cuda")
    C = to_dev(C0) if C0 is not None else torch.full((m, n), 7.0, dtype=torch.float64, device="cuda")
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(oz.NUM_STAGE_EVENTS)] if events else None
    for e in ev or []:
        e.record()  # creates the event; the library records it again in place
    oz.ozaki25_dgemm_accurate(to_dev(A), to_dev(B), C, subtract=C0 is not None, workspace=ws,
                              stage_events=ev, set=set, quantiser=quant)
    torch.cuda.synchronize()
    if ev:
        log("stages ms: " + " ".join(f"{ev[i].elapsed_time(ev[i + 1]):.3f}" for i in range(4)))
    return C.cpu().numpy()


def _check_exps(A, B, set, what):
    ga, gb = _exps(A, B, set)
    sa, tb, _, _, _ = oracle.accurate_exponents(A, B, set)
    for got, want, side in ((ga, sa, "sigma"), (gb, tb, "tau")):
        bad = np.nonzero(got != want)[0]
        assert bad.size == 0, (f"{what}: {bad.size} {side} differ; first at {bad[0]}: "
                               f"{got[bad[0]]} vs {want[bad[0]]}")
    return sa, tb


# (m, n, k, s, seed): one tile; ragged multi-tile; n > 128 (256 x 256
# tiles); long k with few tiles (split bound product); one element
SHAPES = [(64, 64, 64, 0.5, 1), (300, 257, 129, 4.0, 2), (513, 77, 1000, 2.0, 3),
          (64, 48, 8192, 1.0, 4), (700, 300, 2000, 4.0, 5), (1, 1, 1, 1.0, 6), (130, 3, 70000, 1.0, 7)]


@pytest.mark.parametrize("set", [0, 1])
@pytest.mark.parametrize("m,n,k,s,seed", SHAPES)
def test_accurate_exponents_match_oracle(set, m, n, k, s, seed):
    log(f"accurate exponents set={set} m={m} n={n} k={k} s={s}")
    A = workloads.random_matrix(m, k, s, seed)
    B = workloads.random_matrix(k, n, s, seed + 100)
    _check_exps(A, B, set, f"{m}x{n}x{k}")


@pytest.mark.parametrize("set", [0, 1])
def test_accurate_exponents_saturating_zero_and_nonfinite(set):
    m, n, k = 260, 140, 4099
    top = 1 - 2.0 ** -53
    A = np.full((m, k), top) * np.exp2(np.arange(m) % 7 - 3.0)[:, None]
    B = np.full((k, n), -top) * np.exp2(np.arange(n) % 5 - 2.0)[None, :]
    A[::3] = workloads.random_matrix((m + 2) // 3, k, 2.0, 31)
    A[5] = 0.0
    A[17, 100] = np.nan
    B[:, 9] = 0.0
    B[2000, 33] = -np.inf
    B[0, 139] = 5e-324
    log(f"accurate exponents, saturating rows, zero and non-finite vectors, set={set}")
    sa, tb = _check_exps(A, B, set, "saturating")
    assert sa[17] == oz.EXP_NONFINITE and tb[33] == oz.EXP_NONFINITE


@pytest.mark.parametrize("set", [0, 1])
@pytest.mark.parametrize("m,n,k,s,seed", [(200, 150, 300, 2.0, 11), (257, 129, 1000, 4.0, 12),
                                          (33, 500, 8192, 1.0, 13)])
def test_accurate_dgemm_matches_oracle(set, m, n, k, s, seed):
    log(f"accurate dgemm set={set} m={m} n={n} k={k} s={s}")
    A = workloads.random_matrix(m, k, s, seed)
    B = workloads.random_matrix(k, n, s, seed + 100)
    want = oracle.dgemm(A, B, set=set, accurate=True, want_planes=False).C
    assert_bits_equal(_dgemm(A, B, set, events=True), want, "C")


@pytest.mark.parametrize("set", [0, 1])
def test_accurate_subtract_tz_and_nonfinite(set):
    m, n, k = 300, 200, 700
    A = workloads.random_matrix(m, k, 3.0, 21)
    B = workloads.random_matrix(k, n, 3.0, 22)
    C0 = workloads.random_matrix(m, n, 1.0, 23)
    A[7, 3] = np.inf
    B[5, 150] = np.nan
    A[40] = 0.0
    log(f"accurate C -= AB with non-finite and zero vectors, set={set}")
    want = oracle.dgemm(A, B, C_in=C0, set=set, accurate=True, want_planes=False).C
    assert_bits_equal(_dgemm(A, B, set, C0=C0), want, "C -= AB")
    log(f"accurate, truncating quantiser, set={set}")
    want = oracle.dgemm(A, B, set=set, accurate=True, want_planes=False, quant=oracle.TZ).C
    assert_bits_equal(_dgemm(A, B, set, quant=oz.TZ), want, "C (TZ)")


@pytest.mark.parametrize("set", [0, 1])
@pytest.mark.parametrize("m,n,k,s,seed", [(1100, 90, 300, 3.0, 41), (2049, 128, 4096, 1.0, 42)])
def test_accurate_fused_path(set, m, n, k, s, seed):
    """At most 128 columns and at least 1024 rows: A is converted inside the
    product kernel (storage mode F), here at the accurate mode's shifts."""
    log(f"accurate fused set={set} m={m} n={n} k={k}")
    A = workloads.random_matrix(m, k, s, seed)
    B = workloads.random_matrix(k, n, s, seed + 100)
    A[3, 3] = -np.inf
    want = oracle.dgemm(A, B, set=set, accurate=True, want_planes=False).C
    assert_bits_equal(_dgemm(A, B, set), want, "C")


@pytest.mark.parametrize("set", [0, 1])
def test_accurate_fused_subtract_tz(set):
    """Storage mode F at the accurate mode's shifts with C -= AB, the
    truncating quantiser, a non-finite column and a zero row."""
    m, n, k = 1200, 64, 520
    A = workloads.random_matrix(m, k, 2.0, 51)
    B = workloads.random_matrix(k, n, 2.0, 52)
    C0 = workloads.random_matrix(m, n, 1.0, 53)
    B[9, 33] = np.nan
    A[77] = 0.0
    log(f"accurate fused C -= AB, set={set}")
    want = oracle.dgemm(A, B, C_in=C0, set=set, accurate=True, want_planes=False).C
    assert_bits_equal(_dgemm(A, B, set, C0=C0), want, "C -= AB")
    log(f"accurate fused, truncating quantiser, set={set}")
    want = oracle.dgemm(A, B, set=set, accurate=True, want_planes=False, quant=oracle.TZ).C
    assert_bits_equal(_dgemm(A, B, set, quant=oz.TZ), want, "C (TZ)")


@pytest.mark.parametrize("set", [0, 1])
def test_accurate_fused_edge_rows(set):
    """Storage mode F at the accurate mode's shifts with zero, subnormal,
    huge, tie, boundary and non-finite rows of A and columns of B."""
    m, n, k = 1040, 24, 600
    A = workloads.edge_rows(workloads.random_matrix(m, k, 1.0, 71), 72)
    B = np.ascontiguousarray(workloads.edge_rows(workloads.random_matrix(n, k, 1.0, 73), 74).T)
    log(f"accurate fused edge rows and columns, set={set}")
    want = oracle.dgemm(A, B, set=set, accurate=True, want_planes=False).C
    assert_bits_equal(_dgemm(A, B, set), want, "C")


def test_accurate_k_zero_and_errors():
    import torch
    A = torch.zeros((4, 0), dtype=torch.float64, device="cuda")
    B = torch.zeros((0, 3), dtype=torch.float64, device="cuda")
    C = oz.ozaki25_dgemm_accurate(A, B)
    torch.cuda.synchronize()
    assert C.shape == (4, 3) and not C.cpu().numpy().any()
    A = torch.ones((4, 5), dtype=torch.float64, device="cuda")
    B = torch.ones((5, 3), dtype=torch.float64, device="cuda")
    small = torch.empty(16, dtype=torch.uint8, device="cuda")
    with pytest.raises(oz.Ozaki25Error) as e:
        oz.ozaki25_dgemm_accurate(A, B, workspace=small)
    assert e.value.status == oz.ERR_WORKSPACE
    with pytest.raises(oz.Ozaki25Error) as e:
        oz.ozaki25_accurate_exponents(A, B, workspace=small)
    assert e.value.status == oz.ERR_WORKSPACE


def test_accurate_square_8192():
    """The square workload in the accurate mode: all 16384 exponents in
    full, and outputs of 256 sampled rows x 256 sampled columns."""
    A, B, _ = workloads.make_inputs("square")
    log("accurate square 8192^3: GPU exponents and product")
    ga, gb = _exps(A, B, 0)
    import torch
    Ad, Bd = to_dev(A), to_dev(B)
    C = oz.ozaki25_dgemm_accurate(Ad, Bd)
    torch.cuda.synchronize()
    log("accurate square 8192^3: oracle exponents")
    sa, tb, _, _, _ = oracle.accurate_exponents(A, B, 0)
    assert np.array_equal(ga, sa) and np.array_equal(gb, tb)
    rows, cols = sample_indices(8192, 256, 1), sample_indices(8192, 256, 2)
    log("accurate square 8192^3: oracle outputs on the sample")
    want = oracle.dgemm(A, B, rows=rows, cols=cols, accurate=True, accurate_exps=(sa, tb),
                        want_planes=False).C
    got = C[torch.from_numpy(rows).cuda()][:, torch.from_numpy(cols).cuda()].cpu().numpy()
    assert_bits_equal(got, want, "C sample")
    fast = oracle.dgemm(A, B, rows=rows, cols=cols, want_planes=False).C
    exact = A[rows].astype(np.longdouble) @ B[:, cols].astype(np.longdouble)
    err_acc = np.abs(want - exact).max()
    err_fast = np.abs(fast - exact).max()
    log(f"max |C - AB| on the sample (long double reference): accurate {float(err_acc):.3e}, "
        f"fast {float(err_fast):.3e}")
    assert err_acc <= err_fast
