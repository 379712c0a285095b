"""ozaki25_dgemm_noalloc (the entry point for callers that cannot allocate:
its workspace is the library's static per-GPU array) against
ozaki25_dgemm_ex with a caller workspace, bit for bit, through the C ABI.

Two calls in a row share the array, the second with a smaller input, so
anything the first call left behind that the second depended on would
show; one product splits its k range (per-split partials in the array).
The published and the all-byte set, C = AB and C -= AB; the first product
is also held to the oracle."""
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


def _ex(A, B, C0, subtract, set):
    import torch
    m, k = A.shape
    n = B.shape[1]
    ws = torch.empty(oz.ozaki25_dgemm_workspace_size(m, n, k, set), dtype=torch.uint8, device="cuda")
    C = to_dev(C0) if subtract else torch.empty((m, n), dtype=torch.float64, device="cuda")
    oz.ozaki25_dgemm_ex(to_dev(A), to_dev(B), C, subtract=subtract, workspace=ws, set=set)
    torch.cuda.synchronize()
    return C.cpu().numpy()


def _noalloc(A, B, C0, subtract, set):
    import torch
    m, k = A.shape
    n = B.shape[1]
    assert oz.ozaki25_dgemm_workspace_size(m, n, k, set) <= oz.NOALLOC_SCRATCH_BYTES
    C = to_dev(C0) if subtract else torch.full((m, n), 7.0, dtype=torch.float64, device="cuda")
    oz.ozaki25_dgemm_noalloc(to_dev(A), to_dev(B), C, subtract=subtract, set=set)
    torch.cuda.synchronize()
    return C.cpu().numpy()


@pytest.mark.parametrize("set", [oz.S12, oz.A15])
@pytest.mark.parametrize("subtract", [False, True])
def test_noalloc_matches_dgemm_ex_twice(set, subtract):
    shapes = [(1000, 1024, 1000), (130, 257, 300)]
    for call, (m, n, k) in enumerate(shapes):
        log(f"noalloc set={set} subtract={subtract} call {call}: m={m} n={n} k={k}")
        A = workloads.random_matrix(m, k, 1.0, 300 + call)
        B = workloads.random_matrix(k, n, 1.0, 310 + call)
        C0 = workloads.random_matrix(m, n, 1.0, 320 + call) if subtract else None
        got = _noalloc(A, B, C0, subtract, set)
        assert_bits_equal(got, _ex(A, B, C0, subtract, set), f"call {call}: noalloc vs dgemm_ex")
        if call == 1:
            want = oracle.dgemm(A, B, C_in=C0, set=set, want_planes=False).C
            assert_bits_equal(got, want, f"call {call}: noalloc vs oracle")


def test_noalloc_split_k_then_smaller():
    """256 x 256 x 2048 splits the k range of its few tiles (partials in the
    array), then a smaller product without split."""
    for call, (m, n, k) in enumerate([(256, 256, 2048), (64, 64, 64)]):
        log(f"noalloc split-k sequence call {call}: m={m} n={n} k={k}")
        A = workloads.random_matrix(m, k, 0.5, 400 + call)
        B = workloads.random_matrix(k, n, 0.5, 410 + call)
        got = _noalloc(A, B, None, False, oz.S12)
        assert_bits_equal(got, _ex(A, B, None, False, oz.S12), f"call {call}: noalloc vs dgemm_ex")


@pytest.mark.parametrize("set", [oz.S12, oz.A15])
def test_noalloc_tall_skinny_then_smaller(set):
    """Tall and skinny products (storage mode F for A: B's planes and the
    products in the array, A converted inside the product kernel), the
    second one smaller."""
    for call, (m, n, k) in enumerate([(2048, 100, 700), (1024, 64, 130)]):
        log(f"noalloc tall/skinny set={set} call {call}: m={m} n={n} k={k}")
        A = workloads.random_matrix(m, k, 1.0, 500 + call)
        B = workloads.random_matrix(k, n, 1.0, 510 + call)
        got = _noalloc(A, B, None, False, set)
        assert_bits_equal(got, _ex(A, B, None, False, set), f"call {call}: noalloc vs dgemm_ex")
        if call == 1:
            want = oracle.dgemm(A, B, set=set, want_planes=False).C
            assert_bits_equal(got, want, f"call {call}: noalloc vs oracle")


def test_noalloc_refuses_beyond_its_array():
    import torch
    m = n = k = 2048
    A = torch.zeros((m, k), dtype=torch.float64, device="cuda")
    B = torch.zeros((k, n), dtype=torch.float64, device="cuda")
    C = torch.full((m, n), 3.0, dtype=torch.float64, device="cuda")
    with pytest.raises(oz.Ozaki25Error) as e:
        oz.ozaki25_dgemm_noalloc(A, B, C)
    assert e.value.status == oz.ERR_WORKSPACE
    torch.cuda.synchronize()
    assert bool((C == 3.0).all())
