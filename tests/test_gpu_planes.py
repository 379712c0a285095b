"""Storage mode P: ozaki25_dgemm_planes on planes kept from ozaki25_deconstruct
gives ozaki25_dgemm_ex's result bit for bit (both sets, both quantisers), and
one stored A serves several B."""
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


@pytest.mark.parametrize("dset,oset", [(oz.S12, 0), (oz.A15, 1)])
@pytest.mark.parametrize("quant", [oz.RN, oz.TZ])
@pytest.mark.parametrize("m,n,k,seed", [(130, 129, 65, 1), (257, 300, 1000, 2), (64, 70, 8192, 3)])
def test_planes_gemm_matches_dgemm_ex_and_oracle(dset, oset, quant, m, n, k, seed):
    import torch
    log(f"[mode P] set={dset} quant={quant} m={m} n={n} k={k}")
    A = to_dev(workloads.random_matrix(m, k, 1.0, seed))
    planesA, expsA = oz.ozaki25_deconstruct(0, A, set=dset, quantiser=quant)
    Bs = [workloads.random_matrix(k, n, 1.0, seed + 10 * i) for i in (1, 2)]
    for i, Bh in enumerate(Bs):
        B = to_dev(Bh)
        planesB, expsB = oz.ozaki25_deconstruct(1, B, set=dset, quantiser=quant)
        C = oz.ozaki25_dgemm_planes(k, planesA, expsA, planesB, expsB, set=dset)
        ref = torch.empty((m, n), dtype=torch.float64, device="cuda")
        oz.ozaki25_dgemm_ex(A, B, ref, set=dset, quantiser=quant)
        # subtract form with a caller workspace
        C0 = workloads.random_matrix(m, n, 1.0, seed + 5)
        Cs = to_dev(C0)
        ws = torch.empty(oz.ozaki25_dgemm_planes_workspace_size(m, n, k, dset), dtype=torch.uint8, device="cuda")
        oz.ozaki25_dgemm_planes(k, planesA, expsA, planesB, expsB, Cs, subtract=True, workspace=ws, set=dset)
        torch.cuda.synchronize()
        assert torch.equal(C.view(torch.int64), ref.view(torch.int64)), f"B #{i}"
        if i == 0:
            r = oracle.dgemm(A.cpu().numpy(), Bh, C_in=C0, want_planes=False, set=oset, quant=quant)
            assert_bits_equal(Cs.cpu().numpy(), r.C, "C - AB from planes")


def test_planes_gemm_k_zero():
    import torch
    e = torch.zeros(3, dtype=torch.int32, device="cuda")
    p = torch.zeros(16, dtype=torch.uint8, device="cuda")
    C = torch.full((3, 3), 5.0, dtype=torch.float64, device="cuda")
    oz.ozaki25_dgemm_planes(0, p, e, p, e, C)
    torch.cuda.synchronize()
    assert np.all(C.cpu().numpy() == 0)
