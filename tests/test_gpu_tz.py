"""Parity of the truncating quantiser (Ozaki-II-TZ) with the oracle, for both
modulus sets: exponents and planes bit for bit, the FP64 output to 0 ulp."""
import numpy as np
import pytest

import oracle
import paper_2609_09095_amd as oz
import workloads
from gpu_util import (device_layout, assert_bits_equal, assert_int_equal, e4m3_bytes, int8_bytes, log, require_gpu,
                      to_dev)

pytestmark = pytest.mark.gpu
SETS = [(oz.S12, 0, e4m3_bytes), (oz.A15, 1, int8_bytes)]


@pytest.fixture(scope="module", autouse=True)
def gpu():
    require_gpu()


@pytest.mark.parametrize("dset,oset,enc", SETS)
@pytest.mark.parametrize("side", [0, 1])
@pytest.mark.parametrize("shape,s,seed", [((64, 64), 0.5, 1), ((130, 129), 2.0, 3), ((9, 8192), 1.0, 6)])
def test_deconstruct_tz_matches_oracle(dset, oset, enc, side, shape, s, seed):
    import torch
    X = workloads.random_matrix(shape[0], shape[1], s, seed)
    if side == 1:
        X = np.ascontiguousarray(X.T)
    log(f"[TZ] deconstruct set={dset} side={side} shape={X.shape}")
    planes, exps = oz.ozaki25_deconstruct(side, to_dev(X), set=dset, quantiser=oz.TZ)
    torch.cuda.synchronize()
    k = X.shape[1] if side == 0 else X.shape[0]
    e = oracle.exponents(X, side, oracle.scale_bits(k, oset))
    Z = oracle.quantise_vectors(X, side, e, oracle.TZ)
    assert_int_equal(exps.cpu().numpy(), e, "exponents")
    assert_int_equal(planes.cpu().numpy(), device_layout(enc(oracle.planes(Z, set=oset))), "planes")


@pytest.mark.parametrize("dset,oset,enc", SETS)
@pytest.mark.parametrize("m,n,k,s,seed,subtract", [(64, 64, 64, 0.5, 1, False), (3, 5, 7, 1.0, 3, False),
                                                   (130, 129, 65, 2.0, 4, True), (200, 190, 1000, 4.0, 7, False),
                                                   (70, 260, 8192, 1.0, 8, True)])
def test_dgemm_tz_matches_oracle(dset, oset, enc, m, n, k, s, seed, subtract):
    import torch
    log(f"[TZ] dgemm set={dset} m={m} n={n} k={k} subtract={subtract}")
    A = workloads.random_matrix(m, k, s, seed)
    B = workloads.random_matrix(k, n, s, seed + 1)
    C0 = workloads.random_matrix(m, n, 1.0, seed + 2) if subtract else None
    Cd = to_dev(C0) if subtract else torch.empty((m, n), dtype=torch.float64, device="cuda")
    oz.ozaki25_dgemm_ex(to_dev(A), to_dev(B), Cd, subtract=subtract, set=dset, quantiser=oz.TZ)
    torch.cuda.synchronize()
    r = oracle.dgemm(A, B, C_in=C0, want_planes=False, set=oset, quant=oracle.TZ)
    assert_bits_equal(Cd.cpu().numpy(), r.C, "C")
    # the two quantisers do give different results on these inputs
    if k > 7:
        rn = oracle.dgemm(A, B, C_in=C0, want_planes=False, set=oset)
        assert not np.array_equal(rn.C, r.C)
