"""Parity at the full workload sizes, through the entry points the benchmark
times (ozaki25_dgemm_ex with a caller workspace) and the stage API.

Per workload and modulus set:
 * every exponent of A's rows and B's columns, bit for bit;
 * every byte of both operands' stored planes (padding included), against the
   oracle's quantiser, residues and limb split, streamed in slabs of 1024
   vectors (tests/plane_check.py);
 * the per-modulus products C^(i) (int32, stage API) and the final C of
   ozaki25_dgemm_ex on a seeded sample of 256 rows x 256 columns (all columns
   when n < 256) that always includes the first two and last two rows and
   columns, i.e. the ragged tiles, bit for bit."""
import numpy as np
import pytest

import oracle
import paper_2609_09095_amd as oz
import workloads
from gpu_util import assert_bits_equal, assert_int_equal, log, require_gpu, sample_indices
from plane_check import compare_planes_full

pytestmark = pytest.mark.gpu

NSAMPLE = 256


@pytest.fixture(scope="module", autouse=True)
def gpu():
    require_gpu()


def _run(name, set=oz.S12):
    """set: the library's modulus set (the oracle numbers them alike)."""
    import torch
    w = workloads.WORKLOADS[name]
    log(f"[large] {name} set={set}: generating m={w.m} n={w.n} k={w.k}")
    A, B, C0 = workloads.make_inputs(w)
    rows = sample_indices(w.m, NSAMPLE, 11)
    cols = sample_indices(w.n, NSAMPLE, 12)
    Ad = torch.from_numpy(A).cuda()
    Bd = torch.from_numpy(B).cuda()
    Cd = torch.from_numpy(C0).cuda() if C0 is not None else torch.empty((w.m, w.n), dtype=torch.float64, device="cuda")
    ws = torch.empty(oz.ozaki25_dgemm_workspace_size(w.m, w.n, w.k, set), dtype=torch.uint8,
                     device="cuda")
    log(f"[large] {name}: ozaki25_dgemm_ex")
    oz.ozaki25_dgemm_ex(Ad, Bd, Cd, subtract=w.subtract, workspace=ws, set=set)
    torch.cuda.synchronize()
    ri = torch.from_numpy(rows).cuda()
    ci = torch.from_numpy(cols).cuda()
    C_s = Cd.index_select(0, ri).index_select(1, ci).cpu().numpy()
    del ws, Cd
    torch.cuda.empty_cache()

    log(f"[large] {name}: stage API (exponents, planes, products)")
    planesA, expsA = oz.ozaki25_deconstruct(0, Ad, set=set)
    planesB, expsB = oz.ozaki25_deconstruct(1, Bd, set=set)
    torch.cuda.synchronize()
    del Ad, Bd
    Cres = oz.ozaki25_residue_gemm(w.m, w.n, w.k, planesA, planesB, set=set)
    torch.cuda.synchronize()
    Cres_s = Cres.index_select(1, ri).index_select(2, ci).cpu().numpy()
    del Cres
    torch.cuda.empty_cache()

    t = oracle.scale_bits(w.k, set)
    sigma = oracle.exponents(A, 0, t)
    tau = oracle.exponents(B, 1, t)
    assert_int_equal(expsA.cpu().numpy(), sigma, "sigma (all rows)")
    assert_int_equal(expsB.cpu().numpy(), tau, "tau (all columns)")
    compare_planes_full(planesA, A, 0, sigma, set, f"{name} planes of A")
    compare_planes_full(planesB, B, 1, tau, set, f"{name} planes of B")
    del planesA, planesB
    torch.cuda.empty_cache()

    log(f"[large] {name}: oracle on {len(rows)} x {len(cols)} outputs")
    r = oracle.dgemm(A, B, C_in=C0, rows=rows, cols=cols, set=set, want_planes=False)
    assert_int_equal(Cres_s, r.Cres, "per-modulus products (sampled)")
    assert_bits_equal(C_s, r.C, "C (sampled)")
    log(f"[large] {name}: ok")


def test_square_8192():
    _run("square")


def test_ragged_8191_8209_7937():
    _run("ragged")


def test_hpl_trailing_update_32768_1024():
    _run("hpl")


def test_block_krylov_262144_128_4096():
    _run("krylov")


def test_long_k_single_output():
    """k far beyond the workloads (1024 K stages), one output row/column."""
    import torch
    A = workloads.random_matrix(3, 131072, 1.0, 91)
    B = workloads.random_matrix(131072, 2, 1.0, 92)
    C = oz.ozaki25_dgemm(torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda())
    torch.cuda.synchronize()
    assert_bits_equal(C.cpu().numpy(), oracle.dgemm(A, B, want_planes=False).C, "C")


def test_square_8192_all_byte_set():
    _run("square", set=oz.A15)


def test_ragged_8191_8209_7937_all_byte_set():
    _run("ragged", set=oz.A15)


def test_hpl_trailing_update_32768_1024_all_byte_set():
    _run("hpl", set=oz.A15)


def test_krylov_262144_128_4096_all_byte_set():
    _run("krylov", set=oz.A15)
