"""Emulated DGEMM at shapes where the residue GEMM (compact output, whole
k) runs one block per compute unit and each block walks several output
tiles in turn, loading the next tile's first K stage while it stores the
current one: for the published set 12 moduli x (1800/256 -> 8) x
(1500/256 -> 6) = 576 tiles, for the all-byte set 15 x 8 x 6 = 720, and more
below, against 256 CUs.  Ragged and exact tile edges, C = AB
and C -= AB, both quantisers (Eq. (scale)), the accurate mode (Sec. 2,
Eq. (alpha)) and k from 2 to 16 K stages of 128 (the form serves short k
only).  The final C on a seeded sample of
rows and columns (both ends included) is compared bit for bit with the
oracle's."""
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


CASES = [
    dict(m=1800, n=1500, k=256, sub=True, tz=False, accurate=False, ns=128, seed=8100),
    dict(m=1800, n=1500, k=256, sub=False, tz=True, accurate=True, ns=128, seed=8110),
    dict(m=2048, n=2048, k=512, sub=False, tz=False, accurate=False, ns=128, seed=8120),
    dict(m=1800, n=1800, k=2048, sub=True, tz=False, accurate=False, ns=64, seed=8130),
]
SETS = [pytest.param(oz.S12, id="S12"), pytest.param(oz.A15, id="A15")]


@pytest.mark.parametrize("set", SETS)
@pytest.mark.parametrize("c", CASES, ids=lambda c: f"{c['m']}x{c['n']}x{c['k']}"
                         f"{'-acc' if c['accurate'] else ''}{'-sub' if c['sub'] else ''}")
def test_multitile(c, set):
    import torch
    m, n, k = c["m"], c["n"], c["k"]
    log(f"[multitile] set={set} {c}")
    A = workloads.random_matrix(m, k, 1.0, c["seed"])
    B = workloads.random_matrix(k, n, 1.0, c["seed"] + 1)
    C0 = workloads.random_matrix(m, n, 1.0, c["seed"] + 2) if c["sub"] else None
    rows = sample_indices(m, c["ns"], c["seed"] + 3)
    cols = sample_indices(n, c["ns"], c["seed"] + 4)
    quant = oz.TZ if c["tz"] else oz.RN
    size = oz.ozaki25_dgemm_accurate_workspace_size if c["accurate"] else oz.ozaki25_dgemm_workspace_size
    ws = torch.empty(size(m, n, k, set), dtype=torch.uint8, device="cuda")
    Cd = to_dev(C0) if C0 is not None else torch.full((m, n), 7.0, dtype=torch.float64, device="cuda")
    call = oz.ozaki25_dgemm_accurate if c["accurate"] else oz.ozaki25_dgemm_ex
    call(to_dev(A), to_dev(B), Cd, subtract=c["sub"], workspace=ws, set=set, quantiser=quant)
    torch.cuda.synchronize()
    got = Cd.cpu().numpy()[np.ix_(rows, cols)]
    want = oracle.dgemm(A, B, C_in=C0, rows=rows, cols=cols, set=set, accurate=c["accurate"],
                        want_planes=False, quant=oracle.TZ if c["tz"] else oracle.RN).C
    assert_bits_equal(got, want, "C (sampled)")


@pytest.mark.parametrize("set", SETS)
def test_stored_planes_tall_narrow(set):
    """Storage mode P at most 128 columns wide (the 512 x 128 tile shape) at
    short k: 43 tile rows x 12 or 15 moduli, again over two tiles per CU."""
    import torch
    m, n, k = 22000, 100, 256
    log(f"[multitile] mode P set={set} m={m} n={n} k={k}")
    A = workloads.random_matrix(m, k, 1.0, 8200)
    B = workloads.random_matrix(k, n, 1.0, 8201)
    planesA, expsA = oz.ozaki25_deconstruct(0, to_dev(A), set=set)
    planesB, expsB = oz.ozaki25_deconstruct(1, to_dev(B), set=set)
    C = oz.ozaki25_dgemm_planes(k, planesA, expsA, planesB, expsB, set=set)
    torch.cuda.synchronize()
    rows = sample_indices(m, 128, 8202)
    want = oracle.dgemm(A, B, rows=rows, set=set, want_planes=False).C
    assert_bits_equal(C.cpu().numpy()[rows], want, "C (sampled rows)")
