"""ozaki25_dgemm_ex with a caller workspace enqueues kernels only (no
allocation, no memset), so a HIP graph can capture it: every replay of the
captured graph, with eager work and synchronisations between replays, gives
the eager result bit for bit (both modulus sets; the split-k path included,
and at 1800 x 1500 x 256 the published set's residue GEMM in its form with
one block per CU walking 576 tiles)."""
import numpy as np
import pytest

import paper_2609_09095_amd as oz
import workloads
from gpu_util import log, require_gpu, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    require_gpu()


@pytest.mark.parametrize("dset", [oz.S12, oz.A15])
@pytest.mark.parametrize("m,n,k", [(64, 64, 64), (300, 129, 700), (256, 256, 4096), (1800, 1500, 256)])
def test_graph_replays_match_eager(dset, m, n, k):
    import torch
    log(f"graph capture set={dset} m={m} n={n} k={k}")
    A = to_dev(workloads.random_matrix(m, k, 1.0, 7))
    B = to_dev(workloads.random_matrix(k, n, 1.0, 8))
    ws = torch.empty(oz.ozaki25_dgemm_workspace_size(m, n, k, dset), dtype=torch.uint8, device="cuda")
    ref = torch.empty((m, n), dtype=torch.float64, device="cuda")
    oz.ozaki25_dgemm_ex(A, B, ref, workspace=ws, set=dset)
    torch.cuda.synchronize()
    C = torch.empty((m, n), dtype=torch.float64, device="cuda")
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):   # warm up on the capture stream's side
        oz.ozaki25_dgemm_ex(A, B, C, workspace=ws, set=dset)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        oz.ozaki25_dgemm_ex(A, B, C, workspace=ws, set=dset)
    for rep in range(4):
        C.fill_(float("nan"))
        ws.zero_()                    # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(C.view(torch.int64), ref.view(torch.int64)), f"replay {rep}"
