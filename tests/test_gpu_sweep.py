"""Seeded random shapes through the emulated DGEMM, bit for bit against the
oracle (any NaN matching any NaN): ragged m, n and k on both sides of the
tall/skinny threshold (storage mode F for A at most 128 columns and at least
1024 rows, the materialised planes otherwise), both modulus sets, both
quantisers (Eq. (scale)), C = AB and C -= AB, the fixed-t scales and the
accurate mode (Sec. 2, Eq. (alpha)), and a spread of exponent ranges, each
drawn per case from one seeded generator."""
import numpy as np
import pytest

import oracle
import paper_2609_09095_amd as oz
import workloads
from gpu_util import assert_bits_equal, log, require_gpu, to_dev

pytestmark = pytest.mark.gpu

NCASES = 24


@pytest.fixture(scope="module", autouse=True)
def gpu():
    require_gpu()


def _case(i):
    rng = np.random.default_rng(7000 + i)
    fused = i % 4 < 2
    m = int(rng.integers(1024, 1400)) if fused else int(rng.integers(1, 700))
    n = int(rng.integers(1, 129)) if fused else int(rng.integers(1, 300))
    k = int(rng.integers(1, 700))
    return dict(m=m, n=n, k=k, set=i % 2, tz=bool(rng.integers(0, 2)), sub=bool(rng.integers(0, 2)),
                accurate=(i // 2) % 3 == 2, s=float(rng.choice([0.5, 1.0, 2.0, 4.0])), seed=7100 + 3 * i)


def _run(A, B, C0, c):
    import torch
    m, k = A.shape
    n = B.shape[1]
    quant = oz.TZ if c["tz"] else oz.RN
    size = (oz.ozaki25_dgemm_accurate_workspace_size if c["accurate"] else oz.ozaki25_dgemm_workspace_size)
    ws = torch.empty(size(m, n, k, c["set"]), dtype=torch.uint8, device="cuda")
    C = to_dev(C0) if C0 is not None else torch.full((m, n), 7.0, dtype=torch.float64, device="cuda")
    call = oz.ozaki25_dgemm_accurate if c["accurate"] else oz.ozaki25_dgemm_ex
    call(to_dev(A), to_dev(B), C, subtract=C0 is not None, workspace=ws, set=c["set"], quantiser=quant)
    torch.cuda.synchronize()
    return C.cpu().numpy()


@pytest.mark.parametrize("i", range(NCASES))
def test_random_shape(i):
    c = _case(i)
    log(f"sweep case {i}: {c}")
    A = workloads.random_matrix(c["m"], c["k"], c["s"], c["seed"])
    B = workloads.random_matrix(c["k"], c["n"], c["s"], c["seed"] + 1)
    C0 = workloads.random_matrix(c["m"], c["n"], 1.0, c["seed"] + 2) if c["sub"] else None
    want = oracle.dgemm(A, B, C_in=C0, set=c["set"], accurate=c["accurate"], want_planes=False,
                        quant=oracle.TZ if c["tz"] else oracle.RN).C
    assert_bits_equal(_run(A, B, C0, c), want, f"C (case {i})")
