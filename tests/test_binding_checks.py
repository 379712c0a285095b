"""The Python binding rejects mismatched shapes, dtypes and undersized
buffers with ValueError before it calls into the library (a wrong-sized
buffer would otherwise reach a kernel as a raw device pointer).  Shape and
size checks come before the device check, so CPU tensors exercise them
here; a correctly shaped CPU tensor is then refused for not being on the
GPU."""
import pytest
import torch

import paper_2609_09095_amd as oz


@pytest.fixture(scope="module", autouse=True)
def built_library():
    import os
    if not os.path.exists(oz.library_path()):
        from paper_2609_09095_amd import build
        build.build()
    oz.lib()


def f64(*shape):
    return torch.zeros(shape, dtype=torch.float64)


def raises(match, fn, *a, **kw):
    with pytest.raises(ValueError, match=match):
        fn(*a, **kw)


def test_dgemm_shapes():
    raises("B has 5 rows", oz.ozaki25_dgemm, f64(3, 4), f64(5, 2))
    raises(r"C has shape \(3, 3\)", oz.ozaki25_dgemm, f64(3, 4), f64(4, 2), f64(3, 3))
    raises("2-D float64", oz.ozaki25_dgemm, f64(3, 4).float(), f64(4, 2))
    raises("CUDA tensor", oz.ozaki25_dgemm, f64(3, 4), f64(4, 2))


def test_dgemm_sub_shapes():
    raises("B has 5 rows", oz.ozaki25_dgemm_sub, f64(3, 4), f64(5, 2), f64(3, 2))
    raises(r"C has shape \(2, 3\)", oz.ozaki25_dgemm_sub, f64(3, 4), f64(4, 2), f64(2, 3))
    raises("CUDA tensor", oz.ozaki25_dgemm_sub, f64(3, 4), f64(4, 2), f64(3, 2))


def test_dgemm_ex_shapes():
    raises("B has 3 rows", oz.ozaki25_dgemm_ex, f64(3, 4), f64(3, 2), f64(3, 2))
    raises(r"C has shape \(3, 1\)", oz.ozaki25_dgemm_ex, f64(3, 4), f64(4, 2), f64(3, 1))
    raises("workspace must be a tensor of dtype", oz.ozaki25_dgemm_ex, f64(3, 4), f64(4, 2), f64(3, 2),
           workspace=torch.zeros(10, dtype=torch.float32))
    raises("row-major", oz.ozaki25_dgemm_ex, f64(4, 3).t(), f64(4, 2), f64(3, 2))


def test_deconstruct_buffers():
    X = f64(10, 70)
    need = 30 * 10 * 128
    raises("planes holds", oz.ozaki25_deconstruct, 0, X, planes=torch.zeros(need - 1, dtype=torch.uint8))
    raises("planes must be a tensor", oz.ozaki25_deconstruct, 0, X, planes=torch.zeros(need, dtype=torch.int32))
    raises("exps holds", oz.ozaki25_deconstruct, 0, X, exps=torch.zeros(9, dtype=torch.int32))
    raises("exps holds", oz.ozaki25_deconstruct, 1, X, exps=torch.zeros(69, dtype=torch.int32))
    raises("side must be", oz.ozaki25_deconstruct, 2, X)
    raises("CUDA tensor", oz.ozaki25_deconstruct, 0, X)


def test_residue_gemm_buffers():
    m, n, k = 10, 6, 130
    pa = torch.zeros(oz.ozaki25_planes_bytes(m, k), dtype=torch.uint8)
    pb = torch.zeros(oz.ozaki25_planes_bytes(n, k), dtype=torch.uint8)
    raises("planesA holds", oz.ozaki25_residue_gemm, m, n, k, pa[:-1], pb)
    raises("planesB holds", oz.ozaki25_residue_gemm, m, n, k, pa, pb[:-1])
    raises("planesA holds", oz.ozaki25_residue_gemm, m + 1, n, k, pa, pb)
    raises("Cres holds", oz.ozaki25_residue_gemm, m, n, k, pa, pb, Cres=torch.zeros(12 * m * n - 1, dtype=torch.int32))
    raises("Cres must be", oz.ozaki25_residue_gemm, m, n, k, pa, pb, Cres=torch.zeros(12 * m * n, dtype=torch.int64))
    pa15 = torch.zeros(oz.ozaki25_planes_bytes(m, k, oz.A15), dtype=torch.uint8)
    raises("planesB holds", oz.ozaki25_residue_gemm, m, n, k, pa15, pa15[:15 * n * 256 - 1], set=oz.A15)
    raises("CUDA tensor", oz.ozaki25_residue_gemm, m, n, k, pa, pb)


def test_reconstruct_buffers():
    m, n = 7, 5
    ea, eb = torch.zeros(m, dtype=torch.int32), torch.zeros(n, dtype=torch.int32)
    raises("Cres holds", oz.ozaki25_reconstruct, torch.zeros(12 * m * n - 1, dtype=torch.int32), ea, eb)
    raises("Cres holds", oz.ozaki25_reconstruct, torch.zeros(12 * m * n, dtype=torch.int32), ea, eb, set=oz.A15)
    raises(r"C has shape \(5, 7\)", oz.ozaki25_reconstruct, torch.zeros(12 * m * n, dtype=torch.int32), ea, eb,
           C=f64(5, 7))
    raises("expsA must be", oz.ozaki25_reconstruct, torch.zeros(12 * m * n, dtype=torch.int32), ea.long(), eb)
    raises("CUDA tensor", oz.ozaki25_reconstruct, torch.zeros(12 * m * n, dtype=torch.int32), ea, eb)


def test_dgemm_planes_buffers():
    m, n, k = 9, 4, 200
    ea, eb = torch.zeros(m, dtype=torch.int32), torch.zeros(n, dtype=torch.int32)
    pa = torch.zeros(oz.ozaki25_planes_bytes(m, k), dtype=torch.uint8)
    pb = torch.zeros(oz.ozaki25_planes_bytes(n, k), dtype=torch.uint8)
    raises("planesA holds", oz.ozaki25_dgemm_planes, k, pa[:-1], ea, pb, eb)
    raises("planesA holds", oz.ozaki25_dgemm_planes, k + 128, pa, ea, pb, eb)
    raises("planesB holds", oz.ozaki25_dgemm_planes, k, pa, ea, pb[:-1], eb)
    raises(r"C has shape \(4, 9\)", oz.ozaki25_dgemm_planes, k, pa, ea, pb, eb, C=f64(4, 9))
    raises("CUDA tensor", oz.ozaki25_dgemm_planes, k, pa, ea, pb, eb)
