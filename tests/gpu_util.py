"""Helpers for the GPU parity tests: move seeded inputs to the device, run
the library through its C ABI, bring results back, and compare with the
oracle bit for bit."""
from __future__ import annotations

import os

import numpy as np

import paper_2609_09095_amd as oz


def require_gpu():
    import pytest
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    if not os.path.exists(oz.library_path()):
        raise RuntimeError("libozaki25.so is not built; GPU tests need the HIP library")
    oz.lib()


def log(msg: str):
    print(msg, flush=True)


def to_dev(a: np.ndarray):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def gpu_deconstruct(X: np.ndarray, side: int, set: int = oz.S12):
    import torch
    planes, exps = oz.ozaki25_deconstruct(side, to_dev(X), set=set)
    torch.cuda.synchronize()
    return planes, exps


def gpu_dgemm(A: np.ndarray, B: np.ndarray, C_in: np.ndarray | None = None, set: int = oz.S12):
    import torch
    Ad, Bd = to_dev(A), to_dev(B)
    if C_in is None:
        C = oz.ozaki25_dgemm(Ad, Bd, set=set)
    else:
        C = to_dev(C_in)
        oz.ozaki25_dgemm_sub(Ad, Bd, C, set=set)
    torch.cuda.synchronize()
    return C


def assert_bits_equal(got: np.ndarray, want: np.ndarray, what: str):
    """Bitwise equality of float64 arrays, except that any NaN matches any NaN."""
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    assert got.shape == want.shape, (what, got.shape, want.shape)
    gn, wn = np.isnan(got), np.isnan(want)
    assert np.array_equal(gn, wn), f"{what}: NaN pattern differs"
    g = got.view(np.uint64)[~gn]
    w = want.view(np.uint64)[~wn]
    bad = np.nonzero(g != w)[0]
    if bad.size:
        i = bad[0]
        raise AssertionError(f"{what}: {bad.size} outputs differ; first: got {got[~gn][i]!r} want {want[~wn][i]!r}")


def assert_int_equal(got: np.ndarray, want: np.ndarray, what: str):
    got = np.asarray(got)
    want = np.asarray(want)
    assert got.shape == want.shape, (what, got.shape, want.shape)
    bad = np.argwhere(got != want)
    if bad.size:
        idx = tuple(bad[0])
        raise AssertionError(f"{what}: {len(bad)} entries differ; first at {idx}: got {got[idx]} want {want[idx]}")


def device_layout(planes: np.ndarray) -> np.ndarray:
    """The library's plane layout [k_pad/128][planes][vecs][128] from the
    oracle's [planes][vecs][k_pad] (a pure index permutation)."""
    P = np.asarray(planes)
    npl, vecs, kp = P.shape
    assert kp % 128 == 0
    return np.ascontiguousarray(P.reshape(npl, vecs, kp // 128, 128).transpose(2, 0, 1, 3))


def int8_bytes(residues: np.ndarray) -> np.ndarray:
    """The all-byte set's plane format: each centred residue as a two's
    complement byte."""
    v = np.asarray(residues).astype(np.int64)
    if np.any(v < -128) or np.any(v > 127):
        raise ValueError("residue beyond int8")
    return (v & 0xFF).astype(np.uint8)


def e4m3_bytes(limbs: np.ndarray) -> np.ndarray:
    """OCP FP8 E4M3FN encoding of integer limbs (the stored plane format),
    written from the format: sign bit, 4-bit exponent of bias 7, 3-bit
    mantissa; zero is 0x00.  Integers need no subnormals.  Raises if a value
    is not exactly representable (Lemma 1 says every limb is)."""
    v = np.asarray(limbs).astype(np.int64)
    a = np.abs(v)
    if np.any(a > 240):
        raise ValueError("limb beyond the e4m3 integer range")
    e = (a >= 2).astype(np.int64) + (a >= 4) + (a >= 8) + (a >= 16) + (a >= 32) + (a >= 64) + (a >= 128)
    frac = (a - (np.int64(1) << e)) * 8  # mantissa * 2^e
    if np.any((a > 0) & (frac % (np.int64(1) << e) != 0)):
        raise ValueError("limb not exactly representable in e4m3")
    mant = frac >> e
    code = ((v < 0).astype(np.int64) << 7) | ((e + 7) << 3) | mant
    return np.where(a == 0, 0, code).astype(np.uint8)


def sample_indices(n: int, count: int, seed: int) -> np.ndarray:
    """Sorted sample of indices that always includes both ends (ragged tails)."""
    rng = np.random.default_rng(seed)
    if n <= count:
        return np.arange(n)
    idx = set(rng.choice(n, size=count - 4, replace=False).tolist())
    idx.update([0, 1, n - 2, n - 1])
    return np.array(sorted(idx))
