"""The stored plane format: limbs as OCP FP8 E4M3FN bytes.

The encoder the GPU tests use (gpu_util.e4m3_bytes, written from the format)
is pinned here against torch's float8_e4m3fn conversion, and every limb the
oracle produces must be encodable (Lemma 1: all three planes are
e4m3-exact)."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import e4m3_bytes


def _e4m3_integers():
    vals = list(range(0, 17))
    for step, lo, hi in ((2, 18, 32), (4, 32, 64), (8, 64, 128), (16, 128, 241)):
        vals += list(range(lo, hi, step))
    vals = sorted(set(vals))
    return np.array(sorted(set(vals + [-v for v in vals])), dtype=np.int64)


def test_encoder_matches_torch_float8():
    v = _e4m3_integers()
    want = torch.tensor(v, dtype=torch.float32).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    got = e4m3_bytes(v)
    assert np.array_equal(got, want)
    assert e4m3_bytes(np.array([0]))[0] == 0  # +0, never the -0 pattern 0x80


@pytest.mark.parametrize("bad", [17, -19, 21, 23, 33, 250])
def test_encoder_rejects_inexact(bad):
    with pytest.raises(ValueError):
        e4m3_bytes(np.array([bad]))


def test_oracle_limbs_are_encodable_and_round_trip():
    rng = np.random.default_rng(3)
    Z = rng.integers(-(1 << 55), 1 << 55, size=(24, 4096), dtype=np.int64)
    P = oracle.planes(Z)
    codes = e4m3_bytes(P)
    back = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float32).numpy()
    assert np.array_equal(back.astype(np.int64), P.astype(np.int64))
