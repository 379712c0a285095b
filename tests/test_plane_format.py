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



@pytest.mark.parametrize("set", [0, 1])
@pytest.mark.parametrize("side", [0, 1])
def test_plane_tables_match_oracle_planes(set, side):
    """The full-size GPU tests compare planes through tables of oracle.limbs
    over each modulus's centred residues; those tables must give exactly the
    bytes of oracle.planes (the oracle's direct per-element split), and the
    C comparison must find a planted difference and a nonzero pad byte."""
    import workloads
    from plane_check import CodeTables, oracle_residues
    X = workloads.random_matrix(300, 200, 2.0, 40 + side)
    X[3] = 0.0
    X[5, 7] = np.nan
    if side == 1:
        X = np.ascontiguousarray(X.T)
    k = X.shape[1] if side == 0 else X.shape[0]
    vecs = X.shape[0] if side == 0 else X.shape[1]
    exps = oracle.exponents(X, side, oracle.scale_bits(k, set))
    tabs = CodeTables(set)
    R = oracle_residues(X, side, exps, 0, vecs, set)
    P = oracle.planes(oracle.quantise_vectors(X, side, exps), set=set)
    want = (P.astype(np.int64) & 0xFF).astype(np.uint8) if set == 1 else e4m3_bytes(P)
    assert np.array_equal(tabs.codes(R), want[:, :, :k])
    assert tabs.compare(R, want) == (0, -1)
    bad = want.copy()
    bad[2, 17, 33] ^= 0x01
    assert tabs.compare(R, bad) == (1, (2 * vecs + 17) * want.shape[2] + 33)
    bad = want.copy()
    bad[-1, vecs - 1, -1] = 0x08
    assert tabs.compare(R, bad)[0] == 1
