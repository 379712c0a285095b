"""Seeded synthetic workloads for the emulated DGEMM.

This module only draws input matrices and names the workload shapes. It holds
none of the emulation method's arithmetic, so both the CPU oracle's tests and
the HIP path's tests and benchmark can use it without sharing method code.

Distribution (the paper's configurations): every entry is
``(U(0,1) - 0.5) * exp(s * N(0,1))`` in float64, with ``s`` fixed per
workload.  The generator is numpy's PCG64 seeded per workload; matrices are
drawn in the order A, B, C_in, each in chunks of 1024 rows, and within a chunk
the uniform block is drawn before the normal block.  Drawing by chunks keeps
the host memory of the draw bounded and makes the stream independent of how
the caller later tiles the matrix.
"""
from __future__ import annotations

import dataclasses
import numpy as np

CHUNK_ROWS = 1024


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    m: int
    n: int
    k: int
    s: float
    seed: int
    subtract: bool = False   # HPL-style trailing update C -= A.B

    @property
    def flops(self) -> float:
        """Emulated FP64 work, 2mnk."""
        return 2.0 * self.m * self.n * self.k


# The five workload classes: tiny, single-tile reach, large square, ragged
# square, and the HPL trailing update / block-Krylov pair.
WORKLOADS = {
    "tiny":   Workload("tiny", 64, 64, 64, 0.5, 1),
    "reach":  Workload("reach", 256, 256, 8192, 0.5, 2),
    "square": Workload("square", 8192, 8192, 8192, 1.0, 3),
    "ragged": Workload("ragged", 8191, 8209, 7937, 2.0, 4),
    "hpl":    Workload("hpl", 32768, 32768, 1024, 1.0, 5, subtract=True),
    "krylov": Workload("krylov", 262144, 128, 4096, 1.0, 6),
}


def draw(rng: np.random.Generator, rows: int, cols: int, s: float) -> np.ndarray:
    """One float64 matrix of (U - 0.5) * exp(s * N), drawn in row chunks."""
    out = np.empty((rows, cols), dtype=np.float64)
    for r0 in range(0, rows, CHUNK_ROWS):
        r1 = min(rows, r0 + CHUNK_ROWS)
        u = rng.random((r1 - r0, cols))
        g = rng.standard_normal((r1 - r0, cols))
        np.multiply(u - 0.5, np.exp(s * g), out=out[r0:r1])
    return out


def make_inputs(w: Workload | str, seed: int | None = None):
    """Return (A, B, C_in) for a workload; C_in is None unless it subtracts.

    A is m x k and B is k x n, both row-major float64.
    """
    if isinstance(w, str):
        w = WORKLOADS[w]
    rng = np.random.default_rng(w.seed if seed is None else seed)
    a = draw(rng, w.m, w.k, w.s)
    b = draw(rng, w.k, w.n, w.s)
    c = draw(rng, w.m, w.n, w.s) if w.subtract else None
    return a, b, c


def random_matrix(rows: int, cols: int, s: float, seed: int) -> np.ndarray:
    """A single seeded matrix of the same distribution (for ad-hoc shapes)."""
    return draw(np.random.default_rng(seed), rows, cols, s)


def edge_rows(X: np.ndarray, seed: int) -> np.ndarray:
    """Overwrite the first eleven rows of X (it needs at least eleven) with
    edge cases: zeros, subnormals, a lone smallest subnormal, a NaN, an
    infinity, huge values up to 1.7e308, small integers, one dominant entry,
    values that tie once scaled, negative zeros, and values at the
    normal/subnormal boundary.  Returns X."""
    rng = np.random.default_rng(seed)
    k = X.shape[1]
    X[0] = 0.0
    X[1] = rng.standard_normal(k) * 1e-310
    X[2] = 0.0
    X[2, k // 2] = 5e-324
    X[3, 3 % k] = np.nan
    X[4, 1 % k] = -np.inf
    X[5] = rng.standard_normal(k) * 1e300
    X[5, 0] = 1.7e308
    X[6] = np.round(rng.standard_normal(k) * 1000)
    X[7, 0] = 1e6
    X[8] = (rng.integers(-64, 64, size=k) + 0.5) * 2.0 ** -50
    X[8, 0] = 1.0
    X[9] = -0.0
    X[10] = rng.standard_normal(k) * 2.0 ** -1020
    return X


def boundary_values(M: int, P: int) -> list:
    """Integers in [-M/2, M/2) at or next to FP64 rounding boundaries at
    every magnitude from 2^54 up: powers of two and midpoints between
    neighbouring doubles, each with small offsets on both sides; values near
    small multiples of P (the weight of the reconstruction's high half) and
    the two ends of the range."""
    h = M // 2
    xs = []
    top = h.bit_length() - 1
    for b in range(54, top + 1):
        pw = 1 << b
        mid = pw + (5 << (b - 53)) + (1 << (b - 54))   # a midpoint with an odd neighbour below
        for base in (pw, mid):
            for d in (0, 1, -1, 2, -2, 17, -17, 33, -33, 64, -64, 1 << 12, -(1 << 12)):
                xs.append(base + d)
    for q in (1, 2, 3, 5):
        for d in (0, 1, -1, P // 2, -(P // 2), P // 2 - 1, 1 << 40):
            xs.append(q * P + d)
    xs += [h - 1, h - 2, -h, -h + 1]
    out = []
    for x in xs:
        for s in (x, -x):
            if -h <= s < h:
                out.append(s)
    return out
