"""Full-operand comparison of the library's stored planes with the oracle's,
streamed in slabs of vectors so that host memory stays bounded at any size.

The oracle side of each slab is the oracle's own chain -- exponents,
quantiser (Eq. (scale)), centred residues (Eq. (residueprod)) -- followed by
the oracle's limb split (Eq. (pieces), Lemma 1) evaluated once per residue
value of each modulus: ``oracle.limbs(i, d)`` is a function of the modulus
and the residue alone, so a table of it over the centred range of each
modulus gives the same bytes as ``oracle.planes`` (checked by
``test_plane_tables_match_oracle_planes``).  The lookup and the byte
comparison run in a small C helper (tests/host/plane_compare.c, built with
gcc on first use), slabs on a thread pool (ctypes calls release the GIL).
Device slabs are permuted from the library's ``[k_pad/128][plane][vec][128]``
layout to ``[plane][vec][k_pad]`` on the GPU before they are copied back."""
from __future__ import annotations

import concurrent.futures as cf
import ctypes
import os
import subprocess

import numpy as np

import oracle
from gpu_util import e4m3_bytes, log

SLAB = 1024
_HOST = os.path.join(os.path.dirname(os.path.abspath(__file__)), "host")
_SRC = os.path.join(_HOST, "plane_compare.c")
_LIB = os.path.join(_HOST, "libplanecmp.so")
_lib = None


def workers() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def _helper():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            tmp = _LIB + ".tmp%d" % os.getpid()
            subprocess.check_call(["gcc", "-O2", "-std=gnu11", "-shared", "-fPIC", "-o", tmp, _SRC])
            os.replace(tmp, _LIB)
        L = ctypes.CDLL(_LIB)
        P, i64 = ctypes.c_void_p, ctypes.c_int64
        L.plane_compare.argtypes = [ctypes.c_int, P, P, P, P, i64, i64, i64, P, P, P]
        L.plane_compare.restype = i64
        _lib = L
    return _lib


def _p(a):
    return a.ctypes.data_as(ctypes.c_void_p)


class CodeTables:
    """Per modulus i, the stored bytes of every centred residue d (S12: the
    oracle's limbs as e4m3 codes; A15: the residue as a two's complement
    byte), packed as rows tab_off[i] + d + m//2 of a [sum m][3] table."""

    def __init__(self, set: int):
        self.mods = np.array(oracle.moduli(set), np.int64)
        rows, nl = [], []
        for i, m in enumerate(self.mods):
            lo = -(int(m) // 2)
            T = np.zeros((m, 3), np.uint8)
            if set == 1:
                T[:, 0] = (np.arange(lo, lo + m, dtype=np.int64) & 0xFF).astype(np.uint8)
                nl.append(1)
            else:
                L = e4m3_bytes(np.array([oracle.limbs(i, d) for d in range(lo, lo + m)], np.int64))
                T[:, :L.shape[1]] = L
                nl.append(L.shape[1])
            rows.append(T)
        self.tab = np.ascontiguousarray(np.concatenate(rows))
        self.nlimbs = np.array(nl, np.int32)
        self.tab_off = np.concatenate([[0], np.cumsum(self.mods)[:-1]]).astype(np.int64)
        self.nplanes = int(self.nlimbs.sum())

    def codes(self, R: np.ndarray) -> np.ndarray:
        """[planes][nv][k] bytes from residues [r][nv][k] (numpy; small inputs)."""
        out = []
        for i, m in enumerate(self.mods):
            rows = self.tab[self.tab_off[i] + R[i].astype(np.int64) + m // 2]
            out += [rows[..., p] for p in range(self.nlimbs[i])]
        return np.stack(out)

    def compare(self, R: np.ndarray, got: np.ndarray):
        """(number of differing bytes, first flat index into got or -1)."""
        r, nv, k = R.shape
        npl, nv2, kp = got.shape
        assert r == len(self.mods) and npl == self.nplanes and nv2 == nv and kp >= k
        R = np.ascontiguousarray(R, dtype=np.int16)
        got = np.ascontiguousarray(got, dtype=np.uint8)
        first = np.zeros(1, np.int64)
        bad = _helper().plane_compare(len(self.mods), _p(self.mods), _p(self.nlimbs), _p(self.tab_off),
                                      _p(self.tab), nv, k, kp, _p(R), _p(got), _p(first))
        return int(bad), int(first[0])


def oracle_residues(X: np.ndarray, side: int, exps: np.ndarray, v0: int, v1: int, set: int,
                    quant: int = oracle.RN) -> np.ndarray:
    """The oracle's centred residues [r][v1 - v0][k] of vectors v0..v1-1 (rows
    of A for side 0, columns of B for side 1)."""
    Xs = X[v0:v1] if side == 0 else np.ascontiguousarray(X[:, v0:v1])
    return oracle.residues(oracle.quantise_vectors(Xs, side, exps[v0:v1], quant), set)


def device_slab(planes_dev, v0: int, v1: int) -> np.ndarray:
    """Library planes of vectors v0..v1-1 as [plane][vec][k_pad] on the host."""
    kb, npl, _, ka = planes_dev.shape
    s = planes_dev[:, :, v0:v1, :].permute(1, 2, 0, 3).contiguous().reshape(npl, v1 - v0, kb * ka)
    return s.cpu().numpy()


def compare_planes_full(planes_dev, X: np.ndarray, side: int, exps: np.ndarray, set: int,
                        what: str, quant: int = oracle.RN) -> None:
    """Every byte of the library's planes of one operand (padding included)
    against the oracle, slab by slab."""
    k = X.shape[1] if side == 0 else X.shape[0]
    vecs = X.shape[0] if side == 0 else X.shape[1]
    tabs = CodeTables(set)
    slabs = [(v0, min(vecs, v0 + SLAB)) for v0 in range(0, vecs, SLAB)]
    nw = workers()
    log(f"[planes] {what}: {vecs} vectors x k={k} in {len(slabs)} slabs on {nw} threads")

    def one(s):
        R = oracle_residues(X, side, exps, s[0], s[1], set, quant)
        return s, tabs.compare(R, got_slabs.pop(s))

    got_slabs = {}
    with cf.ThreadPoolExecutor(max_workers=nw) as ex:
        futs = []
        for s in slabs:
            got_slabs[s] = device_slab(planes_dev, s[0], s[1])
            futs.append(ex.submit(one, s))
            while sum(not f.done() for f in futs) >= 2 * nw:
                futs[[f.done() for f in futs].index(False)].result()
        for j, f in enumerate(futs):
            s, (bad, first) = f.result()
            if j % 64 == 63:
                log(f"[planes] {what}: {j + 1} of {len(slabs)} slabs compared")
            if bad:
                npl, kp = tabs.nplanes, planes_dev.shape[0] * planes_dev.shape[3]
                nv = s[1] - s[0]
                q, rest = divmod(first, nv * kp)
                v, l = divmod(rest, kp)
                raise AssertionError(f"{what}: {bad} plane bytes differ in vectors {s[0]}..{s[1] - 1}; "
                                     f"first: plane {q} vector {s[0] + v} k {l}")
    log(f"[planes] {what}: all {len(slabs)} slabs equal")
