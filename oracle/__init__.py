"""CPU oracle for the Ozaki Scheme II emulated DGEMM -- TEST INFRASTRUCTURE.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may use
this package.  It shares no code with the HIP library: the arithmetic lives in
``ozaki_oracle.c`` (plain scalar C, exact integer arithmetic, one IEEE
rounding), built with gcc into ``liboracle.so`` next to it; this module only
marshals numpy arrays into it and chains its steps in the paper's order
(Eq. (scale) -> Eq. (residueprod) -> Eq. (pieces)/Lemma 1 -> Eq. (garner),
Eq. (horner) -> single rounding).

``quant`` selects the quantiser of Eq. (scale): RN (round to nearest, ties
to even; Ozaki-II-RN) or TZ (truncation toward zero; Ozaki-II-TZ of Table
variants).  ``set`` selects the modulus set: 0 is the published twelve-modulus set, 1 the
all-byte candidate set A of Sec. 5.1 on the INT8 route (its centred residues
are the int8 planes, one per modulus).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ozaki_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

R = 12
NPLANES = 30
R_A = 15
NONFINITE = -(2 ** 31)


def num_moduli(set: int = 0) -> int:
    return R_A if set == 1 else R


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (plain -O2, single thread)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=gnu11", "-ffp-contract=off", "-shared", "-fPIC", "-o", tmp,
                               _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i64, i32 = ctypes.c_int64, ctypes.c_int32
        L.oracle_scale_bits.argtypes = [i64]
        L.oracle_scale_bits.restype = ctypes.c_int
        L.oracle_modulus.argtypes = [ctypes.c_int]
        L.oracle_modulus.restype = i64
        L.oracle_planes_of.argtypes = [ctypes.c_int]
        L.oracle_plane_base.argtypes = [ctypes.c_int]
        L.oracle_product_of_moduli.argtypes = [P, P]
        L.oracle_exponents.argtypes = [i64, i64, P, i64, i64, ctypes.c_int, P]
        L.oracle_quantise.argtypes = [ctypes.c_double, i32]
        L.oracle_quantise.restype = i64
        L.oracle_quantise_vectors.argtypes = [i64, i64, P, i64, i64, P, P]
        L.oracle_quantise_vectors_q.argtypes = [ctypes.c_int, i64, i64, P, i64, i64, P, P]
        L.oracle_quantise_tz.argtypes = [ctypes.c_double, i32]
        L.oracle_quantise_tz.restype = i64
        L.oracle_centred_mod.argtypes = [i64, i64]
        L.oracle_centred_mod.restype = i64
        L.oracle_residues.argtypes = [i64, i64, P, P]
        L.oracle_in_e4m3.argtypes = [i64]
        L.oracle_limbs.argtypes = [ctypes.c_int, i64, P]
        L.oracle_split16.argtypes = [i64, P]
        L.oracle_limb_product_table.argtypes = [ctypes.c_int, P]
        L.oracle_limb_product.argtypes = [ctypes.c_int, P, P]
        L.oracle_limb_product.restype = i64
        L.oracle_planes.argtypes = [i64, i64, i64, P, P]
        L.oracle_residue_gemm.argtypes = [i64, i64, i64, P, P, P]
        L.oracle_garner_constants.argtypes = [P]
        L.oracle_garner.argtypes = [i64, i64, P, P, P]
        L.oracle_exact_product.argtypes = [i64, i64, i64, P, P, P, P]
        L.oracle_round_scaled.argtypes = [i64, ctypes.c_uint64, ctypes.c_int]
        L.oracle_round_scaled.restype = ctypes.c_double
        L.oracle_reconstruct.argtypes = [i64, i64, P, P, P, P, ctypes.c_int, P, i64]
        L.oracle_native_fallback.argtypes = [i64, i64, i64, P, i64, P, i64, P, P, P, P, i64]
        L.oracle_mag_digit.argtypes = [ctypes.c_double, ctypes.c_int]
        L.oracle_mag_digits.argtypes = [i64, i64, P, i64, i64, P, P]
        L.oracle_bound_gemm.argtypes = [i64, i64, i64, P, P, P]
        L.oracle_acc_total.argtypes = [ctypes.c_int, i64]
        L.oracle_acc_shifts.argtypes = [ctypes.c_int, i64, i64, P, P, P, P, P]
        ci = ctypes.c_int
        L.oracle_set_num_moduli.argtypes = [ci]
        L.oracle_set_modulus.argtypes = [ci, ci]
        L.oracle_set_modulus.restype = i64
        L.oracle_set_product_of_moduli.argtypes = [ci, P, P]
        L.oracle_set_scale_bits.argtypes = [ci, i64]
        L.oracle_set_residues.argtypes = [ci, i64, i64, P, P]
        L.oracle_set_a_planes.argtypes = [i64, i64, i64, P, P]
        L.oracle_set_residue_gemm.argtypes = [ci, i64, i64, i64, P, P, P]
        L.oracle_set_garner_constants.argtypes = [ci, P]
        L.oracle_set_garner.argtypes = [ci, i64, i64, P, P, P]
        _lib = L
    return _lib


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


# ---------------------------------------------------------------- constants
def moduli(set: int = 0) -> list[int]:
    return [int(lib().oracle_set_modulus(set, i)) for i in range(num_moduli(set))]


def planes_of(i: int) -> int:
    return int(lib().oracle_planes_of(i))


def plane_base(i: int) -> int:
    return int(lib().oracle_plane_base(i))


def product_of_moduli(set: int = 0) -> int:
    hi = np.zeros(1, np.uint64)
    lo = np.zeros(1, np.uint64)
    lib().oracle_set_product_of_moduli(set, _p(hi), _p(lo))
    return (int(hi[0]) << 64) | int(lo[0])


def scale_bits(k: int, set: int = 0) -> int:
    return int(lib().oracle_set_scale_bits(set, k))


def garner_constants(set: int = 0) -> list[int]:
    w = np.zeros(num_moduli(set), np.int64)
    lib().oracle_set_garner_constants(set, _p(w))
    return [int(x) for x in w]


def k_pad(k: int) -> int:
    return (k + 127) // 128 * 128


# ---------------------------------------------------------------- scalars
def centred_mod(z: int, x: int) -> int:
    return int(lib().oracle_centred_mod(z, x))


def in_e4m3(v: int) -> bool:
    return bool(lib().oracle_in_e4m3(v))


def limbs(i: int, d: int) -> list[int]:
    out = np.zeros(3, np.int8)
    n = lib().oracle_limbs(i, d, _p(out))
    return [int(x) for x in out[:n]]


def limb_product(i: int, dl, el) -> int:
    a = np.zeros(3, np.int8)
    b = np.zeros(3, np.int8)
    a[: len(dl)] = dl
    b[: len(el)] = el
    return int(lib().oracle_limb_product(i, _p(a), _p(b)))


def split16(d: int) -> list[int]:
    out = np.zeros(3, np.int64)
    lib().oracle_split16(d, _p(out))
    return [int(x) for x in out]


def limb_product_table(i: int) -> np.ndarray:
    m = moduli()[i]
    out = np.zeros((m, m), np.int32)
    lib().oracle_limb_product_table(i, _p(out))
    return out


RN, TZ = 0, 1   # quantisers of Eq. (scale): Ozaki-II-RN and Ozaki-II-TZ


def quantise(x: float, sigma: int, quant: int = RN) -> int:
    if quant == TZ:
        return int(lib().oracle_quantise_tz(x, sigma))
    return int(lib().oracle_quantise(x, sigma))


def round_scaled(X: int, e: int) -> float:
    hi = X >> 64
    lo = X & ((1 << 64) - 1)
    return float(lib().oracle_round_scaled(hi, lo, e))


# ---------------------------------------------------------------- vectors
def _vec_view(X: np.ndarray, side: int):
    """(nvec, k, sv, sk) element strides for A rows (side 0) or B columns (1)."""
    X = np.ascontiguousarray(X, dtype=np.float64)
    if side == 0:
        nvec, k = X.shape
        return X, nvec, k, X.strides[0] // 8, 1
    k, nvec = X.shape
    return X, nvec, k, 1, X.strides[0] // 8


def exponents(X: np.ndarray, side: int, t: int) -> np.ndarray:
    """sigma (side 0: rows of A) or tau (side 1: columns of B)."""
    X, nvec, k, sv, sk = _vec_view(X, side)
    out = np.zeros(nvec, np.int32)
    lib().oracle_exponents(nvec, k, _p(X), sv, sk, t, _p(out))
    return out


def quantise_vectors(X: np.ndarray, side: int, exps: np.ndarray, quant: int = RN) -> np.ndarray:
    """Z[v][l]: the scaled, quantised integers of each row of A / column of B."""
    X, nvec, k, sv, sk = _vec_view(X, side)
    exps = np.ascontiguousarray(exps, dtype=np.int32)
    Z = np.zeros((nvec, k), np.int64)
    lib().oracle_quantise_vectors_q(quant, nvec, k, _p(X), sv, sk, _p(exps), _p(Z))
    return Z


def residues(Z: np.ndarray, set: int = 0) -> np.ndarray:
    Z = np.ascontiguousarray(Z, dtype=np.int64)
    nvec, k = Z.shape
    out = np.zeros((num_moduli(set), nvec, k), np.int16)
    lib().oracle_set_residues(set, nvec, k, _p(Z), _p(out))
    return out


def planes(Z: np.ndarray, kp: int | None = None, set: int = 0) -> np.ndarray:
    """Stored planes: the published set's limbs (30 planes), or set A's int8
    residues (15 planes)."""
    Z = np.ascontiguousarray(Z, dtype=np.int64)
    nvec, k = Z.shape
    kp = k_pad(k) if kp is None else kp
    if set == 1:
        out = np.zeros((R_A, nvec, kp), np.int8)
        lib().oracle_set_a_planes(nvec, k, kp, _p(Z), _p(out))
        return out
    out = np.zeros((NPLANES, nvec, kp), np.int8)
    lib().oracle_planes(nvec, k, kp, _p(Z), _p(out))
    return out


def residue_gemm(resA: np.ndarray, resB: np.ndarray, set: int = 0) -> np.ndarray:
    resA = np.ascontiguousarray(resA, dtype=np.int16)
    resB = np.ascontiguousarray(resB, dtype=np.int16)
    _, m, k = resA.shape
    _, n, k2 = resB.shape
    assert k == k2
    C = np.zeros((num_moduli(set), m, n), np.int32)
    lib().oracle_set_residue_gemm(set, m, n, k, _p(resA), _p(resB), _p(C))
    return C


def garner(Cres: np.ndarray, set: int = 0):
    """Returns (Xhi int64, Xlo uint64) of the reconstructed integers."""
    Cres = np.ascontiguousarray(Cres, dtype=np.int32)
    _, m, n = Cres.shape
    hi = np.zeros((m, n), np.int64)
    lo = np.zeros((m, n), np.uint64)
    lib().oracle_set_garner(set, m, n, _p(Cres), _p(hi), _p(lo))
    return hi, lo


def exact_product(ZA: np.ndarray, ZB: np.ndarray):
    ZA = np.ascontiguousarray(ZA, dtype=np.int64)
    ZB = np.ascontiguousarray(ZB, dtype=np.int64)
    m, k = ZA.shape
    n, _ = ZB.shape
    hi = np.zeros((m, n), np.int64)
    lo = np.zeros((m, n), np.uint64)
    lib().oracle_exact_product(m, n, k, _p(ZA), _p(ZB), _p(hi), _p(lo))
    return hi, lo


def reconstruct(Xhi, Xlo, expsA, expsB, C_in: np.ndarray | None = None) -> np.ndarray:
    Xhi = np.ascontiguousarray(Xhi, dtype=np.int64)
    Xlo = np.ascontiguousarray(Xlo, dtype=np.uint64)
    expsA = np.ascontiguousarray(expsA, dtype=np.int32)
    expsB = np.ascontiguousarray(expsB, dtype=np.int32)
    m, n = Xhi.shape
    if C_in is None:
        C = np.zeros((m, n), np.float64)
        sub = 0
    else:
        C = np.array(C_in, dtype=np.float64, copy=True, order="C")
        sub = 1
    lib().oracle_reconstruct(m, n, _p(Xhi), _p(Xlo), _p(expsA), _p(expsB), sub, _p(C), n)
    return C


def native_fallback(A: np.ndarray, B: np.ndarray, expsA, expsB, C: np.ndarray,
                    C_in: np.ndarray | None = None) -> np.ndarray:
    """Alg. 1's last step: outputs whose row of A or column of B is flagged
    non-finite by the exponent scan are overwritten, in place in C, by the
    index-order FP64 dot product (C_in minus it when C_in is given)."""
    A = np.ascontiguousarray(A, dtype=np.float64)
    B = np.ascontiguousarray(B, dtype=np.float64)
    expsA = np.ascontiguousarray(expsA, dtype=np.int32)
    expsB = np.ascontiguousarray(expsB, dtype=np.int32)
    m, k = A.shape
    _, n = B.shape
    assert C.shape == (m, n) and C.flags.c_contiguous and C.dtype == np.float64
    cin = None
    if C_in is not None:
        cin = np.ascontiguousarray(C_in, dtype=np.float64)
        assert cin.shape == (m, n)
    lib().oracle_native_fallback(m, n, k, _p(A), k, _p(B), n, _p(expsA), _p(expsB),
                                 _p(cin) if cin is not None else None, _p(C), n)
    return C


# ---------------------------------------------------------------- accurate mode
ACC_CAP = 58
ACC_INF = 100000


def frexp_exponents(X: np.ndarray, side: int) -> np.ndarray:
    """e of each row (side 0) / column (side 1): the frexp exponent of its
    largest magnitude (0 for a zero vector), NONFINITE for a non-finite one
    (the exponent scan at t = 0 gives -e)."""
    sig = exponents(X, side, 0).astype(np.int64)
    return np.where(sig == NONFINITE, NONFINITE, -sig).astype(np.int32)


def mag_digit(x: float, e: int) -> int:
    return int(lib().oracle_mag_digit(x, e))


def mag_digits(X: np.ndarray, side: int, e: np.ndarray) -> np.ndarray:
    """ceil(16 |x| 2^-e) per element, [vecs][k] uint8 (0 on non-finite vectors)."""
    X, nvec, k, sv, sk = _vec_view(X, side)
    e = np.ascontiguousarray(e, dtype=np.int32)
    D = np.zeros((nvec, k), np.uint8)
    lib().oracle_mag_digits(nvec, k, _p(X), sv, sk, _p(e), _p(D))
    return D


def bound_gemm(DA: np.ndarray, DB: np.ndarray, loops: bool | None = None) -> np.ndarray:
    """U = DA DB^T of the digit planes.  Plain int64 loops in C, or (large
    products, or loops=False) numpy's FP64 matmul: every partial sum is an
    integer at most 256 k < 2^53, so that product is exact in any order."""
    DA = np.ascontiguousarray(DA, dtype=np.uint8)
    DB = np.ascontiguousarray(DB, dtype=np.uint8)
    m, k = DA.shape
    n = DB.shape[0]
    if loops is None:
        loops = m * n * k <= (1 << 26)
    if not loops:
        return (DA.astype(np.float64) @ DB.astype(np.float64).T).astype(np.int64)
    U = np.zeros((m, n), np.int64)
    lib().oracle_bound_gemm(m, n, k, _p(DA), _p(DB), _p(U))
    return U


def acc_total(Uij: int, set: int = 0) -> int:
    return int(lib().oracle_acc_total(set, int(Uij)))


def acc_shifts(U: np.ndarray, flagA, flagB, set: int = 0):
    U = np.ascontiguousarray(U, dtype=np.int64)
    m, n = U.shape
    fa = np.ascontiguousarray(flagA, dtype=np.int32)
    fb = np.ascontiguousarray(flagB, dtype=np.int32)
    s = np.zeros(m, np.int32)
    u = np.zeros(n, np.int32)
    rc = lib().oracle_acc_shifts(set, m, n, _p(U), _p(fa), _p(fb), _p(s), _p(u))
    if rc == -2:
        raise MemoryError("oracle_acc_shifts: no host memory for the totals")
    if rc != 0:
        raise ValueError("accurate-mode shift below 4")
    return s, u


def accurate_exponents(A: np.ndarray, B: np.ndarray, set: int = 0):
    """sigma (rows of A) and tau (columns of B) of the accurate mode (the
    magnitude digits, the bound GEMM, the shifts), for the whole of A and B:
    every sigma_i depends on all columns of B and every tau_j on all rows of A."""
    eA = frexp_exponents(A, 0)
    eB = frexp_exponents(B, 1)
    U = bound_gemm(mag_digits(A, 0, eA), mag_digits(B, 1, eB))
    fa, fb = (eA == NONFINITE), (eB == NONFINITE)
    s, u = acc_shifts(U, fa, fb, set)
    sigma = np.where(fa, NONFINITE, s.astype(np.int64) - eA).astype(np.int32)
    tau = np.where(fb, NONFINITE, u.astype(np.int64) - eB).astype(np.int32)
    return sigma, tau, U, s, u


def to_int(hi, lo) -> np.ndarray:
    """Object array of Python ints from (hi, lo) words."""
    hi = np.asarray(hi)
    lo = np.asarray(lo)
    out = np.empty(hi.shape, dtype=object)
    for idx in np.ndindex(hi.shape):
        out[idx] = (int(hi[idx]) << 64) | int(lo[idx])
    return out


# ---------------------------------------------------------------- pipeline
class Result:
    """Every intermediate of one oracle run (for parity on each stage)."""

    def __init__(self, **kw):
        self.__dict__.update(kw)


def dgemm(A: np.ndarray, B: np.ndarray, C_in: np.ndarray | None = None,
          rows=None, cols=None, want_planes: bool = True, check_exact: bool = True,
          set: int = 0, quant: int = RN, fallback: bool = True, accurate: bool = False,
          accurate_exps=None) -> Result:
    """Oracle emulated DGEMM on the full k, for all outputs or for the sampled
    rows of A and columns of B (each output depends only on its row and
    column).  Steps in the order of Alg. 1: exponent scan, quantise, residues
    and limbs, per-modulus products, Garner, single rounding.  With
    ``check_exact`` the CRT result is compared with the direct integer
    product (they must be equal, since |A'B'| < M/2).  ``accurate`` takes
    sigma and tau from the accurate mode (accurate_exponents) instead of
    the fast rule t(k); ``accurate_exps`` may hand in the (sigma, tau) that
    accurate_exponents already gave for the whole of A and B.  With ``fallback``
    (Alg. 1's last step) outputs of rows / columns holding a NaN or an
    infinity are re-issued on the native FP64 path (``native_fallback``);
    without it they stay NaN, as the stage-wise reconstruction leaves them."""
    m, k = A.shape
    k2, n = B.shape
    assert k == k2
    rows = np.arange(m) if rows is None else np.asarray(rows)
    cols = np.arange(n) if cols is None else np.asarray(cols)
    t = scale_bits(k, set)
    As = np.ascontiguousarray(A[rows])
    Bs = np.ascontiguousarray(B[:, cols])
    if accurate:
        if accurate_exps is None:
            sig_all, tau_all, _, _, _ = accurate_exponents(A, B, set)
        else:
            sig_all, tau_all = accurate_exps
        sigma, tau = sig_all[rows], tau_all[cols]
    else:
        sigma = exponents(As, 0, t)
        tau = exponents(Bs, 1, t)
    ZA = quantise_vectors(As, 0, sigma, quant)
    ZB = quantise_vectors(Bs, 1, tau, quant)
    resA = residues(ZA, set)
    resB = residues(ZB, set)
    Cres = residue_gemm(resA, resB, set)
    Xhi, Xlo = garner(Cres, set)
    if check_exact:
        Ehi, Elo = exact_product(ZA, ZB)
        if not (np.array_equal(Ehi, Xhi) and np.array_equal(Elo, Xlo)):
            raise AssertionError("oracle: CRT reconstruction differs from the exact integer product")
    Cs = None if C_in is None else np.ascontiguousarray(C_in[np.ix_(rows, cols)])
    C = reconstruct(Xhi, Xlo, sigma, tau, Cs)
    if fallback:
        native_fallback(As, Bs, sigma, tau, C, Cs)
    r = Result(t=t, sigma=sigma, tau=tau, ZA=ZA, ZB=ZB, Cres=Cres, Xhi=Xhi, Xlo=Xlo, C=C,
               rows=rows, cols=cols)
    if want_planes:
        r.planesA = planes(ZA, set=set)
        r.planesB = planes(ZB, set=set)
    return r
