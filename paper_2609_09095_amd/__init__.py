"""MI355X-native emulated FP64 GEMM by Ozaki Scheme II on FP8 MFMA (published
moduli) or int8 MFMA (the all-byte moduli of Sec. 5.1, candidate A).

Python binding of ``libozaki25.so`` (the C ABI declared in
``include/ozaki25.h``).  Argument marshalling only: every step of the
computation runs in the library's HIP kernels.  PyTorch supplies device memory
and the current stream.  The binding fails loudly when the library has not
been built -- there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
import re

__all__ = [
    "Ozaki25Error", "lib", "library_path", "exported_symbols",
    "ozaki25_status_string", "ozaki25_num_moduli", "ozaki25_num_planes", "ozaki25_modulus",
    "ozaki25_scale_bits", "ozaki25_k_pad", "ozaki25_planes_bytes", "ozaki25_dgemm_workspace_size",
    "ozaki25_deconstruct", "ozaki25_residue_gemm", "ozaki25_reconstruct",
    "ozaki25_dgemm", "ozaki25_dgemm_sub", "ozaki25_dgemm_ex",
    "ozaki25_dgemm_planes_workspace_size", "ozaki25_dgemm_planes", "ozaki25_dgemm_noalloc",
    "ozaki25_accurate_exponents_workspace_size", "ozaki25_accurate_exponents",
    "ozaki25_dgemm_accurate_workspace_size", "ozaki25_dgemm_accurate",
]

_PKG = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_PKG, "libozaki25.so")
_HEADER = os.path.join(os.path.dirname(_PKG), "include", "ozaki25.h")

S12 = 0           # published moduli, FP8 limb route
A15 = 1           # all-byte moduli (Sec. 5.1 candidate A), int8 route
RN = 0            # quantiser: round to nearest, ties to even (Ozaki-II-RN)
TZ = 1            # quantiser: toward zero (Ozaki-II-TZ)
NUM_MODULI = 12
NUM_PLANES = 30
NUM_MODULI_A15 = 15
K_ALIGN = 128
MAX_K = 4194304
MAX_N = 8388608
EXP_NONFINITE = -(2 ** 31)
NUM_STAGE_EVENTS = 5
NOALLOC_SCRATCH_BYTES = 128 << 20

SUCCESS, ERR_INVALID_VALUE, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP = range(5)


class Ozaki25Error(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {ozaki25_status_string(status)} (status {status})")
        self.status = status


_lib = None


def library_path() -> str:
    return _LIB_PATH


def lib():
    """The loaded C library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise ImportError(f"{_LIB_PATH} is not built: run `python -m paper_2609_09095_amd.build`")
        L = ctypes.CDLL(_LIB_PATH)
        P, i64, i32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_size_t
        sig = {
            "ozaki25_status_string": ([i32], ctypes.c_char_p),
            "ozaki25_num_moduli": ([i32], i32),
            "ozaki25_num_planes": ([i32], i32),
            "ozaki25_modulus": ([i32, i32], i64),
            "ozaki25_scale_bits": ([i64, i32], i32),
            "ozaki25_k_pad": ([i64], i64),
            "ozaki25_planes_bytes": ([i64, i64, i32], sz),
            "ozaki25_deconstruct": ([i32, i64, i64, P, i64, i32, i32, P, P, P], i32),
            "ozaki25_residue_gemm": ([i64, i64, i64, P, P, i32, P, P], i32),
            "ozaki25_reconstruct": ([i64, i64, P, P, P, i32, P, i64, i32, P], i32),
            "ozaki25_dgemm_workspace_size": ([i64, i64, i64, i32], sz),
            "ozaki25_dgemm": ([i64, i64, i64, P, i64, P, i64, P, i64, i32, P], i32),
            "ozaki25_dgemm_sub": ([i64, i64, i64, P, i64, P, i64, P, i64, i32, P], i32),
            "ozaki25_dgemm_ex": ([i64, i64, i64, P, i64, P, i64, P, i64, i32, i32, i32, P, sz, P, P], i32),
            "ozaki25_dgemm_planes_workspace_size": ([i64, i64, i64, i32], sz),
            "ozaki25_dgemm_planes": ([i64, i64, i64, P, P, P, P, P, i64, i32, i32, P, sz, P], i32),
            "ozaki25_dgemm_noalloc": ([i64, i64, i64, P, i64, P, i64, P, i64, i32, i32, i32, P], i32),
            "ozaki25_accurate_exponents_workspace_size": ([i64, i64, i64], sz),
            "ozaki25_accurate_exponents": ([i64, i64, i64, P, i64, P, i64, i32, P, P, P, sz, P], i32),
            "ozaki25_dgemm_accurate_workspace_size": ([i64, i64, i64, i32], sz),
            "ozaki25_dgemm_accurate": ([i64, i64, i64, P, i64, P, i64, P, i64, i32, i32, i32, P, sz, P, P],
                                       i32),
        }
        for name, (args, res) in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = res
        _lib = L
    return _lib


def exported_symbols() -> list[str]:
    """Function names that include/ozaki25.h declares."""
    with open(_HEADER) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ozaki25_[a-z0-9_]+)\s*\(", text)))


# ----------------------------------------------------------------- helpers
def _check(status: int, what: str):
    if status != SUCCESS:
        raise Ozaki25Error(status, what)


def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def _on_gpu(ts):
    """Every tensor on one CUDA device (checked after the shapes and sizes,
    so that shape errors are reported first)."""
    dev = None
    for name, t in ts:
        if t is None:
            continue
        if not t.is_cuda:
            raise ValueError(f"{name} must be a CUDA tensor")
        if dev is None:
            dev = t.device
        elif t.device != dev:
            raise ValueError(f"{name} is on {t.device}, not on {dev} like the other operands")


def _matrix(t, name, shape=None):
    """A 2-D float64 row-major matrix; returns (t, leading dimension)."""
    import torch
    if not (isinstance(t, torch.Tensor) and t.dtype == torch.float64 and t.dim() == 2):
        raise ValueError(f"{name} must be a 2-D float64 tensor")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if t.stride(1) != 1 and t.shape[1] > 1:
        raise ValueError(f"{name} must be row-major (unit column stride)")
    if t.shape[0] > 1 and t.stride(0) < t.shape[1]:
        raise ValueError(f"{name} rows overlap (row stride below the row length)")
    return t, max(t.stride(0), t.shape[1], 1)


def _buffer(t, name, dtypes, numel):
    """A contiguous tensor of one of `dtypes` holding at least `numel` elements."""
    import torch
    if not isinstance(t, torch.Tensor) or t.dtype not in dtypes:
        raise ValueError(f"{name} must be a tensor of dtype {' or '.join(str(d) for d in dtypes)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.numel() < numel:
        raise ValueError(f"{name} holds {t.numel()} elements, needs at least {numel}")
    return t


def _u8():
    import torch
    return (torch.uint8, torch.int8)


def _i32():
    import torch
    return (torch.int32,)


# ----------------------------------------------------------------- host-only
def ozaki25_status_string(status: int) -> str:
    return lib().ozaki25_status_string(status).decode()


def ozaki25_num_moduli(set: int = S12) -> int:
    return lib().ozaki25_num_moduli(set)


def ozaki25_num_planes(set: int = S12) -> int:
    return lib().ozaki25_num_planes(set)


def ozaki25_modulus(i: int, set: int = S12) -> int:
    return lib().ozaki25_modulus(set, i)


def ozaki25_scale_bits(k: int, set: int = S12) -> int:
    return lib().ozaki25_scale_bits(k, set)


def ozaki25_k_pad(k: int) -> int:
    return lib().ozaki25_k_pad(k)


def ozaki25_planes_bytes(vecs: int, k: int, set: int = S12) -> int:
    return lib().ozaki25_planes_bytes(vecs, k, set)


def ozaki25_dgemm_workspace_size(m: int, n: int, k: int, set: int = S12) -> int:
    return lib().ozaki25_dgemm_workspace_size(m, n, k, set)


# ----------------------------------------------------------------- stages
def ozaki25_deconstruct(side: int, X, planes=None, exps=None, set: int = S12, quantiser: int = RN,
                        stream=None):
    """side 0: X is A (rows); side 1: X is B (columns).  Returns (planes, exps):
    planes uint8 [k_pad/128][num_planes][vecs][128] (S12: limbs as OCP e4m3
    bytes; A15: int8 residues as two's complement bytes), exps int32 [vecs]."""
    import torch
    if side not in (0, 1):
        raise ValueError(f"side must be 0 (A) or 1 (B), not {side}")
    X, ldx = _matrix(X, "X")
    vecs, k = (X.shape[0], X.shape[1]) if side == 0 else (X.shape[1], X.shape[0])
    kp = ozaki25_k_pad(k)
    npl = ozaki25_num_planes(set)
    if npl < 0:
        raise ValueError(f"unknown modulus set {set}")
    if planes is None:
        planes = torch.empty((kp // K_ALIGN, npl, vecs, K_ALIGN), dtype=torch.uint8, device=X.device)
    if exps is None:
        exps = torch.empty((vecs,), dtype=torch.int32, device=X.device)
    _buffer(planes, "planes", _u8(), npl * vecs * kp)
    _buffer(exps, "exps", _i32(), vecs)
    _on_gpu([("X", X), ("planes", planes), ("exps", exps)])
    _check(lib().ozaki25_deconstruct(side, vecs, k, _ptr(X), ldx, set, quantiser, _ptr(planes),
                                     _ptr(exps), _stream(stream)), "ozaki25_deconstruct")
    return planes, exps


def ozaki25_residue_gemm(m: int, n: int, k: int, planesA, planesB, Cres=None, set: int = S12,
                         stream=None):
    """Centred per-modulus products, int32 [r][m][n]."""
    import torch
    r = ozaki25_num_moduli(set)
    if r < 0:
        raise ValueError(f"unknown modulus set {set}")
    if min(m, n, k) < 0:
        raise ValueError("negative dimension")
    _buffer(planesA, "planesA", _u8(), ozaki25_planes_bytes(m, k, set))
    _buffer(planesB, "planesB", _u8(), ozaki25_planes_bytes(n, k, set))
    if Cres is None:
        Cres = torch.empty((r, m, n), dtype=torch.int32, device=planesA.device)
    _buffer(Cres, "Cres", _i32(), r * m * n)
    _on_gpu([("planesA", planesA), ("planesB", planesB), ("Cres", Cres)])
    _check(lib().ozaki25_residue_gemm(m, n, k, _ptr(planesA), _ptr(planesB), set, _ptr(Cres),
                                      _stream(stream)), "ozaki25_residue_gemm")
    return Cres


def ozaki25_reconstruct(Cres, expsA, expsB, C=None, subtract: bool = False, set: int = S12,
                        stream=None):
    """C (m x n float64) from int32 residues [r][m][n] and the exponents."""
    import torch
    r = ozaki25_num_moduli(set)
    if r < 0:
        raise ValueError(f"unknown modulus set {set}")
    _buffer(expsA, "expsA", _i32(), 0)
    _buffer(expsB, "expsB", _i32(), 0)
    m, n = expsA.numel(), expsB.numel()
    _buffer(Cres, "Cres", _i32(), r * m * n)
    if C is None:
        C = torch.empty((m, n), dtype=torch.float64, device=Cres.device)
    C, ldc = _matrix(C, "C", (m, n))
    _on_gpu([("Cres", Cres), ("expsA", expsA), ("expsB", expsB), ("C", C)])
    _check(lib().ozaki25_reconstruct(m, n, _ptr(Cres), _ptr(expsA), _ptr(expsB), set, _ptr(C), ldc,
                                     1 if subtract else 0, _stream(stream)), "ozaki25_reconstruct")
    return C


# ----------------------------------------------------------------- GEMM
def _workspace(workspace):
    if workspace is None:
        return ctypes.c_void_p(0), 0
    _buffer(workspace, "workspace", _u8(), 0)
    return _ptr(workspace), workspace.numel()


def _events(stage_events):
    if stage_events is None:
        return None
    handles = []
    for e in stage_events:
        if not hasattr(e, "cuda_event") or not e.cuda_event:
            raise ValueError("stage events must be recorded torch.cuda.Event objects")
        handles.append(e.cuda_event)
    if len(handles) != NUM_STAGE_EVENTS:
        raise ValueError(f"need {NUM_STAGE_EVENTS} stage events")
    return ctypes.cast((ctypes.c_void_p * NUM_STAGE_EVENTS)(*handles), ctypes.c_void_p)


def _operands(A, B):
    A, lda = _matrix(A, "A")
    m, k = A.shape
    B, ldb = _matrix(B, "B")
    if B.shape[0] != k:
        raise ValueError(f"B has {B.shape[0]} rows, A has {k} columns")
    return A, lda, B, ldb, m, B.shape[1], k


def ozaki25_dgemm_ex(A, B, C, subtract: bool = False, workspace=None, stage_events=None,
                     set: int = S12, quantiser: int = RN, stream=None):
    A, lda, B, ldb, m, n, k = _operands(A, B)
    C, ldc = _matrix(C, "C", (m, n))
    ev = _events(stage_events)
    ws_ptr, ws_bytes = _workspace(workspace)
    _on_gpu([("A", A), ("B", B), ("C", C), ("workspace", workspace)])
    _check(lib().ozaki25_dgemm_ex(m, n, k, _ptr(A), lda, _ptr(B), ldb, _ptr(C), ldc, set, quantiser,
                                  1 if subtract else 0, ws_ptr, ws_bytes, ev, _stream(stream)),
           "ozaki25_dgemm_ex")
    return C


def ozaki25_accurate_exponents_workspace_size(m: int, n: int, k: int) -> int:
    return lib().ozaki25_accurate_exponents_workspace_size(m, n, k)


def ozaki25_accurate_exponents(A, B, expsA=None, expsB=None, set: int = S12, workspace=None,
                               stream=None):
    """The accurate mode's sigma (rows of A) and tau (columns of B): the
    magnitude digits, their int8 bound product and the shifts it admits.
    Returns (expsA, expsB), int32 CUDA tensors."""
    import torch
    A, lda, B, ldb, m, n, k = _operands(A, B)
    if expsA is None:
        expsA = torch.empty(m, dtype=torch.int32, device=A.device)
    if expsB is None:
        expsB = torch.empty(n, dtype=torch.int32, device=A.device)
    _buffer(expsA, "expsA", _i32(), m)
    _buffer(expsB, "expsB", _i32(), n)
    ws_ptr, ws_bytes = _workspace(workspace)
    _on_gpu([("A", A), ("B", B), ("expsA", expsA), ("expsB", expsB), ("workspace", workspace)])
    _check(lib().ozaki25_accurate_exponents(m, n, k, _ptr(A), lda, _ptr(B), ldb, set, _ptr(expsA),
                                            _ptr(expsB), ws_ptr, ws_bytes, _stream(stream)),
           "ozaki25_accurate_exponents")
    return expsA, expsB


def ozaki25_dgemm_accurate_workspace_size(m: int, n: int, k: int, set: int = S12) -> int:
    return lib().ozaki25_dgemm_accurate_workspace_size(m, n, k, set)


def ozaki25_dgemm_accurate(A, B, C=None, subtract: bool = False, workspace=None, stage_events=None,
                           set: int = S12, quantiser: int = RN, stream=None):
    """C = A B (or C -= A B) in the accurate mode: per-row and per-column
    shifts from the magnitude-bound product instead of the fixed t(k)."""
    import torch
    A, lda, B, ldb, m, n, k = _operands(A, B)
    if C is None:
        if subtract:
            raise ValueError("subtract needs C")
        C = torch.empty((m, n), dtype=torch.float64, device=A.device)
    C, ldc = _matrix(C, "C", (m, n))
    ev = _events(stage_events)
    ws_ptr, ws_bytes = _workspace(workspace)
    _on_gpu([("A", A), ("B", B), ("C", C), ("workspace", workspace)])
    _check(lib().ozaki25_dgemm_accurate(m, n, k, _ptr(A), lda, _ptr(B), ldb, _ptr(C), ldc, set, quantiser,
                                        1 if subtract else 0, ws_ptr, ws_bytes, ev, _stream(stream)),
           "ozaki25_dgemm_accurate")
    return C


def ozaki25_dgemm(A, B, C=None, set: int = S12, stream=None):
    """C = A B (float64, row-major CUDA tensors)."""
    import torch
    A, lda = _matrix(A, "A")
    m, k = A.shape
    B, ldb = _matrix(B, "B")
    if B.shape[0] != k:
        raise ValueError(f"B has {B.shape[0]} rows, A has {k} columns")
    n = B.shape[1]
    if C is None:
        C = torch.empty((m, n), dtype=torch.float64, device=A.device)
    C, ldc = _matrix(C, "C", (m, n))
    _on_gpu([("A", A), ("B", B), ("C", C)])
    _check(lib().ozaki25_dgemm(m, n, k, _ptr(A), lda, _ptr(B), ldb, _ptr(C), ldc, set,
                               _stream(stream)), "ozaki25_dgemm")
    return C


def ozaki25_dgemm_sub(A, B, C, set: int = S12, stream=None):
    """C <- C - A B in place."""
    A, lda = _matrix(A, "A")
    m, k = A.shape
    B, ldb = _matrix(B, "B")
    if B.shape[0] != k:
        raise ValueError(f"B has {B.shape[0]} rows, A has {k} columns")
    n = B.shape[1]
    C, ldc = _matrix(C, "C", (m, n))
    _on_gpu([("A", A), ("B", B), ("C", C)])
    _check(lib().ozaki25_dgemm_sub(m, n, k, _ptr(A), lda, _ptr(B), ldb, _ptr(C), ldc, set,
                                   _stream(stream)), "ozaki25_dgemm_sub")
    return C


def ozaki25_dgemm_planes_workspace_size(m: int, n: int, k: int, set: int = S12) -> int:
    return lib().ozaki25_dgemm_planes_workspace_size(m, n, k, set)


def ozaki25_dgemm_planes(k: int, planesA, expsA, planesB, expsB, C=None, subtract: bool = False,
                         workspace=None, set: int = S12, stream=None):
    """C = A B (or C -= A B) from stored planes (storage mode P): planes and
    exponents from ozaki25_deconstruct of A (side 0) and B (side 1) with this
    k and set.  m and n come from the exponent vectors."""
    import torch
    npl = ozaki25_num_planes(set)
    if npl < 0:
        raise ValueError(f"unknown modulus set {set}")
    if k < 0:
        raise ValueError("negative k")
    _buffer(expsA, "expsA", _i32(), 0)
    _buffer(expsB, "expsB", _i32(), 0)
    m, n = expsA.numel(), expsB.numel()
    _buffer(planesA, "planesA", _u8(), ozaki25_planes_bytes(m, k, set))
    _buffer(planesB, "planesB", _u8(), ozaki25_planes_bytes(n, k, set))
    if C is None:
        C = torch.empty((m, n), dtype=torch.float64, device=expsA.device)
    C, ldc = _matrix(C, "C", (m, n))
    ws_ptr, ws_bytes = _workspace(workspace)
    _on_gpu([("planesA", planesA), ("expsA", expsA), ("planesB", planesB), ("expsB", expsB), ("C", C),
             ("workspace", workspace)])
    _check(lib().ozaki25_dgemm_planes(m, n, k, _ptr(planesA), _ptr(expsA), _ptr(planesB), _ptr(expsB),
                                      _ptr(C), ldc, set, 1 if subtract else 0, ws_ptr, ws_bytes,
                                      _stream(stream)), "ozaki25_dgemm_planes")
    return C


def ozaki25_dgemm_noalloc(A, B, C=None, subtract: bool = False, set: int = S12, quantiser: int = RN,
                          stream=None):
    """C = A B (or C -= A B) with the library's static per-GPU workspace of
    NOALLOC_SCRATCH_BYTES: no device allocation.  Products whose workspace
    (ozaki25_dgemm_workspace_size) exceeds it raise Ozaki25Error with
    ERR_WORKSPACE.  Calls that overlap on one GPU race on that workspace."""
    import torch
    A, lda = _matrix(A, "A")
    m, k = A.shape
    B, ldb = _matrix(B, "B")
    if B.shape[0] != k:
        raise ValueError(f"B has {B.shape[0]} rows, A has {k} columns")
    n = B.shape[1]
    if C is None:
        if subtract:
            raise ValueError("subtract needs C")
        C = torch.empty((m, n), dtype=torch.float64, device=A.device)
    C, ldc = _matrix(C, "C", (m, n))
    _on_gpu([("A", A), ("B", B), ("C", C)])
    _check(lib().ozaki25_dgemm_noalloc(m, n, k, _ptr(A), lda, _ptr(B), ldb, _ptr(C), ldc, set, quantiser,
                                       1 if subtract else 0, _stream(stream)), "ozaki25_dgemm_noalloc")
    return C
