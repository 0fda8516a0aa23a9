"""2M + Ozaki-II complex GEMM / HERK / SYRK / HER2K / SYR2K on MI355X (gfx950).

Thin ctypes binding over the C-ABI library ``libo2m.so`` (include/o2m.h).
Every step of the computation runs in the library's HIP kernels; this module
only marshals torch tensors (device memory and the current stream) into the
C calls.  There is no fallback: if the library is missing, importing this
package raises.

Matrices are column-major: a tensor ``A`` of shape (m, k) must have
``A.stride(0) == 1`` (``colmajor(x)`` makes such a tensor).  Outputs are
allocated column-major as well.
"""
from __future__ import annotations

import ctypes
import os

import torch

__all__ = [
    "zgemm_2m", "zgemm_2m_noalloc", "cgemm_2m", "zgemm_2m_op", "cgemm_2m_op", "zherk_2m", "dsyrk_2m",
    "zher2k_2m", "dsyr2k_2m", "gauss_gemm_2m",
    "zgemm_2m_residues", "moduli", "budget", "shifts", "workspace_bytes", "set_workspace",
    "release_workspace", "get_status", "STATUS_OVERFLOW", "STATUS_NONFINITE", "phase_timing", "phase_times", "colmajor", "O2MError", "LIB_PATH", "SCALING",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libo2m.so")
if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it first (python -c 'import __graft_entry__ as g; g.build()')")

_L = ctypes.CDLL(LIB_PATH)
_I, _P, _D = ctypes.c_int, ctypes.c_void_p, ctypes.c_double
_C = ctypes.c_char
_L.zgemm_2m.argtypes = [_I, _I, _I, _P, _I, _P, _I, _P, _I, _I, _P]
_L.cgemm_2m.argtypes = [_I, _I, _I, _P, _I, _P, _I, _P, _I, _I, _P]
_L.zgemm_2m_noalloc.argtypes = [_I, _I, _I, _P, _I, _P, _I, _P, _I, _I, _I, _P]
_L.zherk_2m.argtypes = [_C, _I, _I, _P, _I, _P, _I, _I, _P]
_L.dsyrk_2m.argtypes = [_C, _I, _I, _P, _I, _P, _I, _I, _P]
_L.zher2k_2m.argtypes = [_C, _I, _I, _P, _I, _P, _I, _P, _I, _I, _P]
_L.dsyr2k_2m.argtypes = [_C, _I, _I, _P, _I, _P, _I, _P, _I, _I, _P]
_L.zgemm_2m_ex.argtypes = [_I, _I, _I, _P, _I, _P, _I, _P, _I, _I, _I, _P]
_L.cgemm_2m_ex.argtypes = [_I, _I, _I, _P, _I, _P, _I, _P, _I, _I, _I, _P]
_L.zgemm_2m_op.argtypes = [_C, _C, _I, _I, _I, _P, _I, _P, _I, _P, _I, _I, _I, _P]
_L.cgemm_2m_op.argtypes = [_C, _C, _I, _I, _I, _P, _I, _P, _I, _P, _I, _I, _I, _P]
_L.zherk_2m_ex.argtypes = [_C, _I, _I, _P, _I, _P, _I, _I, _I, _P]
_L.dsyrk_2m_ex.argtypes = [_C, _I, _I, _P, _I, _P, _I, _I, _I, _P]
_L.zher2k_2m_ex.argtypes = [_C, _I, _I, _P, _I, _P, _I, _P, _I, _I, _I, _P]
_L.dsyr2k_2m_ex.argtypes = [_C, _I, _I, _P, _I, _P, _I, _P, _I, _I, _I, _P]
_L.gauss_gemm_2m.argtypes = [_I, _I, _I, _P, _I, _P, _I, _P, _I, _I, _P]
_L.zgemm_2m_residues.argtypes = [_I, _I, _I, _P, _I, _P, _I, _I, _P, _P, _P, _P]
_L.zgemm_2m_residues_ex.argtypes = [_I, _I, _I, _P, _I, _P, _I, _I, _I, _P, _P, _P, _P]
_L.o2m_moduli.argtypes = [_I, _P, _P, _P]
_L.o2m_budget.argtypes = [_I, _I, _P]
_L.o2m_shifts.argtypes = [_C, _I, _I, _I, _P, _P]
_L.o2m_workspace_bytes.argtypes = [ctypes.c_char, _I, _I, _I, _I]
_L.o2m_workspace_bytes.restype = ctypes.c_size_t
_L.o2m_set_workspace.argtypes = [_P, ctypes.c_size_t, _P]
_L.o2m_release_workspace.argtypes = [_P]
_L.o2m_get_status.argtypes = [_P, _P]
_L.o2m_phase_timing.argtypes = [_I]
_L.o2m_phase_times.argtypes = [_P, _I]
_L.o2m_status_string.argtypes = [_I]
_L.o2m_status_string.restype = ctypes.c_char_p
for _f in ("zgemm_2m", "zgemm_2m_noalloc", "cgemm_2m", "zherk_2m", "dsyrk_2m", "zher2k_2m", "dsyr2k_2m", "zgemm_2m_ex",
           "cgemm_2m_ex", "zgemm_2m_op", "cgemm_2m_op", "zherk_2m_ex", "dsyrk_2m_ex", "zher2k_2m_ex", "dsyr2k_2m_ex", "gauss_gemm_2m",
           "zgemm_2m_residues", "zgemm_2m_residues_ex", "o2m_moduli", "o2m_budget", "o2m_shifts",
           "o2m_set_workspace", "o2m_release_workspace", "o2m_get_status", "o2m_phase_timing",
           "o2m_phase_times"):
    getattr(_L, _f).restype = _I

STATUS_OVERFLOW = 1
STATUS_NONFINITE = 2
# scaling rules: "max" (per-row maximum) and "cs" (Cauchy-Schwarz, 2-norm)
SCALING = {"max": 0, "cs": 1}


def _rule(scaling: str) -> int:
    try:
        return SCALING[scaling]
    except KeyError:
        raise ValueError(f"unknown scaling rule {scaling!r}; expected one of {sorted(SCALING)}") from None


class O2MError(RuntimeError):
    def __init__(self, status: int, where: str):
        msg = _L.o2m_status_string(status).decode()
        super().__init__(f"{where}: status {status} ({msg})")
        self.status = status


def _check(status: int, where: str) -> None:
    if status != 0:
        raise O2MError(status, where)


def colmajor(x: torch.Tensor) -> torch.Tensor:
    """Same values, column-major storage (stride(0) == 1)."""
    return x.t().contiguous().t()


def _ld(x: torch.Tensor) -> int:
    if x.dim() != 2:
        raise ValueError("expected a matrix")
    if x.numel() == 0:
        return max(x.size(0), 1)                 # nothing is read or written
    if x.size(0) > 1 and x.stride(0) != 1:
        raise ValueError("matrix must be column-major (stride(0) == 1); use colmajor()")
    return max(x.stride(1), x.size(0), 1)


def _stream(stream) -> int:
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _empty_colmajor(rows: int, cols: int, dtype, device) -> torch.Tensor:
    return torch.empty((cols, rows), dtype=dtype, device=device).t()


def _check_operands(A, B, dtype):
    for name, x in (("A", A), ("B", B)):
        if x.dtype != dtype:
            raise TypeError(f"{name} must be {dtype}, got {x.dtype}")
        if not x.is_cuda:
            raise ValueError(f"{name} must be a device tensor")
    if A.size(1) != B.size(0):
        raise ValueError(f"inner dimensions differ: {tuple(A.shape)} x {tuple(B.shape)}")


def zgemm_2m(A: torch.Tensor, B: torch.Tensor, n_moduli: int = 16, out: torch.Tensor | None = None,
             stream=None, scaling: str = "max") -> torch.Tensor:
    """C = A B for complex128 A (m x k), B (k x n) by 2M + Ozaki-II."""
    _check_operands(A, B, torch.complex128)
    m, k = A.shape
    n = B.size(1)
    C = _empty_colmajor(m, n, torch.complex128, A.device) if out is None else out
    _check(_L.zgemm_2m_ex(m, n, k, A.data_ptr(), _ld(A), B.data_ptr(), _ld(B), C.data_ptr(), _ld(C),
                          n_moduli, _rule(scaling), _stream(stream)), "zgemm_2m")
    return C


NOALLOC_SCRATCH_BYTES = 256 << 20


def zgemm_2m_noalloc(A: torch.Tensor, B: torch.Tensor, out: torch.Tensor, n_moduli: int = 16, stream=None,
                     scaling: str = "max") -> torch.Tensor:
    """zgemm_2m into the caller's ``out`` through the entry point that
    allocates no device memory (its scratch is a static array of
    NOALLOC_SCRATCH_BYTES per GPU; calls that overlap on one GPU race)."""
    _check_operands(A, B, torch.complex128)
    m, k = A.shape
    n = B.size(1)
    if out.dtype != torch.complex128 or not out.is_cuda or tuple(out.shape) != (m, n):
        raise ValueError(f"out must be a complex128 device tensor of shape {(m, n)}")
    _check(_L.zgemm_2m_noalloc(m, n, k, A.data_ptr(), _ld(A), B.data_ptr(), _ld(B), out.data_ptr(), _ld(out),
                               n_moduli, _rule(scaling), _stream(stream)), "zgemm_2m_noalloc")
    return out


def cgemm_2m(A: torch.Tensor, B: torch.Tensor, n_moduli: int = 8, out: torch.Tensor | None = None,
             stream=None, scaling: str = "max") -> torch.Tensor:
    """C = A B for complex64 A, B by 2M + Ozaki-II (result rounded to fp32)."""
    _check_operands(A, B, torch.complex64)
    m, k = A.shape
    n = B.size(1)
    C = _empty_colmajor(m, n, torch.complex64, A.device) if out is None else out
    _check(_L.cgemm_2m_ex(m, n, k, A.data_ptr(), _ld(A), B.data_ptr(), _ld(B), C.data_ptr(), _ld(C),
                          n_moduli, _rule(scaling), _stream(stream)), "cgemm_2m")
    return C


def _gemm_op(fn, name, A, B, transa, transb, dtype, n_moduli, out, stream, scaling):
    for nm, x in (("A", A), ("B", B)):
        if x.dtype != dtype:
            raise TypeError(f"{nm} must be {dtype}, got {x.dtype}")
        if not x.is_cuda:
            raise ValueError(f"{nm} must be a device tensor")
    ta, tb = transa.upper(), transb.upper()
    if ta not in ("N", "T", "C") or tb not in ("N", "T", "C"):
        raise ValueError(f"transa, transb must be 'N', 'T' or 'C', got {transa!r}, {transb!r}")
    m, k = A.shape if ta == "N" else (A.size(1), A.size(0))
    kb, n = B.shape if tb == "N" else (B.size(1), B.size(0))
    if k != kb:
        raise ValueError(f"inner dimensions differ: op(A) {m} x {k}, op(B) {kb} x {n}")
    C = _empty_colmajor(m, n, dtype, A.device) if out is None else out
    _check(fn(ta.encode(), tb.encode(), m, n, k, A.data_ptr(), _ld(A), B.data_ptr(), _ld(B), C.data_ptr(),
              _ld(C), n_moduli, _rule(scaling), _stream(stream)), name)
    return C


def zgemm_2m_op(A: torch.Tensor, B: torch.Tensor, transa: str = "N", transb: str = "N", n_moduli: int = 16,
                out: torch.Tensor | None = None, stream=None, scaling: str = "max") -> torch.Tensor:
    """C = op(A) op(B) for complex128 tensors, op = 'N' (as is), 'T'
    (transpose) or 'C' (conjugate transpose); A and B as stored (column-major)."""
    return _gemm_op(_L.zgemm_2m_op, "zgemm_2m_op", A, B, transa, transb, torch.complex128, n_moduli, out, stream,
                    scaling)


def cgemm_2m_op(A: torch.Tensor, B: torch.Tensor, transa: str = "N", transb: str = "N", n_moduli: int = 8,
                out: torch.Tensor | None = None, stream=None, scaling: str = "max") -> torch.Tensor:
    """As zgemm_2m_op for complex64 tensors (result rounded once to fp32)."""
    return _gemm_op(_L.cgemm_2m_op, "cgemm_2m_op", A, B, transa, transb, torch.complex64, n_moduli, out, stream,
                    scaling)


def _sym_out(out, n, dtype, device):
    return colmajor(torch.zeros((n, n), dtype=dtype, device=device)) if out is None else out


def _uplo(uplo: str) -> bytes:
    if uplo not in ("L", "U", "l", "u"):
        raise ValueError(f"uplo must be 'L' or 'U', got {uplo!r}")
    return uplo.upper().encode()


def zherk_2m(A: torch.Tensor, n_moduli: int = 16, out: torch.Tensor | None = None, stream=None,
             scaling: str = "max", uplo: str = "L") -> torch.Tensor:
    """Lower (uplo 'L') or upper ('U') triangle of C = A A^H (complex128 A,
    n x k).  The other strict triangle of a fresh output is zero-initialised;
    of ``out`` it is left alone."""
    if A.dtype != torch.complex128 or not A.is_cuda:
        raise TypeError("A must be a complex128 device tensor")
    n, k = A.shape
    out = _sym_out(out, n, torch.complex128, A.device)
    _check(_L.zherk_2m_ex(_uplo(uplo), n, k, A.data_ptr(), _ld(A), out.data_ptr(), _ld(out), n_moduli,
                          _rule(scaling), _stream(stream)), "zherk_2m")
    return out


def dsyrk_2m(A: torch.Tensor, n_moduli: int = 16, out: torch.Tensor | None = None, stream=None,
             scaling: str = "max", uplo: str = "L") -> torch.Tensor:
    """Lower or upper triangle of C = A A^T (float64 A, n x k) via the half-k
    2M HERK."""
    if A.dtype != torch.float64 or not A.is_cuda:
        raise TypeError("A must be a float64 device tensor")
    n, k = A.shape
    out = _sym_out(out, n, torch.float64, A.device)
    _check(_L.dsyrk_2m_ex(_uplo(uplo), n, k, A.data_ptr(), _ld(A), out.data_ptr(), _ld(out), n_moduli,
                          _rule(scaling), _stream(stream)), "dsyrk_2m")
    return out


def _check_pair(A, B, dtype):
    for name, x in (("A", A), ("B", B)):
        if x.dtype != dtype or not x.is_cuda:
            raise TypeError(f"{name} must be a {dtype} device tensor")
    if A.shape != B.shape:
        raise ValueError(f"A and B must have the same shape: {tuple(A.shape)} vs {tuple(B.shape)}")


def zher2k_2m(A: torch.Tensor, B: torch.Tensor, n_moduli: int = 16, out: torch.Tensor | None = None,
              stream=None, scaling: str = "max", uplo: str = "L") -> torch.Tensor:
    """Lower or upper triangle of C = A B^H + B A^H (complex128 A, B: n x k)."""
    _check_pair(A, B, torch.complex128)
    n, k = A.shape
    out = _sym_out(out, n, torch.complex128, A.device)
    _check(_L.zher2k_2m_ex(_uplo(uplo), n, k, A.data_ptr(), _ld(A), B.data_ptr(), _ld(B), out.data_ptr(), _ld(out),
                           n_moduli, _rule(scaling), _stream(stream)), "zher2k_2m")
    return out


def dsyr2k_2m(A: torch.Tensor, B: torch.Tensor, n_moduli: int = 16, out: torch.Tensor | None = None,
              stream=None, scaling: str = "max", uplo: str = "L") -> torch.Tensor:
    """Lower or upper triangle of C = A B^T + B A^T (float64 A, B: n x k) via
    the half-k 2M HER2K."""
    _check_pair(A, B, torch.float64)
    n, k = A.shape
    out = _sym_out(out, n, torch.float64, A.device)
    _check(_L.dsyr2k_2m_ex(_uplo(uplo), n, k, A.data_ptr(), _ld(A), B.data_ptr(), _ld(B), out.data_ptr(), _ld(out),
                           n_moduli, _rule(scaling), _stream(stream)), "dsyr2k_2m")
    return out


def gauss_gemm_2m(A: torch.Tensor, B: torch.Tensor, n_moduli: int = 4, out: torch.Tensor | None = None,
                  stream=None) -> torch.Tensor:
    """Exact Gaussian-integer product.  A: int32 tensor of shape (m, k, 2) whose
    storage is column-major complex (stride (2, 2*lda, 1)); likewise B.  The
    result is int64 of shape (m, n, 2), column-major complex."""
    def ld3(x):
        if x.dtype != torch.int32 or x.dim() != 3 or x.size(2) != 2 or x.stride(2) != 1 or x.stride(0) != 2:
            raise ValueError("expected int32 (rows, cols, 2) with column-major complex storage")
        return max(x.stride(1) // 2, x.size(0), 1)
    m, k = A.shape[:2]
    n = B.size(1)
    if B.size(0) != k:
        raise ValueError("inner dimensions differ")
    if out is None:
        out = torch.empty((n, m, 2), dtype=torch.int64, device=A.device).transpose(0, 1)
    _check(_L.gauss_gemm_2m(m, n, k, A.data_ptr(), ld3(A), B.data_ptr(), ld3(B), out.data_ptr(),
                            max(out.stride(1) // 2, m, 1), n_moduli, _stream(stream)), "gauss_gemm_2m")
    return out


def zgemm_2m_residues(A: torch.Tensor, B: torch.Tensor, n_moduli: int = 16, stream=None, scaling: str = "max"):
    """Test hook: per-modulus (Re c mod m_l, Im c mod m_l) of the quantized
    product, int8 [n_moduli, 2, n, m] (symmetric residues), and the row /
    column exponents E (m,), F (n,) of the scaling rule."""
    _check_operands(A, B, torch.complex128)
    m, k = A.shape
    n = B.size(1)
    res = torch.empty((n_moduli, 2, n, m), dtype=torch.int8, device=A.device)
    E = torch.empty(m, dtype=torch.int32, device=A.device)
    F = torch.empty(n, dtype=torch.int32, device=A.device)
    _check(_L.zgemm_2m_residues_ex(m, n, k, A.data_ptr(), _ld(A), B.data_ptr(), _ld(B), n_moduli,
                                   _rule(scaling), res.data_ptr(), E.data_ptr(), F.data_ptr(),
                                   _stream(stream)), "zgemm_2m_residues")
    return res, E, F


def moduli(n_moduli: int):
    """(moduli, roots of -1, log2 M) of the first n_moduli 2M moduli (host only)."""
    ms = (ctypes.c_int32 * n_moduli)()
    ss = (ctypes.c_int32 * n_moduli)()
    l2 = ctypes.c_double()
    _check(_L.o2m_moduli(n_moduli, ctypes.addressof(ms), ctypes.addressof(ss), ctypes.addressof(l2)),
           "o2m_moduli")
    return list(ms), list(ss), l2.value


def budget(n_moduli: int, k: int) -> int:
    P = ctypes.c_int()
    _check(_L.o2m_budget(n_moduli, k, ctypes.addressof(P)), "o2m_budget")
    return P.value


def shifts(op: str, n_moduli: int, k: int, scaling: str = "max") -> tuple[int, int]:
    """Quantization shifts (pA, pB) a call of kind op ('z', 'c', 'h', 's', 'x'
    zher2k, 'y' dsyr2k, 'r') with inner dimension k uses (host only)."""
    pA, pB = ctypes.c_int(), ctypes.c_int()
    _check(_L.o2m_shifts(op.encode()[:1], n_moduli, k, _rule(scaling), ctypes.addressof(pA),
                         ctypes.addressof(pB)), "o2m_shifts")
    return pA.value, pB.value


def workspace_bytes(op: str, m: int, n: int, k: int, n_moduli: int) -> int:
    return int(_L.o2m_workspace_bytes(op.encode()[:1], m, n, k, n_moduli))


# caller workspaces bound to (device, stream): held here so that their memory
# stays allocated while the library may write into it
_workspaces: dict = {}


def set_workspace(buf: torch.Tensor | None, stream=None) -> None:
    """Bind a caller-owned device buffer (contiguous, on the current device) as
    the workspace of the calls on ``stream`` (default: the current stream);
    None returns the stream to library-managed memory.  The binding keeps a
    reference to ``buf`` until it is replaced or cleared."""
    dev = torch.cuda.current_device()
    handle = _stream(stream)
    if buf is None:
        _check(_L.o2m_set_workspace(None, 0, handle), "o2m_set_workspace")
        _workspaces.pop((dev, handle), None)
        return
    if not buf.is_cuda or buf.device.index != dev:
        raise ValueError(f"workspace must be a tensor on the current device cuda:{dev}")
    if not buf.is_contiguous():
        raise ValueError("workspace must be contiguous")
    _check(_L.o2m_set_workspace(buf.data_ptr(), buf.numel() * buf.element_size(), handle), "o2m_set_workspace")
    _workspaces[(dev, handle)] = buf


def release_workspace(stream=None) -> None:
    """Free the library-owned workspace of ``stream`` on the current device."""
    _check(_L.o2m_release_workspace(_stream(stream)), "o2m_release_workspace")


def get_status(stream=None) -> int:
    st = ctypes.c_int()
    _check(_L.o2m_get_status(_stream(stream), ctypes.addressof(st)), "o2m_get_status")
    return st.value


def phase_timing(enable: bool) -> None:
    _check(_L.o2m_phase_timing(1 if enable else 0), "o2m_phase_timing")


PHASES = ("scale", "residues", "int8_gemm", "crt")


def phase_times() -> dict:
    """Mean milliseconds per phase over the calls since phase_timing(True)."""
    buf = (ctypes.c_float * 4)()
    n = _L.o2m_phase_times(ctypes.addressof(buf), 4)
    if n < 0:
        raise RuntimeError("o2m_phase_times failed")
    return {PHASES[i]: float(buf[i]) for i in range(n)}
