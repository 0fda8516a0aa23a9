"""Seeded synthetic inputs for the 2M + Ozaki-II complex GEMM workloads.

This module only draws random numbers; it holds none of the method's
arithmetic.  Both the CPU oracle tests and the GPU path read the arrays it
returns, so the two sides always see bit-identical inputs.

The paper measures on synthetic data only (Section 6: Uchino et al.'s
distribution with parameter phi for the accuracy study, square problems for
the performance sweeps).  The recipes here follow that:

* ``normal``   real and imaginary parts i.i.d. N(0, 1)
* ``uniform``  real and imaginary parts i.i.d. U(-1, 1)
* ``phi``      each part is u * exp(phi * g) with u ~ U(-0.5, 0.5) and
               g ~ N(0, 1) drawn independently (Section 6, phi in {0.5, 2})
* ``gauss``    Gaussian-integer matrices, parts uniform integers in [lo, hi]

Layout: every matrix is returned as a numpy array in Fortran (column-major)
order, complex interleaved (re, im), which is the layout the C-ABI takes.
Draw order is fixed: the full real plane first, then the full imaginary
plane; each plane is drawn as a C-order array of shape (cols, rows) and read
as column-major rows x cols.  For ``phi`` the uniform plane is drawn before
the normal plane, per part.
"""
from __future__ import annotations

import numpy as np

__all__ = ["complex_matrix", "real_matrix", "gauss_matrix", "config_seeds", "CONFIGS"]


def _plane(rng: np.random.Generator, rows: int, cols: int, dist: str, phi: float) -> np.ndarray:
    shape = (cols, rows)
    if dist == "normal":
        p = rng.standard_normal(shape)
    elif dist == "uniform":
        p = rng.uniform(-1.0, 1.0, shape)
    elif dist == "phi":
        u = rng.uniform(-0.5, 0.5, shape)
        g = rng.standard_normal(shape)
        p = u * np.exp(phi * g)
    else:
        raise ValueError(f"unknown distribution {dist!r}")
    return p.T  # (rows, cols) view, Fortran-contiguous


def complex_matrix(rows: int, cols: int, seed: int, dist: str = "normal", phi: float = 0.5,
                   dtype=np.complex128) -> np.ndarray:
    """rows x cols complex matrix, column-major, seeded with PCG64(seed)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    out = np.empty((rows, cols), dtype=np.complex128, order="F")
    out.real = _plane(rng, rows, cols, dist, phi)
    out.imag = _plane(rng, rows, cols, dist, phi)
    if dtype != np.complex128:
        out = np.asfortranarray(out.astype(dtype))
    return out


def real_matrix(rows: int, cols: int, seed: int, dist: str = "normal", phi: float = 0.5,
                dtype=np.float64) -> np.ndarray:
    """rows x cols real matrix, column-major."""
    rng = np.random.Generator(np.random.PCG64(seed))
    out = np.asfortranarray(_plane(rng, rows, cols, dist, phi))
    return np.asfortranarray(out.astype(dtype))


def gauss_matrix(rows: int, cols: int, seed: int, lo: int = -100, hi: int = 100) -> np.ndarray:
    """rows x cols Gaussian-integer matrix as int32 (rows, cols, 2) = (re, im).

    Returned in the C-ABI layout: column-major, (re, im) interleaved, i.e. a
    Fortran-ordered complex matrix whose parts are int32.  Shape of the
    returned array is (cols, rows, 2) in C order.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    re = rng.integers(lo, hi + 1, size=(cols, rows), dtype=np.int64)
    im = rng.integers(lo, hi + 1, size=(cols, rows), dtype=np.int64)
    out = np.empty((cols, rows, 2), dtype=np.int32)
    out[..., 0] = re
    out[..., 1] = im
    return out


def config_seeds(c: int) -> tuple[int, int]:
    """Seeds of operand A and B for workload number c."""
    return 100 * c + 1, 100 * c + 2


# The workloads: shapes, distributions and moduli counts.  ``n_moduli`` is the
# count used for the throughput line; accuracy sweeps vary it.
CONFIGS = {
    1: dict(op="gauss", m=64, n=64, k=64, n_moduli=4, dist="gauss"),
    2: dict(op="zgemm", m=1024, n=1024, k=1024, n_moduli=16, dist="normal"),
    3: dict(op="zgemm", m=8192, n=8192, k=8192, n_moduli=16, dist="phi", phi=0.5),
    4: dict(op="cgemm", m=16384, n=16384, k=16384, n_moduli=8, dist="uniform"),
    5: dict(op="zherk", n=8192, k=8192, n_moduli=16, dist="normal"),
    6: dict(op="zgemm", m=4096, n=4096, k=65536, n_moduli=16, dist="normal"),
}
