"""CPU oracle for 2M + Ozaki-II complex GEMM ("The 2M Multiplication Algorithm
for Complex Matrices", Caday).

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU
baseline leg of the benchmark import this package.  The product path (the HIP
library and its Python binding) never imports, links or calls it, and this
package imports nothing from the product path.  It shares no code, tables or
constants with it: every modulus, root and weight here is derived from the
paper's definitions on its own.

Contents, each following the passage cited:

* number theory: 2M moduli (Section 2), the greedy moduli sets (Section 4),
  square roots of -1, the inverse of 2 (Section 2);
* the 2M identities over integers mod m (Section 2, eqs. 2m-pre / 2m-mul /
  2m-post), with 4M and 3M (Section 1) for cross-checks;
* the CRT with symmetric lift (Section 3.1, Algorithm 1 steps 5-6);
* the scaling rules (Algorithm 1 step 2; the paper leaves the choice open and
  points to the Ozaki-II literature): the per-row / per-column power-of-two
  max rule with its budget, and a Cauchy-Schwarz (2-norm) rule with its own
  budget;
* Algorithm 1 step by step in exact Python integers, for tiny inputs
  (``modular_path``);
* wrappers of the C oracle (o2m_oracle.c): exact Gaussian 4M, the exact output
  of Algorithm 1 (``oq_*``), and the double-double reference (``dd_gemm``).

Parity pins: every function here is checked in tests/test_oracle_*.py against
something other than itself (printed values, brute force, Fractions, closed
forms).  Nothing is "parity unpinned" except the paper's plotted accuracy
numbers, which are absent from the text.
"""
from __future__ import annotations

import ctypes
import math
import os
from fractions import Fraction

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))

# ---------------------------------------------------------------------------
# Number theory (Sections 2 and 4)
# ---------------------------------------------------------------------------


def prime_factors(m: int) -> list[int]:
    """Distinct prime factors of m > 1, by trial division."""
    out, p = [], 2
    while p * p <= m:
        if m % p == 0:
            out.append(p)
            while m % p == 0:
                m //= p
        p += 1
    if m > 1:
        out.append(m)
    return out


def is_2m_modulus(m: int) -> bool:
    """Section 2: m is a 2M modulus iff it is odd and a product of primes that
    are 1 mod 4 (exactly then some s has s^2 = -1 mod m).  m = 1 is excluded
    (it carries no information)."""
    return m > 1 and m % 2 == 1 and all(p % 4 == 1 for p in prime_factors(m))


def greedy_moduli(accept, top: int = 256) -> list[int]:
    """Section 4: scan m = top, top-1, ..., 2 and keep m when accept(m) holds and
    m is coprime to every modulus kept so far."""
    kept: list[int] = []
    for m in range(top, 1, -1):
        if accept(m) and all(math.gcd(m, q) == 1 for q in kept):
            kept.append(m)
    return kept


def moduli_2m(count: int | None = None) -> list[int]:
    """The first ``count`` moduli of the 2M set M_2M (Section 4)."""
    ms = greedy_moduli(is_2m_modulus)
    return ms if count is None else ms[:count]


def moduli_extension() -> list[int]:
    """Hybrid 2M/3M moduli (Section 3.2, Section 4): once the 2M set is
    exhausted, the greedy scan over all integers 256, 255, ..., 2 continues,
    keeping m coprime to every 2M modulus and to every extension modulus kept
    so far.  None of them is a 2M modulus (the 2M greedy already kept every
    coprime one), so each is multiplied with 3M."""
    two = moduli_2m()
    return greedy_moduli(lambda m: all(math.gcd(m, q) == 1 for q in two))


def moduli_set(count: int) -> list[int]:
    """The first ``count`` moduli of Algorithm 1: the 2M set, then (hybrid) the
    extension moduli."""
    two = moduli_2m()
    return two[:count] if count <= len(two) else two + moduli_extension()[:count - len(two)]


def moduli_real() -> list[int]:
    """The real Ozaki-II set M_real (Section 4): no 2M condition."""
    return greedy_moduli(lambda m: True)


def sqrt_minus_one(m: int) -> list[int]:
    """All s in [1, m) with s^2 = -1 (mod m), by exhaustion (Section 2)."""
    return [s for s in range(1, m) if (s * s + 1) % m == 0]


def root_of(m: int) -> int:
    """The root used everywhere: the smallest positive s with s^2 = -1 mod m.
    Any root gives the same product: -s swaps C+ and C- and eq. 2m-post is
    symmetric under that swap."""
    return sqrt_minus_one(m)[0]


def inv2(m: int) -> int:
    """Section 2: the inverse of 2 modulo odd m is (m + 1) / 2."""
    return (m + 1) // 2


def product(ms) -> int:
    out = 1
    for q in ms:
        out *= q
    return out


# ---------------------------------------------------------------------------
# Complex products of integer matrices modulo m (Sections 1 and 2)
# ---------------------------------------------------------------------------


def _mm(x, y):
    """Integer matrix product with Python ints (object arrays): exact."""
    return np.asarray(x, dtype=object).dot(np.asarray(y, dtype=object))


def four_m(Ar, Ai, Br, Bi):
    """Section 1: C = (Ar Br - Ai Bi) + i (Ar Bi + Ai Br), exact."""
    return _mm(Ar, Br) - _mm(Ai, Bi), _mm(Ar, Bi) + _mm(Ai, Br)


def three_m(Ar, Ai, Br, Bi):
    """Section 1, eq. 3m: three products, exact over the integers."""
    P1, P2 = _mm(Ar, Br), _mm(Ai, Bi)
    P3 = _mm(np.asarray(Ar, dtype=object) + Ai, np.asarray(Br, dtype=object) + Bi)
    return P1 - P2, P3 - P1 - P2


def two_m_mod(Ar, Ai, Br, Bi, m: int, s: int):
    """Section 2: the 2M multiplication modulo a 2M modulus m with root s.

    pre   A+- = Ar +- s Ai, B+- = Br +- s Bi           (mod m)   eq. 2m-pre
    mul   C+- = A+- B+-                               (mod m)   eq. 2m-mul
    post  C = 2^-1 (C- + C+) + i s 2^-1 (C- - C+)     (mod m)   eq. 2m-post
    Returns (Re C mod m, Im C mod m) with entries in [0, m).
    """
    Ar, Ai, Br, Bi = (np.asarray(x, dtype=object) for x in (Ar, Ai, Br, Bi))
    Ap, Am = (Ar + s * Ai) % m, (Ar - s * Ai) % m
    Bp, Bm = (Br + s * Bi) % m, (Br - s * Bi) % m
    Cp, Cm = _mm(Ap, Bp) % m, _mm(Am, Bm) % m
    h = inv2(m)
    return (h * (Cm + Cp)) % m, (s * h * (Cm - Cp)) % m


def three_m_mod(Ar, Ai, Br, Bi, m: int):
    """3M (Section 1) applied after reduction modulo m (Section 3.2, for the
    moduli of a hybrid set that are not 2M moduli): T1 = Ar Br, T2 = Ai Bi,
    T3 = (Ar + Ai)(Br + Bi), all mod m; Re C = T1 - T2, Im C = T3 - T1 - T2.
    Returns (Re C mod m, Im C mod m) with entries in [0, m)."""
    Ar, Ai, Br, Bi = (np.asarray(x, dtype=object) % m for x in (Ar, Ai, Br, Bi))
    T1, T2 = _mm(Ar, Br) % m, _mm(Ai, Bi) % m
    T3 = _mm((Ar + Ai) % m, (Br + Bi) % m) % m
    return (T1 - T2) % m, (T3 - T1 - T2) % m


def herk_plus_mod(Ar, Ai, m: int, s: int):
    """Section 5 (HERK): C+ = (Ar + s Ai)(Ar - s Ai)^T mod m; C- = C+^T."""
    Ar, Ai = (np.asarray(x, dtype=object) for x in (Ar, Ai))
    return _mm((Ar + s * Ai) % m, ((Ar - s * Ai) % m).T) % m


def her2k_plus_mod(Ar, Ai, Br, Bi, m: int, s: int):
    """Section 5 (HER2K, sigma = tau): the two products of C = A B^H + B A^H
    added in the residue domain, C+ = A+ B-^T + B+ A-^T (mod m) with
    X+- = Xr +- s Xi; C- = C+^T."""
    Ar, Ai, Br, Bi = (np.asarray(x, dtype=object) for x in (Ar, Ai, Br, Bi))
    Ap, Am = (Ar + s * Ai) % m, (Ar - s * Ai) % m
    Bp, Bm = (Br + s * Bi) % m, (Br - s * Bi) % m
    return (_mm(Ap, Bm.T) + _mm(Bp, Am.T)) % m


# ---------------------------------------------------------------------------
# CRT and symmetric lift (Section 3.1; Algorithm 1 steps 5-6)
# ---------------------------------------------------------------------------


def crt(residues, moduli) -> int:
    """Section 3.1: C = sum_l C_l ((M/m_l) mod m_l)^-1 (M/m_l), reduced mod M
    (the printed sum is not reduced; step 5 of Algorithm 1 wants C mod M)."""
    M = product(moduli)
    x = 0
    for r, q in zip(residues, moduli):
        Ml = M // q
        x += r * pow(Ml % q, -1, q) * Ml
    return x % M


def symmetric_lift(x: int, M: int) -> int:
    """Algorithm 1 step 6: the representative in [-M/2, M/2); M is odd, so this
    is [-(M-1)/2, (M-1)/2]."""
    x %= M
    return x - M if 2 * x >= M else x


# ---------------------------------------------------------------------------
# Scaling (Algorithm 1 step 2)
# ---------------------------------------------------------------------------


def budget(moduli, k: int) -> int:
    """Largest integer P with 2k 2^P <= (M-1)/2 - floor(M / 2^32).

    Quantized entries are bounded by 2^pA and 2^pB with pA + pB = P, so every
    |Re c|, |Im c| <= 2k 2^P stays below (M-1)/2: the CRT then recovers c
    exactly (Section 3.1).  The floor(M/2^32) margin keeps |c|/M a little away
    from 1/2 (reading documented in the design notes)."""
    M = product(moduli)
    bmax = (M - 1) // 2 - (M >> 32)
    two_k = 2 * max(int(k), 1)
    if bmax >= two_k:
        return (bmax // two_k).bit_length() - 1
    q = 1
    while (bmax << q) < two_k:
        q += 1
    return -q


def split_budget(P: int, symmetric: bool = False) -> tuple[int, int]:
    """pA = floor(P/2), pB = P - pA; HERK/SYRK use the same shift on both
    sides (sigma = tau), pA = pB = floor(P/2)."""
    pA = P // 2
    return (pA, pA) if symmetric else (pA, P - pA)


def budget_cs(moduli, k: int, symmetric: bool = False):
    """Shifts (qA, qB) of the Cauchy-Schwarz rule, or None if there are none.

    Under that rule every quantized row of A has 2-norm at most 2^qA + r and
    every quantized column of B at most 2^qB + r, where r = sqrt(k/2) bounds
    the norm of the rounding error of 2k real parts (1/2 each).  By the
    Cauchy-Schwarz inequality |Re c|, |Im c| <= |c| <= (2^qA + r)(2^qB + r),
    so the shifts are the largest S = qA + qB (qA = floor(S/2), qB = S - qA;
    symmetric: qA = qB = floor(S/2)) with (2^qA + R)(2^qB + R) <= (M-1)/2 -
    floor(M/2^32), R = ceil(sqrt(k/2)), checked in exact integers."""
    M = product(moduli)
    hp = (M - 1) // 2 - (M >> 32)
    k = max(int(k), 0)
    R = 0
    while 2 * R * R < k:
        R += 1
    for S in range(hp.bit_length() - 1, -1, -1):
        qA = S // 2
        qB = qA if symmetric else S - qA
        if ((1 << qA) + R) * ((1 << qB) + R) <= hp:
            return qA, qB
    return None


def frexp_exponent(values) -> int:
    """E with max|v| < 2^E (frexp convention); 0 when every value is zero."""
    amax = max((abs(float(v)) for v in values), default=0.0)
    if amax == 0.0:
        return 0
    return math.frexp(amax)[1]


# ---------------------------------------------------------------------------
# Exact tiny oracles (Python integers and Fractions)
# ---------------------------------------------------------------------------


def _round_half_even(q: Fraction) -> int:
    return round(q)  # Fraction.__round__ rounds ties to even


def cs_exponent_exact(values) -> int:
    """The Cauchy-Schwarz exponent G of a complex vector, in exact rationals:
    E = frexp exponent of the largest |Re|, |Im|; U = sum over every real and
    imaginary part v of ceil(|v| 2^(20-E))^2; d = smallest d >= 0 with
    4^d >= U; G = E - 20 + d (a zero vector keeps 0).  Then ||v||_2 <= 2^G."""
    vals = list(values)
    parts = [float(v.real) for v in vals] + [float(v.imag) for v in vals]
    E = frexp_exponent(parts)
    U = 0
    for v in parts:
        q = Fraction(abs(v)) * Fraction(2) ** (20 - E)
        u = -((-q.numerator) // q.denominator)   # ceil
        U += u * u
    if U == 0:
        return E
    d = 0
    while 4 ** d < U:
        d += 1
    return E - 20 + d


def exact_quantize(a: np.ndarray, shifts_by_row) -> tuple[list, list]:
    """round_Z[i](a_ik 2^shift_i), componentwise, ties to even, with Fractions."""
    rows, cols = a.shape
    re = [[_round_half_even(Fraction(float(a[i, p].real)) * Fraction(2) ** shifts_by_row[i])
           for p in range(cols)] for i in range(rows)]
    im = [[_round_half_even(Fraction(float(a[i, p].imag)) * Fraction(2) ** shifts_by_row[i])
           for p in range(cols)] for i in range(rows)]
    return re, im


def exact_oq_tiny(a: np.ndarray, b: np.ndarray, pA: int, pB: int) -> np.ndarray:
    """Algorithm 1's exact output on a tiny finite problem, with Fractions: the
    quantized 4M product, correctly rounded to fp64, times 2^(E_i+F_j-pA-pB)."""
    m, k = a.shape
    n = b.shape[1]
    E = [frexp_exponent(list(a[i, :].real) + list(a[i, :].imag)) for i in range(m)]
    F = [frexp_exponent(list(b[:, j].real) + list(b[:, j].imag)) for j in range(n)]
    Ar, Ai = exact_quantize(a, [pA - e for e in E])
    Btr, Bti = exact_quantize(b.T, [pB - f for f in F])   # rows of b^T = columns of b
    out = np.zeros((m, n), dtype=np.complex128)
    for i in range(m):
        for j in range(n):
            re = sum(Ar[i][p] * Btr[j][p] - Ai[i][p] * Bti[j][p] for p in range(k))
            im = sum(Ar[i][p] * Bti[j][p] + Ai[i][p] * Btr[j][p] for p in range(k))
            sc = E[i] + F[j] - pA - pB
            out[i, j] = complex(math.ldexp(float(re), sc), math.ldexp(float(im), sc))
    return out


def modular_path(a: np.ndarray, b: np.ndarray, n_moduli: int, scaling: str = "max") -> np.ndarray:
    """Algorithm 1 ("2M Ozaki-II") step by step, exact Python integers.

    1. first n_moduli moduli, M = product              2. sigma, tau (max or
       (2M set, then the 3M extension)                    Cauchy-Schwarz rule)
    3. quantize to Z[i]                                4. per modulus 2M pre/mul/post
                                                          (3M for extension moduli)
    5. CRT per component                               6. symmetric lift
    7. reconstruct c sigma_i tau_j
    For tiny finite inputs only."""
    ms = moduli_set(n_moduli)
    M = product(ms)
    m, k = a.shape
    n = b.shape[1]
    if scaling == "cs":
        pA, pB = budget_cs(ms, k)
        E = [cs_exponent_exact(a[i, :]) for i in range(m)]
        F = [cs_exponent_exact(b[:, j]) for j in range(n)]
    else:
        pA, pB = split_budget(budget(ms, k))
        E = [frexp_exponent(list(a[i, :].real) + list(a[i, :].imag)) for i in range(m)]
        F = [frexp_exponent(list(b[:, j].real) + list(b[:, j].imag)) for j in range(n)]
    Ar, Ai = exact_quantize(a, [pA - e for e in E])
    Btr, Bti = exact_quantize(b.T, [pB - f for f in F])
    Br = np.asarray(Btr, dtype=object).T
    Bi = np.asarray(Bti, dtype=object).T
    res_re, res_im = [], []
    for q in ms:
        if is_2m_modulus(q):
            cr, ci = two_m_mod(Ar, Ai, Br, Bi, q, root_of(q))
        else:                                   # hybrid: 3M for the extension moduli
            cr, ci = three_m_mod(Ar, Ai, Br, Bi, q)
        res_re.append(cr)
        res_im.append(ci)
    out = np.zeros((m, n), dtype=np.complex128)
    for i in range(m):
        for j in range(n):
            cre = symmetric_lift(crt([r[i, j] for r in res_re], ms), M)
            cim = symmetric_lift(crt([r[i, j] for r in res_im], ms), M)
            sc = E[i] + F[j] - pA - pB
            out[i, j] = complex(math.ldexp(float(cre), sc), math.ldexp(float(cim), sc))
    return out


# ---------------------------------------------------------------------------
# C oracle wrappers
# ---------------------------------------------------------------------------

_lib = None


def lib():
    """Load oracle/liboracle.so, building it with gcc first if it is missing."""
    global _lib
    if _lib is None:
        path = os.path.join(_HERE, "liboracle.so")
        src = os.path.join(_HERE, "o2m_oracle.c")
        if not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(src):
            from oracle.build import build
            build()
        L = ctypes.CDLL(path)
        P, I = ctypes.c_void_p, ctypes.c_int
        L.oracle_gauss_4m.argtypes = [I, I, I, P, I, P, I, P, I]
        L.oracle_gauss_4m.restype = I
        L.oracle_exponents.argtypes = [I, I, I, P, I, P, I, I, P, P, P, P]
        L.oracle_oq_gemm.argtypes = [I, I, I, P, I, P, I, I, I, I, I, P, I, I, P, P]
        L.oracle_oq_cint.argtypes = [I, I, I, P, I, P, I, I, I, I, I, P, P, P]
        L.oracle_round_i128.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
        L.oracle_round_i128.restype = ctypes.c_double
        L.oracle_round_scaled.argtypes = [P, I, I]
        L.oracle_round_scaled.restype = ctypes.c_double
        L.oracle_dd_gemm.argtypes = [I, I, I, P, I, P, I, P, P, I, I, P, P]
        L.oracle_omp_threads.restype = I
        _lib = L
    return _lib


def _fortran_c128(x: np.ndarray) -> np.ndarray:
    x = np.asarray(x)
    if x.dtype != np.complex128:
        x = x.astype(np.complex128)
    return np.asfortranarray(x)


def _entries(entries):
    if entries is None:
        return -1, None, None
    ei = np.ascontiguousarray([e[0] for e in entries], dtype=np.int32)
    ej = np.ascontiguousarray([e[1] for e in entries], dtype=np.int32)
    return len(ei), ei, ej


def _ptr(x):
    return None if x is None else x.ctypes.data


def gauss_4m(A: np.ndarray, B: np.ndarray) -> np.ndarray:
    """Exact Gaussian-integer C = AB by 4M (Section 1), int128 accumulation.

    A, B: int32 arrays in the (cols, rows, 2) C-order layout of
    workloads.gauss_matrix.  Returns int64 (n, m, 2) in the same layout."""
    A = np.ascontiguousarray(A, dtype=np.int32)
    B = np.ascontiguousarray(B, dtype=np.int32)
    k, m, _ = A.shape
    n, k2, _ = B.shape
    assert k == k2
    C = np.zeros((n, m, 2), dtype=np.int64)
    ovf = lib().oracle_gauss_4m(m, n, k, _ptr(A), m, _ptr(B), k, _ptr(C), m)
    if ovf:
        raise OverflowError(f"{ovf} output components exceed int64")
    return C


_RULES = {"max": 0, "cs": 1}


def shifts(scaling: str, moduli, k: int, symmetric: bool = False) -> tuple[int, int]:
    """Quantization shifts (pA, pB) of the max rule or the Cauchy-Schwarz rule."""
    if scaling == "cs":
        q = budget_cs(moduli, k, symmetric)
        if q is None:
            raise ValueError(f"no Cauchy-Schwarz shifts for {len(moduli)} moduli and k={k}")
        return q
    if scaling != "max":
        raise ValueError(f"unknown scaling rule {scaling!r}")
    return split_budget(budget(moduli, k), symmetric)


def exponents(a: np.ndarray, b: np.ndarray, scaling: str = "max"):
    """(E, E_nonfinite, F, F_nonfinite) of the C oracle."""
    a, b = _fortran_c128(a), _fortran_c128(b)
    m, k = a.shape
    n = b.shape[1]
    E = np.zeros(m, np.int32); Eb = np.zeros(m, np.int32)
    F = np.zeros(n, np.int32); Fb = np.zeros(n, np.int32)
    lib().oracle_exponents(m, n, k, _ptr(a), m, _ptr(b), k, _RULES[scaling], _ptr(E), _ptr(Eb),
                           _ptr(F), _ptr(Fb))
    return E, Eb.astype(bool), F, Fb.astype(bool)


def oq_gemm_shifts(a: np.ndarray, b: np.ndarray, pA: int, pB: int, entries=None,
                   scaling: str = "max", out_dtype=np.complex128) -> np.ndarray:
    """Algorithm 1's exact output for given quantization shifts (C oracle):
    each component is the exact integer product, scaled, rounded once into
    ``out_dtype`` (complex128 or complex64)."""
    a, b = _fortran_c128(a), _fortran_c128(b)
    m, k = a.shape
    k2, n = b.shape
    assert k == k2
    f32 = np.dtype(out_dtype) == np.complex64
    if not f32 and np.dtype(out_dtype) != np.complex128:
        raise ValueError(f"unsupported output type {out_dtype}")
    ne, ei, ej = _entries(entries)
    if ne < 0:
        C = np.zeros((m, n), dtype=out_dtype, order="F")
    else:
        C = np.zeros(ne, dtype=out_dtype)
    lib().oracle_oq_gemm(m, n, k, _ptr(a), m, _ptr(b), k, pA, pB, _RULES[scaling], int(f32), _ptr(C), m, ne,
                         _ptr(ei), _ptr(ej))
    return C


def oq_zgemm(a: np.ndarray, b: np.ndarray, n_moduli: int, entries=None, scaling: str = "max") -> np.ndarray:
    """ZGEMM by Algorithm 1 with the first n_moduli moduli (the 2M set, then the
    hybrid 3M extension): exact output."""
    pA, pB = shifts(scaling, moduli_set(n_moduli), a.shape[1])
    return oq_gemm_shifts(a, b, pA, pB, entries, scaling)


def oq_cgemm(a: np.ndarray, b: np.ndarray, n_moduli: int, entries=None, scaling: str = "max") -> np.ndarray:
    """CGEMM: fp32 inputs (exactly widened), the same algorithm, and step 7
    rounds the exact scaled integer once to fp32 (nearest, ties to even), not
    through an fp64 value first."""
    a = np.asarray(a).astype(np.complex128)
    b = np.asarray(b).astype(np.complex128)
    pA, pB = shifts(scaling, moduli_set(n_moduli), a.shape[1])
    return oq_gemm_shifts(a, b, pA, pB, entries, scaling, out_dtype=np.complex64)


def oq_zherk(a: np.ndarray, n_moduli: int, entries=None, scaling: str = "max") -> np.ndarray:
    """HERK C = A A^H (Section 5) through Algorithm 1 with sigma = tau: the
    exact quantized product with equal shifts on both sides.  Returns the full
    Hermitian matrix (callers take the lower triangle)."""
    k = a.shape[1]
    pA, pB = shifts(scaling, moduli_set(n_moduli), k, symmetric=True)
    return oq_gemm_shifts(a, np.asfortranarray(np.conj(a).T), pA, pB, entries, scaling)


def oq_dsyrk(a: np.ndarray, n_moduli: int, entries=None, scaling: str = "max") -> np.ndarray:
    """SYRK C = A A^T (Section 5) via Z = A1 + i A2 with half the k: the exact
    quantized product A_int A_int^T with the HERK shifts of k' = ceil(k/2)
    (A A^T = Re(Z Z^H) holds exactly for the quantized integers)."""
    k = a.shape[1]
    kc = (k + 1) // 2
    pA, pB = shifts(scaling, moduli_set(n_moduli), kc, symmetric=True)
    ac = a.astype(np.complex128)
    out = oq_gemm_shifts(ac, np.asfortranarray(ac.T), pA, pB, entries, scaling)
    return out.real.copy(order="F") if entries is None else out.real.copy()


def oq_zher2k(a: np.ndarray, b: np.ndarray, n_moduli: int, entries=None, scaling: str = "max") -> np.ndarray:
    """HER2K C = A B^H + B A^H (Section 5) with sigma = tau: row i of A and
    row i of B share one scale, so both products carry the scale
    sigma_i sigma_j and add exactly.  C = Z W^H with Z = [A | B] and
    W = [B | A] (inner dimension 2k): row j of W holds the entries of row j of
    Z, so the column exponents of W^H equal the row exponents of Z.  The exact
    quantized product with equal shifts for inner dimension 2k; returns the
    full Hermitian matrix."""
    k = a.shape[1]
    pA, pB = shifts(scaling, moduli_set(n_moduli), 2 * k, symmetric=True)
    z = np.hstack([np.asarray(a), np.asarray(b)])
    w = np.hstack([np.asarray(b), np.asarray(a)])
    return oq_gemm_shifts(z, np.asfortranarray(np.conj(w).T), pA, pB, entries, scaling)


def oq_dsyr2k(a: np.ndarray, b: np.ndarray, n_moduli: int, entries=None, scaling: str = "max") -> np.ndarray:
    """SYR2K C = A B^T + B A^T (Section 5) as the HER2K of Z_A = A1 + i A2 and
    Z_B = B1 + i B2 with k' = ceil(k/2): the exact quantized product
    [A | B] [B | A]^T with the HER2K shifts of inner dimension 2k'."""
    k = a.shape[1]
    kc = (k + 1) // 2
    pA, pB = shifts(scaling, moduli_set(n_moduli), 2 * kc, symmetric=True)
    z = np.hstack([np.asarray(a), np.asarray(b)]).astype(np.complex128)
    w = np.hstack([np.asarray(b), np.asarray(a)]).astype(np.complex128)
    out = oq_gemm_shifts(z, np.asfortranarray(w.T), pA, pB, entries, scaling)
    return out.real.copy(order="F") if entries is None else out.real.copy()


def oq_cint(a: np.ndarray, b: np.ndarray, pA: int, pB: int, entries, scaling: str = "max") -> list[tuple[int, int]]:
    """Exact integer products (Re c, Im c) of the quantized operands at the
    listed entries, as Python ints."""
    a, b = _fortran_c128(a), _fortran_c128(b)
    m, k = a.shape
    n = b.shape[1]
    ne, ei, ej = _entries(entries)
    out = np.zeros((ne, 8), dtype=np.uint64)
    lib().oracle_oq_cint(m, n, k, _ptr(a), m, _ptr(b), k, pA, pB, _RULES[scaling], ne, _ptr(ei), _ptr(ej),
                         _ptr(out))
    res = []
    for t in range(ne):
        vals = []
        for half in (0, 4):
            v = sum(int(out[t, half + w]) << (64 * w) for w in range(4))
            if v >= 1 << 255:
                v -= 1 << 256
            vals.append(v)
        res.append((vals[0], vals[1]))
    return res


def round_scaled(v: int, scale: int, fmt: str = "f64") -> float:
    """The C oracle's step-7 rounding of the integer v (|v| < 2^255) times
    2^scale into fp64 or fp32 (``fmt``), returned as a Python float."""
    if fmt not in ("f64", "f32"):
        raise ValueError(fmt)
    u = v & ((1 << 256) - 1)
    w = np.array([(u >> (64 * t)) & ((1 << 64) - 1) for t in range(4)], dtype=np.uint64)
    return lib().oracle_round_scaled(w.ctypes.data, scale, int(fmt == "f32"))


def omp_threads() -> int:
    """OpenMP threads the C oracle's parallel loops use."""
    return int(lib().oracle_omp_threads())


def round_i128(v: int) -> float:
    """The C oracle's integer -> fp64 rounding, for pins against Python."""
    u = v & ((1 << 128) - 1)
    return lib().oracle_round_i128(u & ((1 << 64) - 1), u >> 64)


def dd_gemm(a: np.ndarray, b: np.ndarray, entries=None):
    """Double-double 4M product of the unquantized inputs: (hi, lo)."""
    a, b = _fortran_c128(a), _fortran_c128(b)
    m, k = a.shape
    n = b.shape[1]
    ne, ei, ej = _entries(entries)
    if ne < 0:
        hi = np.zeros((m, n), dtype=np.complex128, order="F")
        lo = np.zeros((m, n), dtype=np.complex128, order="F")
    else:
        hi = np.zeros(ne, dtype=np.complex128)
        lo = np.zeros(ne, dtype=np.complex128)
    lib().oracle_dd_gemm(m, n, k, _ptr(a), m, _ptr(b), k, _ptr(hi), _ptr(lo), m, ne, _ptr(ei), _ptr(ej))
    return hi, lo


def error_vs_reference(c: np.ndarray, a_abs_b_abs: np.ndarray, ref_hi: np.ndarray,
                       ref_lo: np.ndarray, k: int, u: float) -> dict:
    """Error of c against the double-double reference.

    ``ratio``: max |c - ref| / (4 u k (|A||B|)_ij) with |.| the complex modulus
    (the tolerance is met when ratio <= 1); ``maxrel``: max |c - ref| / |ref|
    over ref != 0; componentwise maxima likewise."""
    err_re = (c.real - ref_hi.real) - ref_lo.real
    err_im = (c.imag - ref_hi.imag) - ref_lo.imag
    err = np.hypot(err_re, err_im)
    ref = np.abs(ref_hi)
    bound = 4.0 * u * k * a_abs_b_abs
    with np.errstate(divide="ignore", invalid="ignore"):
        ratio = np.where(bound > 0, err / bound, np.where(err > 0, np.inf, 0.0))
        rel = np.where(ref > 0, err / ref, 0.0)
        rel_re = np.where(ref_hi.real != 0, np.abs(err_re) / np.abs(ref_hi.real), 0.0)
        rel_im = np.where(ref_hi.imag != 0, np.abs(err_im) / np.abs(ref_hi.imag), 0.0)
    return dict(ratio=float(np.max(ratio)) if ratio.size else 0.0,
                maxrel=float(np.max(rel)) if rel.size else 0.0,
                maxrel_re=float(np.max(rel_re)) if rel_re.size else 0.0,
                maxrel_im=float(np.max(rel_im)) if rel_im.size else 0.0,
                zeros=int(np.sum(ref == 0)))
