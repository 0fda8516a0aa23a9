"""Pins of the oracle's second scaling rule (Cauchy-Schwarz) and of its rank-2k
updates (HER2K / SYR2K, Section 5) against exact rationals, closed forms,
brute force over small integers and the Cauchy-Schwarz inequality (no GPU)."""
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle as O
import workloads as W
from conftest import same_bits


def _norm2_sq(row) -> Fraction:
    """Exact squared 2-norm of a complex vector."""
    return sum(Fraction(float(v.real)) ** 2 + Fraction(float(v.imag)) ** 2 for v in row)


def _edge_matrix(rng, rows, cols):
    """Rows with wide spreads, subnormals, exact powers of two and zeros."""
    a = (rng.standard_normal((rows, cols)) + 1j * rng.standard_normal((rows, cols)))
    a *= np.exp(3.0 * rng.standard_normal((rows, cols)))
    a[0, :] = 0.0                                   # zero row
    a[1, :] = 0.0
    a[1, 0] = 2.0 ** -1070 + 0j                     # lone subnormal
    a[2, :] = 2.0 ** 40                             # equal powers of two, real parts only
    a[3, ::2] = 1e300 + 1e-300j                     # huge next to tiny
    a[4, :] *= 2.0 ** -1000                         # scaled into the subnormal range in part
    a[5, :] = 0.0
    a[5, 0] = 3.0 - 0.5j
    return np.asfortranarray(a)


# ----------------------------------------------------------- exponent rule


def test_cs_exponent_matches_exact_rationals():
    rng = np.random.default_rng(7)
    a = _edge_matrix(rng, 9, 13)
    b = np.asfortranarray(_edge_matrix(rng, 9, 13).T.copy())   # 13 x 9: columns are the edge vectors
    E, Eb, F, Fb = O.exponents(a, b, "cs")
    assert not Eb.any() and not Fb.any()
    for i in range(a.shape[0]):
        assert E[i] == O.cs_exponent_exact(a[i, :]), i
    for j in range(b.shape[1]):
        assert F[j] == O.cs_exponent_exact(b[:, j]), j


def test_cs_exponent_bounds_the_norm_within_one_bit():
    # ||a_i||_2 <= 2^G (the bound the rule exists for) and ||a_i||_2 > 2^(G-1)
    # up to the 2^-20 resolution of the integer sum of squares
    rng = np.random.default_rng(8)
    for spread in (0.0, 1.0, 4.0):
        a = rng.standard_normal((20, 37)) + 1j * rng.standard_normal((20, 37))
        a = np.asfortranarray(a * np.exp(spread * rng.standard_normal(a.shape)))
        E, _, _, _ = O.exponents(a, np.zeros((37, 1), complex), "cs")
        for i in range(a.shape[0]):
            n2 = _norm2_sq(a[i, :])
            G = int(E[i])
            assert n2 <= Fraction(4) ** G
            assert n2 > Fraction(4) ** (G - 1) * Fraction(63, 64) ** 2


def test_cs_exponent_closed_forms():
    # 4^j equal entries 2^e: the norm is exactly 2^(e+j), so G = e + j
    for e in (-30, 0, 7, 500):
        for j in (0, 1, 3):
            row = np.full((1, 4 ** j), 2.0 ** e, dtype=complex)
            E, _, _, _ = O.exponents(np.asfortranarray(row), np.zeros((4 ** j, 1), complex), "cs")
            assert E[0] == e + j
    # one nonzero part x: G = the smallest g with |x| <= 2^g
    for x in (3.0, 0.75, 1.0 + 2.0 ** -52, 2.0 ** 20, 2.0 ** -1060, 5e-310, 1.5e308):
        f, e = math.frexp(x)
        want = e - 1 if f == 0.5 else e
        row = np.zeros((1, 5), complex)
        row[0, 2] = 1j * x
        E, _, _, _ = O.exponents(np.asfortranarray(row), np.zeros((5, 1), complex), "cs")
        assert E[0] == want, x
    # power-of-two scaling shifts G exactly
    rng = np.random.default_rng(9)
    a = np.asfortranarray(rng.standard_normal((6, 10)) + 1j * rng.standard_normal((6, 10)))
    z = np.zeros((10, 1), complex)
    G0 = O.exponents(a, z, "cs")[0]
    for s in (-200, -1, 1, 300):
        assert (O.exponents(np.asfortranarray(a * 2.0 ** s), z, "cs")[0] == G0 + s).all()


def test_cs_nonfinite_rows_flagged():
    a = np.asfortranarray(np.ones((3, 4), complex))
    a[1, 2] = complex(np.nan, 0.0)
    a[2, 0] = complex(0.0, np.inf)
    E, Eb, _, _ = O.exponents(a, np.zeros((4, 1), complex), "cs")
    assert list(Eb) == [False, True, True]


# ----------------------------------------------------------- budget


def test_budget_cs_hand_values():
    # N = 1: M = 241, h' = 120 - 0 = 120
    assert O.budget_cs([241], 1) == (3, 3)      # R = 1: (8+1)(8+1) = 81 <= 120
    assert O.budget_cs([241], 3) == (3, 3)      # R = 2: 10 * 10 = 100 <= 120
    assert O.budget_cs([241], 9) == (2, 3)      # R = 3: 11 * 11 = 121 > 120; 7 * 11 = 77
    assert O.budget_cs([241], 9, symmetric=True) == (2, 2)
    assert O.budget_cs([241], 8192) is None      # R = 64: (1 + 64)^2 > 120
    # N = 2: M = 56153, h' = 28076; k = 8192, R = 64: S = 14 gives 7, 7 with
    # (128 + 64)^2 = 36864 > h'; S = 13 gives 6, 7: (64 + 64)(128 + 64) = 24576
    assert O.budget_cs([241, 233], 8192) == (6, 7)
    with pytest.raises(ValueError):
        O.oq_zgemm(np.ones((2, 8192), complex), np.ones((8192, 2), complex), 1, scaling="cs")


def _quantized(x, shift_by_row):
    """Exact componentwise round-half-even of x_ik 2^shift_i (Fractions)."""
    re, im = O.exact_quantize(x, shift_by_row)
    return re, im


@pytest.mark.parametrize("N", [2, 3, 5, 16])
def test_cs_no_overflow_on_aligned_inputs(N):
    # rows of A aligned with columns of B make |c| = ||a|| ||b|| (Cauchy-Schwarz
    # is tight); the quantized norms stay within 2^q + sqrt(k/2) and the exact
    # integer product stays within (M-1)/2 - floor(M/2^32), so the CRT path
    # (modular_path) reproduces it
    ms = O.moduli_2m(N)
    M = O.product(ms)
    hp = (M - 1) // 2 - (M >> 32)
    rng = np.random.default_rng(N)
    for k in (1, 4, 7):
        if O.budget_cs(ms, k) is None:
            continue
        x = rng.standard_normal(k) + 1j * rng.standard_normal(k)
        x = x * (1 + 0.49 / np.abs(x))      # values that round away from zero often
        a = np.asfortranarray(np.vstack([x, 2.0 * x, x * 1j]))
        b = np.asfortranarray(np.vstack([np.conj(x), -np.conj(x) * 0.75]).T)
        qA, qB = O.budget_cs(ms, k)
        E = [O.cs_exponent_exact(a[i, :]) for i in range(a.shape[0])]
        F = [O.cs_exponent_exact(b[:, j]) for j in range(b.shape[1])]
        Ar, Ai = _quantized(a, [qA - e for e in E])
        Br, Bi = _quantized(np.asfortranarray(b.T), [qB - f for f in F])
        r = math.sqrt(k / 2)
        for i in range(a.shape[0]):
            assert math.sqrt(sum(v * v for v in Ar[i]) + sum(v * v for v in Ai[i])) <= 2 ** qA + r
        for j in range(b.shape[1]):
            assert math.sqrt(sum(v * v for v in Br[j]) + sum(v * v for v in Bi[j])) <= 2 ** qB + r
        for i in range(a.shape[0]):
            for j in range(b.shape[1]):
                re = sum(Ar[i][p] * Br[j][p] - Ai[i][p] * Bi[j][p] for p in range(k))
                im = sum(Ar[i][p] * Bi[j][p] + Ai[i][p] * Br[j][p] for p in range(k))
                assert abs(re) <= hp and abs(im) <= hp
        got = O.oq_zgemm(a, b, N, scaling="cs")
        assert same_bits(got, O.modular_path(a, b, N, scaling="cs"))


@pytest.mark.parametrize("N,shape,spread", [(3, (3, 5, 2), 0.0), (8, (4, 3, 3), 2.0),
                                            (16, (2, 6, 4), 5.0), (22, (3, 4, 3), 1.0)])
def test_cs_oracle_equals_modular_path(N, shape, spread):
    m, k, n = shape
    rng = np.random.default_rng(N + 100)
    a = rng.standard_normal((m, k)) + 1j * rng.standard_normal((m, k))
    b = rng.standard_normal((k, n)) + 1j * rng.standard_normal((k, n))
    a = np.asfortranarray(a * np.exp(spread * rng.standard_normal(a.shape)))
    b = np.asfortranarray(b * np.exp(spread * rng.standard_normal(b.shape)))
    assert same_bits(O.oq_zgemm(a, b, N, scaling="cs"), O.modular_path(a, b, N, scaling="cs"))


def test_cs_more_accurate_than_max_on_spread_rows():
    # rows with a few dominant entries: the 2-norm is far below sqrt(2k) max,
    # so the Cauchy-Schwarz shifts keep more bits of every entry
    m, k, n = 24, 512, 24
    a = W.complex_matrix(m, k, 11, dist="phi", phi=2.0)
    b = W.complex_matrix(k, n, 12, dist="phi", phi=2.0)
    hi, lo = O.dd_gemm(a, b)
    absab = np.abs(a) @ np.abs(b)
    for N in (10, 12, 14, 16):
        e_max = O.error_vs_reference(O.oq_zgemm(a, b, N), absab, hi, lo, k, 2.0 ** -53)
        e_cs = O.error_vs_reference(O.oq_zgemm(a, b, N, scaling="cs"), absab, hi, lo, k, 2.0 ** -53)
        assert e_cs["maxrel"] < e_max["maxrel"], (N, e_cs, e_max)
    assert e_cs["ratio"] <= 1.0


# ----------------------------------------------------------- HER2K / SYR2K


@pytest.mark.parametrize("m", [5, 13, 205, 221, 241])
def test_her2k_identity_mod_m(m):
    # Section 5: with C+ = A+ B-^T + B+ A-^T and C- = C+^T, the 2M post step
    # (eq. 2m-post) gives A B^H + B A^H mod m, for every root s
    rng = np.random.default_rng(m)
    n, k = 4, 5
    Ar, Ai, Br, Bi = (rng.integers(-300, 300, (n, k)).astype(object) for _ in range(4))
    # A B^H + B A^H by 4M with conj(B) = Br - i Bi
    r1, i1 = O.four_m(Ar, Ai, Br.T, -Bi.T)
    r2, i2 = O.four_m(Br, Bi, Ar.T, -Ai.T)
    want_re, want_im = (r1 + r2) % m, (i1 + i2) % m
    h = O.inv2(m)
    for s in O.sqrt_minus_one(m):
        Cp = O.her2k_plus_mod(Ar, Ai, Br, Bi, m, s)
        Cm = Cp.T
        assert ((h * (Cm + Cp)) % m == want_re).all()
        assert ((s * h * (Cm - Cp)) % m == want_im).all()


def test_syr2k_is_real_part_of_half_k_her2k():
    # Section 5: A B^T + B A^T = Re(Z_A Z_B^H + Z_B Z_A^H), Z_X = X1 + i X2
    rng = np.random.default_rng(3)
    n = 4
    for k in (6, 7):
        A = rng.integers(-1000, 1000, (n, k)).astype(object)
        B = rng.integers(-1000, 1000, (n, k)).astype(object)
        kc = (k + 1) // 2
        pad = np.zeros((n, 2 * kc - k), dtype=object)
        Ap, Bp = np.hstack([A, pad]), np.hstack([B, pad])
        A1, A2, B1, B2 = Ap[:, :kc], Ap[:, kc:], Bp[:, :kc], Bp[:, kc:]
        r1, _ = O.four_m(A1, A2, B1.T, -B2.T)
        r2, _ = O.four_m(B1, B2, A1.T, -A2.T)
        assert ((r1 + r2) == A.dot(B.T) + B.dot(A.T)).all()


@pytest.mark.parametrize("scaling", ["max", "cs"])
def test_oq_zher2k_exact_on_small_integers(scaling):
    # entries with few significant bits quantize exactly and the product is
    # exact in fp64, so Algorithm 1 must return A B^H + B A^H exactly
    rng = np.random.default_rng(4)
    n, k = 7, 9
    a = np.asfortranarray(rng.integers(-500, 500, (n, k)) + 1j * rng.integers(-500, 500, (n, k)))
    b = np.asfortranarray(rng.integers(-500, 500, (n, k)) + 1j * rng.integers(-500, 500, (n, k)))
    want = a @ np.conj(b).T + b @ np.conj(a).T
    got = O.oq_zher2k(a, b, 16, scaling=scaling)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("scaling", ["max", "cs"])
def test_oq_dsyr2k_exact_on_small_integers(scaling):
    rng = np.random.default_rng(5)
    n = 6
    for k in (8, 11):
        a = np.asfortranarray(rng.integers(-500, 500, (n, k)).astype(float))
        b = np.asfortranarray(rng.integers(-500, 500, (n, k)).astype(float))
        got = O.oq_dsyr2k(a, b, 16, scaling=scaling)
        assert np.array_equal(got, a @ b.T + b @ a.T)


def test_oq_zher2k_hermitian_and_accurate():
    n, k = 40, 300
    a = W.complex_matrix(n, k, 21)
    b = W.complex_matrix(n, k, 22)
    for scaling in ("max", "cs"):
        c = O.oq_zher2k(a, b, 16, scaling=scaling)
        assert np.array_equal(c, np.conj(c).T)       # sigma = tau: exactly Hermitian
        assert (np.diag(c).imag == 0).all()
        z = np.hstack([a, b])
        w = np.hstack([b, a])
        hi, lo = O.dd_gemm(z, np.asfortranarray(np.conj(w).T))
        absab = np.abs(z) @ np.abs(w).T
        e = O.error_vs_reference(c, absab, hi, lo, 2 * k, 2.0 ** -53)
        assert e["ratio"] <= 1.0, (scaling, e)
