"""Pins of the C oracle (exact Gaussian 4M, Algorithm 1's exact output and the
double-double reference) against Python integers, Fractions, closed forms and
the paper's error trend (no GPU)."""
import math
import random
from fractions import Fraction

import numpy as np
import pytest

import oracle as O
import workloads as W
from conftest import same_bits


def rand_complex(rng, m, n, spread=0.0):
    a = rng.standard_normal((m, n)) + 1j * rng.standard_normal((m, n))
    if spread:
        a = a * np.exp(spread * rng.standard_normal((m, n)))
    return np.asfortranarray(a)


# --------------------------------------------------------------- rounding pin


def test_integer_rounding_matches_python():
    rng = random.Random(1)
    vals = [0, 1, -1, 2 ** 53 + 1, -(2 ** 53 + 1), 2 ** 54 + 2, 2 ** 54 + 6, 2 ** 120 - 1,
            -(2 ** 126), (2 ** 53 + 1) << 40, ((2 ** 53 + 3) << 40) + (1 << 39), (1 << 100) + 1]
    vals += [rng.randint(-(2 ** 126), 2 ** 126) for _ in range(2000)]
    vals += [rng.randint(-(2 ** 60), 2 ** 60) << rng.randint(0, 60) for _ in range(2000)]
    for v in vals:
        assert O.round_i128(v) == float(v), v  # Python's int -> float is correctly rounded


# --------------------------------------------------------------- O-Z


def test_gauss_4m_against_python_integers():
    A = W.gauss_matrix(5, 7, seed=1, lo=-2 ** 31, hi=2 ** 31 - 1)
    B = W.gauss_matrix(7, 3, seed=2, lo=-2 ** 31, hi=2 ** 31 - 1)
    # products of int32 values overflow int64 sums: expect the overflow report
    with pytest.raises(OverflowError):
        O.gauss_4m(A, B)
    A = W.gauss_matrix(5, 7, seed=1, lo=-2 ** 20, hi=2 ** 20)
    B = W.gauss_matrix(7, 3, seed=2, lo=-2 ** 20, hi=2 ** 20)
    C = O.gauss_4m(A, B)
    for i in range(5):
        for j in range(3):
            re = sum(int(A[p, i, 0]) * int(B[j, p, 0]) - int(A[p, i, 1]) * int(B[j, p, 1]) for p in range(7))
            im = sum(int(A[p, i, 0]) * int(B[j, p, 1]) + int(A[p, i, 1]) * int(B[j, p, 0]) for p in range(7))
            assert (int(C[j, i, 0]), int(C[j, i, 1])) == (re, im)


def test_gauss_4m_config1_against_numpy():
    sa, sb = W.config_seeds(1)
    A = W.gauss_matrix(64, 64, sa)
    B = W.gauss_matrix(64, 64, sb)
    C = O.gauss_4m(A, B)
    a = A[..., 0].T.astype(np.int64) + 1j * 0
    Ar, Ai = A[..., 0].T.astype(np.int64), A[..., 1].T.astype(np.int64)
    Br, Bi = B[..., 0].T.astype(np.int64), B[..., 1].T.astype(np.int64)
    assert (C[..., 0].T == Ar @ Br - Ai @ Bi).all()
    assert (C[..., 1].T == Ar @ Bi + Ai @ Br).all()
    del a


# --------------------------------------------------------------- O-Q


CASES = [
    # (m, k, n, spread, n_moduli)
    (3, 4, 2, 0.0, 16),
    (4, 3, 5, 2.0, 8),
    (2, 6, 3, 6.0, 22),
    (5, 5, 4, 0.5, 1),
    (1, 1, 1, 0.0, 4),
    (3, 2, 3, 1.0, 18),
    (4, 7, 2, 3.0, 20),
]


@pytest.mark.parametrize("case", CASES)
def test_oq_equals_fractions_and_modular_path(case):
    m, k, n, spread, N = case
    rng = np.random.default_rng(sum(case[:3]) * 7 + N)
    a = rand_complex(rng, m, k, spread)
    b = rand_complex(rng, k, n, spread)
    a[0, 0] = 0.0                                   # a zero entry
    if m > 2:
        a[m - 1, :] = 0.0                           # a zero row
    pA, pB = O.split_budget(O.budget(O.moduli_2m(N), k))
    got = O.oq_zgemm(a, b, N)
    tiny = O.exact_oq_tiny(a, b, pA, pB)
    mod = O.modular_path(a, b, N)
    assert same_bits(got, tiny)
    assert same_bits(got, mod)
    ent = [(i, j) for i in range(m) for j in range(n)][::2]
    sub = O.oq_zgemm(a, b, N, entries=ent)
    assert np.array_equal(sub, np.array([got[i, j] for i, j in ent]))


def test_oq_cint_bounded_and_consistent_with_residues():
    rng = np.random.default_rng(4)
    for N in (4, 16, 22):
        a = rand_complex(rng, 6, 9, 1.0)
        b = rand_complex(rng, 9, 5, 1.0)
        ms = O.moduli_2m(N)
        M = O.product(ms)
        pA, pB = O.split_budget(O.budget(ms, 9))
        ent = [(i, j) for i in range(6) for j in range(5)]
        cint = O.oq_cint(a, b, pA, pB, ent)
        out = O.oq_gemm_shifts(a, b, pA, pB, ent)
        E, _, F, _ = O.exponents(a, b)
        for (i, j), (cr, ci), o in zip(ent, cint, out):
            assert abs(cr) <= (M - 1) // 2 and abs(ci) <= (M - 1) // 2
            sc = int(E[i] + F[j] - pA - pB)
            assert o.real == math.ldexp(float(cr), sc) and o.imag == math.ldexp(float(ci), sc)


def test_quantized_entries_within_shift_bound():
    rng = np.random.default_rng(9)
    a = rand_complex(rng, 7, 11, 4.0)
    E, _, _, _ = O.exponents(a, a.T)
    for pA in (3, 22, 51, 68):
        for i in range(7):
            x = np.rint(np.ldexp(a[i].real, pA - E[i]))
            y = np.rint(np.ldexp(a[i].imag, pA - E[i]))
            assert np.max(np.abs(x)) <= 2.0 ** pA and np.max(np.abs(y)) <= 2.0 ** pA
            amax = np.max(np.maximum(np.abs(a[i].real), np.abs(a[i].imag)))
            assert 2.0 ** (E[i] - 1) <= amax < 2.0 ** E[i]


def test_identity_times_integer_matrix_is_exact():
    # A = 4 I (power of two), B with small integer parts: every step is exact
    rng = np.random.default_rng(2)
    n = 6
    a = np.asfortranarray(4.0 * np.eye(n, dtype=np.complex128))
    b = np.asfortranarray(rng.integers(-1000, 1001, (n, 5)) + 1j * rng.integers(-1000, 1001, (n, 5)))
    for N in (8, 16, 22):
        c = O.oq_zgemm(a, b, N)
        assert np.array_equal(c, 4.0 * b)


def test_integer_inputs_match_exact_gaussian_product():
    # integer-valued inputs quantize exactly when 2^pA covers them; then O-Q = O-Z
    A = W.gauss_matrix(9, 13, seed=5, lo=-100, hi=100)
    B = W.gauss_matrix(13, 4, seed=6, lo=-100, hi=100)
    a = np.asfortranarray((A[..., 0] + 1j * A[..., 1]).T.astype(np.complex128))
    b = np.asfortranarray((B[..., 0] + 1j * B[..., 1]).T.astype(np.complex128))
    C = O.gauss_4m(A, B)
    c = O.oq_zgemm(a, b, 16)
    assert np.array_equal(c.real, C[..., 0].T.astype(np.float64))
    assert np.array_equal(c.imag, C[..., 1].T.astype(np.float64))


def test_nonfinite_rows_and_columns_give_nan():
    rng = np.random.default_rng(8)
    a = rand_complex(rng, 5, 6)
    b = rand_complex(rng, 6, 4)
    a2, b2 = a.copy(order="F"), b.copy(order="F")
    a2[2, 3] = np.nan
    b2[1, 1] = complex(np.inf, 0.0)
    c = O.oq_zgemm(a2, b2, 16)
    ref = O.oq_zgemm(a, b, 16)
    assert np.isnan(c[2, :].real).all() and np.isnan(c[:, 1].imag).all()
    keep_i = [0, 1, 3, 4]
    keep_j = [0, 2, 3]
    assert np.array_equal(c[np.ix_(keep_i, keep_j)], ref[np.ix_(keep_i, keep_j)])


def test_herk_and_syrk_oracles():
    rng = np.random.default_rng(12)
    a = rand_complex(rng, 5, 8, 1.0)
    for N in (8, 16):
        c = O.oq_zherk(a, N)
        assert np.array_equal(c, np.conj(c.T))            # Hermitian, exactly
        assert (np.diag(c).imag == 0).all()
        pA, _ = O.split_budget(O.budget(O.moduli_2m(N), 8), symmetric=True)
        tiny = O.exact_oq_tiny(a, np.asfortranarray(np.conj(a).T), pA, pA)
        assert same_bits(c, tiny)
    r = np.asfortranarray(rng.standard_normal((4, 7)))
    for N in (8, 16):
        c = O.oq_dsyrk(r, N)
        assert np.array_equal(c, c.T)
        pA, _ = O.split_budget(O.budget(O.moduli_2m(N), 4), symmetric=True)
        tiny = O.exact_oq_tiny(r.astype(np.complex128), np.asfortranarray(r.T.astype(np.complex128)), pA, pA)
        assert np.array_equal(c, tiny.real)


# --------------------------------------------------------------- O-F


def test_dd_gemm_against_fractions():
    rng = np.random.default_rng(21)
    a = rand_complex(rng, 3, 6, 3.0)
    b = rand_complex(rng, 6, 4, 3.0)
    hi, lo = O.dd_gemm(a, b)
    for i in range(3):
        for j in range(4):
            re = sum(Fraction(a[i, p].real) * Fraction(b[p, j].real) - Fraction(a[i, p].imag) * Fraction(b[p, j].imag) for p in range(6))
            im = sum(Fraction(a[i, p].real) * Fraction(b[p, j].imag) + Fraction(a[i, p].imag) * Fraction(b[p, j].real) for p in range(6))
            scale = sum(abs(a[i, p]) * abs(b[p, j]) for p in range(6))
            got_re = Fraction(hi[i, j].real) + Fraction(lo[i, j].real)
            got_im = Fraction(hi[i, j].imag) + Fraction(lo[i, j].imag)
            assert abs(float(got_re - re)) <= 6 * 2.0 ** -100 * scale
            assert abs(float(got_im - im)) <= 6 * 2.0 ** -100 * scale


def test_dd_gemm_close_to_numpy():
    rng = np.random.default_rng(22)
    a = rand_complex(rng, 20, 30)
    b = rand_complex(rng, 30, 10)
    hi, lo = O.dd_gemm(a, b)
    assert np.allclose(hi, a @ b, rtol=1e-12, atol=1e-12)


# --------------------------------------------------------------- error trend


def test_error_shrinks_with_moduli_count_and_meets_tolerance():
    """Section 3.1: the relative error behaves like M^(-1/2); each added 2M
    modulus (~7.3 bits of M) buys roughly 3.7 bits.  At N = 16 the max-rule
    result meets the tolerance 4 u k |A||B| (u = 2^-53)."""
    k = 64
    a = W.complex_matrix(48, k, seed=31)
    b = W.complex_matrix(k, 40, seed=32)
    hi, lo = O.dd_gemm(a, b)
    absab = np.abs(a) @ np.abs(b)
    errs = {}
    for N in (6, 8, 10, 12, 14, 16):
        c = O.oq_zgemm(a, b, N)
        errs[N] = O.error_vs_reference(c, absab, hi, lo, k, 2.0 ** -53)
    seq = [errs[N]["maxrel"] for N in (6, 8, 10, 12, 14)]
    assert all(x > y for x, y in zip(seq, seq[1:]))
    for N in (6, 8, 10, 12):
        bits = math.log2(errs[N]["maxrel"] / errs[N + 2]["maxrel"]) / 2.0
        assert 2.0 < bits < 6.0, (N, bits)
    assert errs[16]["ratio"] <= 1.0
    assert errs[8]["ratio"] > 1.0


def test_error_vs_reference_closed_form():
    # c - ref = (3, 4) 2^-40 exactly (a 3-4-5 triangle: modulus 5 2^-40);
    # |ref| = 5, |A||B| = 2, k = 8
    d = 2.0 ** -40
    ref_hi = np.array([3.0 + 4.0j, 0.0 + 0.0j, -6.0 + 8.0j])
    ref_lo = np.zeros(3, dtype=complex)
    c = ref_hi + np.array([3 * d + 4j * d, 0.0, 0.0])
    absab = np.array([2.0, 1.0, 1.0])
    u = 2.0 ** -53
    e = O.error_vs_reference(c, absab, ref_hi, ref_lo, 8, u)
    assert math.isclose(e["maxrel"], 5 * d / 5.0, rel_tol=1e-12)
    assert math.isclose(e["ratio"], 5 * d / (4 * u * 8 * 2.0), rel_tol=1e-12)
    assert math.isclose(e["maxrel_re"], 3 * d / 3.0, rel_tol=1e-12)
    assert math.isclose(e["maxrel_im"], 4 * d / 4.0, rel_tol=1e-12)
    assert e["zeros"] == 1
    # the low word of the reference counts: an error hidden in ref_lo is seen
    e2 = O.error_vs_reference(ref_hi, absab, ref_hi, np.array([1e-20, 0, 0], dtype=complex), 8, u)
    assert math.isclose(e2["maxrel"], 1e-20 / 5.0, rel_tol=1e-12)
    # an error where |A||B| is zero is an infinite ratio
    e3 = O.error_vs_reference(np.array([1e-300 + 0j]), np.array([0.0]), np.array([0j]), np.array([0j]), 8, u)
    assert e3["ratio"] == math.inf
