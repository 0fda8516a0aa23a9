"""Pins of the oracle's number theory, 2M identities and CRT against what the
paper prints and against brute force (no GPU)."""
import math
import random

import numpy as np
import pytest

import oracle as O
from conftest import read_golden


def log2(x: int) -> float:
    return math.log2(x)


# --------------------------------------------------------------- moduli sets


def test_moduli_2m_match_printed_list():
    g = read_golden("section4_moduli.txt")
    ms = O.moduli_2m()
    assert ms[: len(g["m2m_head"])] == g["m2m_head"]
    assert ms[-len(g["m2m_tail"]):] == g["m2m_tail"]
    assert all(1 < q <= g["m2m_range_max"] for q in ms)
    assert all(math.gcd(p, q) == 1 for i, p in enumerate(ms) for q in ms[i + 1:])
    assert len(ms) == 22


def test_moduli_2m_precision_claims():
    g = read_golden("section4_moduli.txt")
    l16 = log2(O.product(O.moduli_2m(16)))
    lall = log2(O.product(O.moduli_2m()))
    assert math.floor(l16) == g["m2m_first16_log2M_approx"]
    assert math.floor(lall) == g["m2m_all_log2M_approx"]


def test_moduli_real_match_printed_list():
    g = read_golden("section4_moduli.txt")
    mr = O.moduli_real()
    assert mr[: len(g["mreal_head"])] == g["mreal_head"]
    n = g["mreal_count_for_117"]
    # 15 real moduli give the same level of accuracy as 16 2M moduli (~2^117)
    assert math.floor(log2(O.product(mr[:n]))) == g["m2m_first16_log2M_approx"]
    assert math.floor(log2(O.product(mr[: n - 1]))) < g["m2m_first16_log2M_approx"]
    assert round(log2(O.product(mr))) == g["mreal_all_log2M_approx"]


def test_2m_modulus_iff_root_of_minus_one():
    # Section 2: s with s^2 = -1 (mod m) exists iff m is a product of primes = 1 mod 4
    for m in range(3, 400, 2):
        assert O.is_2m_modulus(m) == bool(O.sqrt_minus_one(m)), m


def test_worked_example_241():
    g = read_golden("section2_identities.txt")
    m, u, v = g["m"], g["u"], g["v"]
    assert u * u + v * v == m and math.gcd(u, v) == 1
    assert (v * g["v_inverse"]) % m == 1
    assert (-u * g["v_inverse"]) % m == g["s_from_w"]
    assert O.sqrt_minus_one(m) == g["roots"]
    assert O.root_of(m) == min(g["roots"])
    assert O.inv2(m) == g["inverse_of_two"]


def test_root_from_gaussian_prime_factor():
    # Section 2.1: for prime m = u^2 + v^2, s = -u v^-1 (mod m) squares to -1
    for m in O.moduli_2m():
        roots = O.sqrt_minus_one(m)
        pf = O.prime_factors(m)
        assert len(roots) == 2 ** len(pf)           # CRT count of roots
        assert all((s * s + 1) % m == 0 for s in roots)
        assert O.inv2(m) * 2 % m == 1
        if len(pf) == 1:
            uv = [(u, v) for u in range(1, m) for v in range(1, m) if u * u + v * v == m]
            assert uv
            for u, v in uv:
                assert (-u * pow(v, -1, m)) % m in roots


# --------------------------------------------------------------- 2M identity


@pytest.mark.parametrize("shape", [(3, 4, 5), (1, 1, 1), (6, 2, 7), (4, 9, 3)])
def test_2m_equals_4m_and_3m_mod_every_modulus_and_root(shape):
    m_, k_, n_ = shape
    rng = np.random.default_rng(11 + m_ * 100 + k_ * 10 + n_)
    Ar, Ai = rng.integers(-300, 301, (2, m_, k_))
    Br, Bi = rng.integers(-300, 301, (2, k_, n_))
    c4 = O.four_m(Ar, Ai, Br, Bi)
    c3 = O.three_m(Ar, Ai, Br, Bi)
    assert (c4[0] == c3[0]).all() and (c4[1] == c3[1]).all()
    for q in O.moduli_2m():
        for s in O.sqrt_minus_one(q):
            cr, ci = O.two_m_mod(Ar, Ai, Br, Bi, q, s)
            assert ((cr - c4[0]) % q == 0).all(), (q, s)
            assert ((ci - c4[1]) % q == 0).all(), (q, s)


def test_planted_mistakes_in_2m_are_caught():
    """A wrong inverse of two or a swapped C+/C- in the imaginary part must not
    agree with 4M: the identity check above is sensitive to both."""
    rng = np.random.default_rng(5)
    Ar, Ai, Br, Bi = rng.integers(-50, 51, (4, 3, 3))
    q, s = 241, 64
    c4 = O.four_m(Ar, Ai, Br, Bi)
    Ap, Am = (Ar + s * Ai) % q, (Ar - s * Ai) % q
    Bp, Bm = (Br + s * Bi) % q, (Br - s * Bi) % q
    Cp, Cm = O._mm(Ap, Bp) % q, O._mm(Am, Bm) % q
    wrong_half = (q - 1) // 2
    assert not (((wrong_half * (Cm + Cp)) - c4[0]) % q == 0).all()
    assert not (((s * O.inv2(q) * (Cp - Cm)) - c4[1]) % q == 0).all()


def test_herk_symmetry_and_result():
    # Section 5: C- = C+^T, so one product per modulus gives A A^H mod m
    rng = np.random.default_rng(3)
    Ar, Ai = rng.integers(-100, 101, (2, 5, 7))
    ref = O.four_m(Ar, Ai, Ar.T, -Ai.T)
    for q in O.moduli_2m():
        s = O.root_of(q)
        Cp = O.herk_plus_mod(Ar, Ai, q, s)
        Cm_direct = O._mm((np.asarray(Ar, dtype=object) - s * Ai) % q,
                          ((np.asarray(Ar, dtype=object) + s * Ai) % q).T) % q
        assert (Cm_direct == Cp.T).all()
        h = O.inv2(q)
        re = (h * (Cp.T + Cp)) % q
        im = (s * h * (Cp.T - Cp)) % q
        assert ((re - ref[0]) % q == 0).all()
        assert ((im - ref[1]) % q == 0).all()
        assert (np.diag(im) == 0).all()


@pytest.mark.parametrize("k", [6, 7])
def test_syrk_is_real_part_of_half_k_herk(k):
    # Section 5: A = [A1 | A2], Z = A1 + i A2  =>  A A^T = Re(Z Z^H); odd k pads a zero column
    rng = np.random.default_rng(k)
    A = rng.integers(-100, 101, (4, k))
    Ap = np.concatenate([A, np.zeros((4, k % 2), dtype=A.dtype)], axis=1)
    kc = Ap.shape[1] // 2
    Z1, Z2 = Ap[:, :kc], Ap[:, kc:]
    re, _ = O.four_m(Z1, Z2, Z1.T, -Z2.T)
    assert (re == O._mm(A, A.T)).all()


# --------------------------------------------------------------- CRT


def test_crt_roundtrip_exhaustive_small_M():
    ms = [241, 233]
    M = O.product(ms)
    h = (M - 1) // 2
    for x in range(-h, h + 1):
        assert O.symmetric_lift(O.crt([x % q for q in ms], ms), M) == x
    # the lift maps onto exactly [-h, h]
    assert O.symmetric_lift(h + 1, M) == -h
    assert O.symmetric_lift(-h - 1, M) == h


def test_crt_roundtrip_random_all_moduli():
    rng = random.Random(7)
    for n in (1, 4, 8, 16, 22):
        ms = O.moduli_2m(n)
        M = O.product(ms)
        h = (M - 1) // 2
        for _ in range(300):
            x = rng.randint(-h, h)
            assert O.symmetric_lift(O.crt([x % q for q in ms], ms), M) == x


# --------------------------------------------------------------- scaling budget


def test_budget_is_the_largest_admissible_shift():
    for n in (1, 2, 4, 8, 16, 22):
        ms = O.moduli_2m(n)
        M = O.product(ms)
        bmax = (M - 1) // 2 - (M >> 32)
        for k in (1, 2, 3, 15, 64, 1000, 8192, 65536, 149130):
            P = O.budget(ms, k)
            lhs = lambda p: Fraction_pow(2 * k, p)
            assert lhs(P) <= bmax < lhs(P + 1), (n, k, P)


def Fraction_pow(a, p):
    from fractions import Fraction
    return Fraction(a) * Fraction(2) ** p


def test_budget_values_at_the_workload_shapes():
    assert O.budget(O.moduli_2m(16), 8192) == 102
    assert O.budget(O.moduli_2m(16), 65536) == 99
    assert O.budget(O.moduli_2m(8), 16384) == 45
    assert O.split_budget(102) == (51, 51)
    assert O.split_budget(45) == (22, 23)
    assert O.split_budget(45, symmetric=True) == (22, 22)
    assert O.split_budget(-3) == (-2, -1)
