"""Pins of the oracle's hybrid 2M/3M moduli (Section 3.2: 3M for the moduli that
are not 2M moduli, once the 22 2M moduli are exhausted, Section 4) against
brute force, the CRT round trip and the exact modular path (no GPU)."""
import math
import random

import numpy as np
import pytest

import oracle as O
import workloads as W
from conftest import same_bits


def test_extension_is_the_greedy_continuation():
    two = O.moduli_2m()
    ext = O.moduli_extension()
    assert len(two) == 22
    assert ext[:6] == [256, 253, 251, 249, 239, 227]
    allm = two + ext
    for i, p in enumerate(allm):                       # pairwise coprime
        for q in allm[i + 1:]:
            assert math.gcd(p, q) == 1, (p, q)
    for m in range(2, 257):                            # maximal: nothing else fits
        if m not in allm:
            assert any(math.gcd(m, q) > 1 for q in allm), m
    for m in ext:                                      # 3M is needed for every one
        assert not O.is_2m_modulus(m)
        assert O.sqrt_minus_one(m) == [] or m % 2 == 0
    assert O.moduli_set(22) == two and O.moduli_set(25) == two + ext[:3]
    assert O.moduli_set(7) == two[:7]


@pytest.mark.parametrize("m", [256, 253, 251, 249, 239, 217, 127])
def test_three_m_mod_equals_four_m(m):
    rng = np.random.default_rng(m)
    for _ in range(4):
        Ar, Ai, Br, Bi = (rng.integers(-10 ** 6, 10 ** 6, s).astype(object)
                          for s in ((3, 4), (3, 4), (4, 5), (4, 5)))
        re, im = O.four_m(Ar, Ai, Br, Bi)
        got_re, got_im = O.three_m_mod(Ar, Ai, Br, Bi, m)
        assert ((re - got_re) % m == 0).all() and ((im - got_im) % m == 0).all()


def test_crt_round_trip_hybrid():
    rnd = random.Random(5)
    for N in (23, 28, 32):
        ms = O.moduli_set(N)
        M = O.product(ms)
        h = (M - 1) // 2
        for v in [0, 1, -1, h, -h] + [rnd.randint(-h, h) for _ in range(200)]:
            assert O.symmetric_lift(O.crt([v % q for q in ms], ms), M) == v


@pytest.mark.parametrize("N,shape,spread", [(23, (3, 5, 2), 1.0), (26, (4, 3, 3), 4.0),
                                            (32, (2, 6, 4), 8.0), (29, (3, 4, 3), 0.0)])
def test_hybrid_oracle_equals_modular_path(N, shape, spread):
    m, k, n = shape
    rng = np.random.default_rng(N)
    a = rng.standard_normal((m, k)) + 1j * rng.standard_normal((m, k))
    b = rng.standard_normal((k, n)) + 1j * rng.standard_normal((k, n))
    a = np.asfortranarray(a * np.exp(spread * rng.standard_normal(a.shape)))
    b = np.asfortranarray(b * np.exp(spread * rng.standard_normal(b.shape)))
    for rule in ("max", "cs"):
        assert same_bits(O.oq_zgemm(a, b, N, scaling=rule), O.modular_path(a, b, N, scaling=rule)), rule


def test_hybrid_moduli_recover_a_wide_exponent_span():
    # every row of A holds one entry 2^40 times its others, facing a zero row of
    # B: the product only sees the small entries, which the scale of the large
    # one leaves few bits under 22 moduli; the 3M extension restores them
    m, k, n = 12, 128, 12
    a = W.complex_matrix(m, k, 31)
    b = W.complex_matrix(k, n, 32)
    a[:, 0] = 2.0 ** 40
    b[0, :] = 0.0
    hi, lo = O.dd_gemm(a, b)
    absab = np.abs(a) @ np.abs(b)
    err = {N: O.error_vs_reference(O.oq_zgemm(a, b, N), absab, hi, lo, k, 2.0 ** -53) for N in (22, 26, 30, 32)}
    assert err[22]["ratio"] > 1.0
    assert err[30]["ratio"] <= 1.0 and err[32]["ratio"] <= 1.0
    assert err[22]["maxrel"] > err[26]["maxrel"] > err[30]["maxrel"]
