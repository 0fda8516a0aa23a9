"""Pins of Algorithm 1's reconstruction step (step 7) in the C oracle: the exact
scaled integer is rounded ONCE into the output format, fp64 or fp32, to
nearest with ties to even, subnormal results included.

The reference here is the definition of rounding to nearest itself, evaluated
by enumeration: the representable neighbours of the exact value (found with
numpy's nextafter on the format's own grid) are compared by exact rational
distance, and a tie goes to the neighbour with an even last significand bit.
For fp64 the correctly rounded integer division of Python is a second,
independent reference.  Values whose fp64 rounding and fp32 rounding differ
from a single rounding (double-rounding ties) are constructed by hand, and
whole CGEMM / ZGEMM calls of the oracle are checked on inputs whose exact
product is such a tie."""
import math
import random
from fractions import Fraction

import numpy as np
import pytest

import oracle as O

F32 = np.float32
F64 = np.float64


def nearest(x: Fraction, ftype) -> float:
    """Round-to-nearest-even of the exact x into ftype by enumerating the
    neighbouring representable values (no floating-point arithmetic on x)."""
    if x == 0:
        return 0.0
    neg = x < 0
    ax = -x if neg else x
    info = np.finfo(ftype)
    top = Fraction(float(info.max))
    ulp_top = top - Fraction(float(np.nextafter(info.max, ftype(0))))
    if ax >= top + ulp_top / 2:
        return -np.inf if neg else np.inf
    # a starting point within a few ulps (ftype(float) may round twice or
    # saturate: the neighbours below and above cover that)
    f = ftype(min(float(ax), float(info.max)))
    cands = {f}
    for _ in range(3):
        cands |= {np.nextafter(c, ftype(np.inf)) for c in cands} | {np.nextafter(c, ftype(0)) for c in cands}
    cands = [c for c in cands if np.isfinite(c)]
    best = min(abs(Fraction(float(c)) - ax) for c in cands)
    near = [c for c in cands if abs(Fraction(float(c)) - ax) == best]
    assert 1 <= len(near) <= 2
    if len(near) == 2:   # tie: the even significand
        ibits = np.uint32 if ftype == F32 else np.uint64
        near = [c for c in near if int(np.array(c, dtype=ftype).view(ibits)) & 1 == 0]
    r = float(near[0])
    return -r if neg else r


def exact(v: int, scale: int) -> Fraction:
    return Fraction(v) * Fraction(2) ** scale


def python_f64(v: int, scale: int) -> float:
    """CPython's correctly rounded int -> float and int / int (subnormals
    included)."""
    try:
        return float(v << scale) if scale >= 0 else v / (1 << -scale)
    except OverflowError:
        return np.inf if v > 0 else -np.inf


def same(x: float, y: float) -> bool:
    return np.array(x, dtype=F64).view(np.uint64) == np.array(y, dtype=F64).view(np.uint64)


# ------------------------------------------------------------ hand-worked ties


def test_fp32_double_rounding_ties_by_hand():
    # c = 2^60 + 2^36 + 1: fp64 drops the +1, the remainder 2^36 is then half
    # an fp32 ulp (2^37) and ties to even (down); one rounding goes up.
    c = (1 << 60) + (1 << 36) + 1
    assert float(F32(float(c))) == 2.0 ** 60                      # twice rounded
    assert O.round_scaled(c, 0, "f32") == 2.0 ** 60 + 2.0 ** 37   # once
    c = -((1 << 58) + (1 << 34) + 3)
    assert float(F32(float(c))) == -(2.0 ** 58)
    assert O.round_scaled(c, 0, "f32") == -(2.0 ** 58 + 2.0 ** 35)
    # an exact tie with nothing below stays a tie: to even
    assert O.round_scaled((1 << 60) + (1 << 36), 0, "f32") == 2.0 ** 60
    assert O.round_scaled((1 << 60) + (3 << 36), 0, "f32") == 2.0 ** 60 + 2.0 ** 38


def test_fp64_subnormal_single_rounding_by_hand():
    # v 2^-1122 with v = 2^90 + 2^47 + 1: the subnormal quantum 2^-1074 is
    # bit 48 of v.  Through a 53-bit value first the +1 is lost and the tie
    # goes to even (2^-1032); rounded once it goes up.
    v = (1 << 90) + (1 << 47) + 1
    assert math.ldexp(float(v), -1122) == 2.0 ** -1032            # twice rounded
    assert O.round_scaled(v, -1122, "f64") == 2.0 ** -1032 + 2.0 ** -1074
    assert O.round_scaled(-v, -1122, "f64") == -(2.0 ** -1032 + 2.0 ** -1074)
    # below half the least subnormal: a signed zero
    assert same(O.round_scaled(1, -1076, "f64"), 0.0)
    assert same(O.round_scaled(-1, -1076, "f64"), -0.0)
    assert O.round_scaled(3, -1076, "f64") == 2.0 ** -1074        # 3/4 of it: up
    assert O.round_scaled(1, -1075, "f64") == 0.0                 # exact half: to even
    assert O.round_scaled(3, -1075, "f64") == 2.0 ** -1073        # 1.5: to even (2)


def test_fp32_subnormal_and_overflow_by_hand():
    assert O.round_scaled(1, -149, "f32") == 2.0 ** -149
    assert O.round_scaled(1, -150, "f32") == 0.0                  # half: to even (0)
    assert O.round_scaled(3, -151, "f32") == 2.0 ** -149
    big = (1 << 24) - 1
    assert O.round_scaled(big, 104, "f32") == float(np.finfo(F32).max)
    # 2^128 (1 - 2^-25) and above overflow; just below rounds to the maximum
    with np.errstate(over="ignore"):
        assert np.isinf(F32(O.round_scaled((1 << 25) - 1, 103, "f32")))
    assert F32(O.round_scaled((1 << 26) - 3, 102, "f32")) == np.finfo(F32).max


# ------------------------------------------------------------ random sweeps


def cases(rng, n, bits, lo_scale, hi_scale):
    out = []
    for _ in range(n):
        v = rng.randint(1, 1 << rng.randint(1, bits))
        out.append((v if rng.random() < 0.5 else -v, rng.randint(lo_scale, hi_scale)))
    for _ in range(n):   # ties of a p-bit significand and their neighbours
        p = rng.choice((24, 53))
        s = rng.randint(2, bits - p - 1)
        m = rng.randint(1 << (p - 1), (1 << p) - 1)
        base = (m << s) + (1 << (s - 1))
        d = rng.choice((-1, 0, 1, rng.randint(1, (1 << (s - 1)) - 1) if s > 1 else 0))
        out.append((base + d, rng.randint(lo_scale, hi_scale)))
    return out


def test_fp64_rounding_random_against_enumeration_and_python():
    rng = random.Random(5)
    cs = cases(rng, 1500, 200, -1300, 200)
    # also land in the subnormal range on purpose
    cs += [(v, -1074 - (abs(v).bit_length() - rng.randint(0, 60))) for v, _ in cases(rng, 600, 200, 0, 0)]
    for v, sc in cs:
        got = O.round_scaled(v, sc, "f64")
        assert same(got, python_f64(v, sc)), (v, sc)
        if abs(v).bit_length() + sc < 1020:
            assert same(got, nearest(exact(v, sc), F64)), (v, sc)


def test_fp32_rounding_random_against_enumeration():
    rng = random.Random(6)
    cs = cases(rng, 1500, 200, -400, 20)
    cs += [(v, -149 - (abs(v).bit_length() - rng.randint(0, 30))) for v, _ in cases(rng, 600, 200, 0, 0)]
    for v, sc in cs:
        if abs(v).bit_length() + sc > 130:
            continue
        with np.errstate(over="ignore"):   # beyond the fp32 range: narrows to inf
            got = float(F32(O.round_scaled(v, sc, "f32")))
        want = nearest(exact(v, sc), F32)
        assert same(got, want), (v, sc, got, want)


# ------------------------------------------------------------ whole calls


def tie_operands(pA, pB, E, F, j, k, imag=False, negate=False):
    """One row of A and one column of B (inner dimension k) whose quantized
    exact product is c = 2^L + 2^(L - j) + 1, L = pA + pB - 1, with row and
    column exponents E and F.  With j1 = j // 2, j2 = j - j1:
    a = [2^(E-1), 2^(E-1), 2^(E-1-j1), 2^(E-pA), 0...] and
    b = [2^(F-1), 2^(F-1), 2^(F-j2), 2^(F-pB), 0...] quantize to
    [2^(pA-1), 2^(pA-1), 2^(pA-1-j1), 1] and [2^(pB-1), 2^(pB-1), 2^(pB-j2), 1]."""
    j1 = j // 2
    j2 = j - j1
    assert pA - 1 >= j1 and pB >= j2
    a = np.zeros((1, k), dtype=np.complex128)
    b = np.zeros((k, 1), dtype=np.complex128)
    av = [2.0 ** (E - 1), 2.0 ** (E - 1), 2.0 ** (E - 1 - j1), 2.0 ** (E - pA)]
    bv = [2.0 ** (F - 1), 2.0 ** (F - 1), 2.0 ** (F - j2), 2.0 ** (F - pB)]
    for p in range(4):
        a[0, p] = (1j if imag else 1.0) * (-av[p] if negate else av[p])
        b[p, 0] = bv[p]
    return np.asfortranarray(a), np.asfortranarray(b)


@pytest.mark.parametrize("N,k", [(8, 4), (8, 300), (12, 64), (20, 16), (26, 8)])
@pytest.mark.parametrize("imag,negate", [(False, False), (True, True)])
def test_cgemm_oracle_rounds_ties_once(N, k, imag, negate):
    pA, pB = O.shifts("max", O.moduli_set(N), k)
    E, F, j = 2, 2, 24
    a, b = tie_operands(pA, pB, E, F, j, k, imag, negate)
    L = pA + pB - 1
    c = (1 << L) + (1 << (L - j)) + 1
    sgn = -1 if negate else 1
    ci = O.oq_cint(a, b, pA, pB, [(0, 0)])[0]
    assert ci == ((0, sgn * c) if imag else (sgn * c, 0))
    sc = E + F - pA - pB
    want = sgn * (2.0 ** (L + sc) + 2.0 ** (L - j + 1 + sc))   # RN24(c) = 2^L + 2^(L-23)
    twice = sgn * 2.0 ** (L + sc)
    got = O.oq_cgemm(a.astype(np.complex64), b.astype(np.complex64), N)[0, 0]
    part, other = (got.imag, got.real) if imag else (got.real, got.imag)
    assert float(part) == want and float(part) != twice and other == 0
    # the fp64 output of the same call rounds the same integer once into fp64
    wide = O.oq_zgemm(a, b, N)[0, 0]
    assert (wide.imag if imag else wide.real) == sgn * float(c) * 2.0 ** sc


def subnormal_f32_exponents(pA, pB, j):
    """E + F = j - 149 puts the fp32 quantum 2^-149 at bit L - j + 1 of c;
    split so that the smallest entries 2^(E-pA), 2^(F-pB) stay representable
    fp32 values (>= 2^-149)."""
    room = j + 149 - pA - pB
    assert room >= 0
    E = pA - 149 + room // 2
    return E, j - 149 - E


@pytest.mark.parametrize("N,k", [(8, 4), (16, 100), (20, 16), (23, 8)])
def test_cgemm_oracle_fp32_subnormal_tie(N, k):
    pA, pB = O.shifts("max", O.moduli_set(N), k)
    j = 20                               # result 2^(j-150) + 2^-149: subnormal for j < 24
    E, F = subnormal_f32_exponents(pA, pB, j)
    a, b = tie_operands(pA, pB, E, F, j, k)
    assert (a.astype(np.complex64) == a).all() and (b.astype(np.complex64) == b).all()
    got = O.oq_cgemm(a.astype(np.complex64), b.astype(np.complex64), N)[0, 0]
    assert float(got.real) == 2.0 ** (j - 150) + 2.0 ** -149
    assert O.oq_zgemm(a, b, N)[0, 0].astype(np.complex64).real == np.float32(2.0 ** (j - 150))


@pytest.mark.parametrize("N,k", [(8, 4), (16, 64), (22, 10), (26, 8)])
def test_zgemm_oracle_fp64_subnormal_tie(N, k):
    pA, pB = O.shifts("max", O.moduli_set(N), k)
    j = 30
    E = -522
    F = j - 1074 - E                     # E + F = j - 1074: quantum 2^-1074 at bit L - j + 1
    a, b = tie_operands(pA, pB, E, F, j, k, negate=True)
    L = pA + pB - 1
    assert O.oq_cint(a, b, pA, pB, [(0, 0)])[0] == (-((1 << L) + (1 << (L - j)) + 1), 0)
    got = O.oq_zgemm(a, b, N)[0, 0]
    assert got.real == -(2.0 ** (j - 1075) + 2.0 ** -1074) and got.imag == 0
    assert math.ldexp(-float((1 << L) + (1 << (L - j)) + 1), E + F - pA - pB) == -(2.0 ** (j - 1075))


@pytest.mark.parametrize("N", [16, 22])
@pytest.mark.parametrize("sign", [1, -1])
def test_zgemm_oracle_normal_boundary_tie(N, sign):
    """Exact product (2^57 - 17) 2^-1079 = 2^-1022 - 2^-1075 - 2^-1079: the
    nearest values are 2^-1022 - 2^-1074 (2^-1075 - 2^-1079 away) and 2^-1022
    (2^-1075 + 2^-1079 away), so the one rounding gives the largest subnormal,
    while rounding to 53 bits first ((2^53 - 1) 2^-1075, a tie on the
    subnormal grid) and then scaling would give 2^-1022."""
    a = np.array([[sign * (2 ** 53 - 1) * 2.0 ** -540, -sign * 2.0 ** -544]], dtype=np.complex128)
    b = np.array([[2.0 ** -535], [2.0 ** -535]], dtype=np.complex128)
    exact = (Fraction(a[0, 0].real) + Fraction(a[0, 1].real)) * Fraction(b[0, 0].real)
    assert exact == sign * Fraction(2 ** 57 - 17, 2 ** 1079)
    want = sign * (2.0 ** -1022 - 2.0 ** -1074)
    assert abs(exact - Fraction(want)) < abs(exact - Fraction(sign * 2.0 ** -1022))
    assert math.ldexp(sign * float(2 ** 57 - 17), -1079) == sign * 2.0 ** -1022   # the double rounding
    got = O.oq_zgemm(a, b, N)[0, 0]
    assert got.real == want and got.imag == 0


def test_cgemm_oracle_matches_enumerated_rounding_of_exact_integers():
    """Random CGEMM entries: the oracle's fp32 output is the enumerated
    nearest fp32 of the exact scaled integer product."""
    rng = np.random.default_rng(13)
    m, k, n, N = 4, 37, 3, 8
    a = np.asfortranarray((rng.standard_normal((m, k)) + 1j * rng.standard_normal((m, k))).astype(np.complex64))
    b = np.asfortranarray((rng.standard_normal((k, n)) + 1j * rng.standard_normal((k, n))).astype(np.complex64))
    c = O.oq_cgemm(a, b, N)
    assert c.dtype == np.complex64
    pA, pB = O.shifts("max", O.moduli_set(N), k)
    E, _, F, _ = O.exponents(a, b)
    ent = [(i, j) for i in range(m) for j in range(n)]
    for (i, j), (re, im) in zip(ent, O.oq_cint(a, b, pA, pB, ent)):
        sc = int(E[i]) + int(F[j]) - pA - pB
        assert float(c[i, j].real) == nearest(exact(re, sc), F32)
        assert float(c[i, j].imag) == nearest(exact(im, sc), F32)
