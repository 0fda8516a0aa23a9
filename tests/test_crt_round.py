"""Host build of the CRT kernel's rounding (crt_round.h) against Python's
correctly rounded int -> float conversion and the oracle's pinned step-7
rounding: the three-term sums (to nearest and to odd), the multiword paths
(192 and 256 bits) into fp64 and fp32 with subnormal results, and the full
lift with real CRT tables built by the oracle (2M and hybrid sets)."""
import ctypes
import math
import os
import random
import subprocess

import numpy as np
import pytest

import oracle as O

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def lib(tmp_path_factory):
    out = tmp_path_factory.mktemp("crt") / "libcrt_round_host.so"
    subprocess.run(["g++", "-O2", "-std=c++20", "-fPIC", "-shared", "-ffp-contract=off",
                    os.path.join(HERE, "crt_round_host.cpp"), "-o", str(out)], check=True)
    L = ctypes.CDLL(str(out))
    D, P, I = ctypes.c_double, ctypes.c_void_p, ctypes.c_int
    L.t_sum3_rn.argtypes = [D, D, D]
    L.t_sum3_rn.restype = D
    L.t_round3_rn.argtypes = [D, D, D]
    L.t_round3_rn.restype = D
    L.t_round_limbs.argtypes = [P, I, I]
    L.t_round_limbs.restype = D
    L.t_lift_round.argtypes = [P, I, P, D, I, I]
    L.t_lift_round.restype = D
    L.t_sum3_ro.argtypes = [D, D, D]
    L.t_sum3_ro.restype = D
    L.t_sum_ro.argtypes = [D, D]
    L.t_sum_ro.restype = D
    L.t_round_limbs_fmt.argtypes = [P, I, I, I]
    L.t_round_limbs_fmt.restype = D
    L.t_round_lifted.argtypes = [P, I, I, I]
    L.t_round_lifted.restype = D
    return L


def narrow(x: float, fmt: str) -> float:
    """The oracle's fp32 rounding returns the rounded value as a double; the
    kernel's fp32 result is that value narrowed (infinite beyond fp32's range)."""
    if fmt == "f64":
        return x
    with np.errstate(over="ignore"):
        return float(np.float32(x))


def round_odd(c: int) -> float:
    """c rounded to odd with 53 bits: truncated toward zero, last bit forced
    to 1 when anything was cut off."""
    a = abs(c)
    n = a.bit_length()
    if n <= 53:
        return float(c)
    sh = n - 53
    mant = a >> sh
    if a & ((1 << sh) - 1):
        mant |= 1
    r = float(mant << sh)
    return -r if c < 0 else r


def split_limbs(c: int, T: int, rng: random.Random):
    """Random (non-normalized) limbs c_t with sum c_t 2^(40t) = c, |c_t| < 2^52."""
    limbs = []
    rest = c
    for t in range(T - 1):
        lo = rest % (1 << 40)
        if rng.random() < 0.5:
            lo -= 1 << 40
        lo += rng.randint(-(1 << 11), 1 << 11) << 40 if t + 1 < T and rng.random() < 0.3 else 0
        limbs.append(lo)
        rest = (rest - lo) >> 40
    limbs.append(rest)
    assert sum(l << (40 * t) for t, l in enumerate(limbs)) == c
    assert all(abs(l) < 1 << 53 for l in limbs)
    return limbs


def interesting_integers(rng, bits):
    vals = [0, 1, -1, (1 << 53) + 1, -((1 << 53) + 1)]
    for _ in range(3000):
        vals.append(rng.randint(-(1 << bits), 1 << bits))
    for _ in range(3000):  # exact ties and their neighbours
        s = rng.randint(1, bits - 54)
        m = rng.randint(1 << 52, (1 << 53) - 1)
        base = (m << s) + (1 << (s - 1))
        for d in (-1, 0, 1):
            v = base + d
            vals.append(v if rng.random() < 0.5 else -v)
    return vals


def test_three_term_sum_is_correctly_rounded(lib):
    rng = random.Random(3)
    for c in interesting_integers(rng, 119):
        c0, c1, c2 = split_limbs(c, 3, rng)
        got = lib.t_sum3_rn(float(c2) * 2.0 ** 80, float(c1) * 2.0 ** 40, float(c0))
        assert got == float(c), c


def three_limb_cases(rng):
    """Integers below 2^119 that stress the three-limb rounding: the generic
    mix above, exact midpoints of the 53-bit grid that are multiples of 2^40
    (where the high part alone ties) moved by a low digit in [-2^39, 2^39],
    and values around powers of two, where the gaps on the two sides differ."""
    vals = interesting_integers(rng, 119)
    for _ in range(4000):
        s = rng.randint(41, 119 - 53)
        m = rng.randint(1 << 52, (1 << 53) - 1)
        mid = (m << s) + (1 << (s - 1))
        d = rng.choice((0, 1, -1, 1 << 39, -(1 << 39), rng.randint(-(1 << 39), 1 << 39)))
        v = mid + d
        vals.append(v if rng.random() < 0.5 else -v)
    for k in range(41, 119):
        p = 1 << k
        for d in (0, 1, -1, 1 << 39, -(1 << 39), p >> 53, -(p >> 54), (p >> 53) + 1, -(p >> 54) - 1,
                  -(p >> 54) + 1, (p >> 53) - 1):
            for v in (p + d, p - (p >> 54) + d):
                vals.append(v if rng.random() < 0.5 else -v)
    return vals


def test_three_limb_rounding(lib):
    """round3_rn (the lift's rounding for three limbs) equals Python's
    correctly rounded int -> float on every case, for limbs split at random
    (carries of up to 2^11 between limbs, as the lift leaves them)."""
    rng = random.Random(5)
    for c in three_limb_cases(rng):
        for _ in range(2):
            c0, c1, c2 = split_limbs(c, 3, rng)
            got = lib.t_round3_rn(float(c0), float(c1), float(c2))
            assert got == float(c), (c, c0, c1, c2)
            assert np.float64(got).view(np.uint64) == np.float64(float(c)).view(np.uint64)


def test_three_limb_rounding_catches_a_dropped_tie_step():
    """The cases above hold inputs on which skipping the past-the-midpoint
    step (returning RN(s + d0) always) or the low-digit carry gives a wrong
    result, so the test would catch either mistake."""
    rng = random.Random(5)

    def model(c0, c1, c2, tie_step=True, carry=True):
        # the same steps on Python integers, each rounding to a double explicit
        h0 = round(c0 / 2 ** 40) if carry else 0
        d0 = c0 - h0 * 2 ** 40
        c1 = c1 + h0
        h1 = round(c1 / 2 ** 40)
        d1 = c1 - h1 * 2 ** 40
        c2 = c2 + h1
        A, B = c2 << 80, d1 << 40
        s = int(float(A + B))
        e = A + B - s
        n = int(float(s + 2 * e))
        if tie_step and n - s == 2 * e and e * d0 > 0:
            return float(n)
        return float(s + d0)

    wrong_tie = wrong_carry = 0
    for c in three_limb_cases(rng)[:20000]:
        c0, c1, c2 = split_limbs(c, 3, rng)
        assert model(c0, c1, c2) == float(c)
        wrong_tie += model(c0, c1, c2, tie_step=False) != float(c)
        wrong_carry += model(c0, c1, c2, carry=False) != float(c)
    assert wrong_tie > 0 and wrong_carry > 0


def test_three_term_sum_rounds_to_odd(lib):
    rng = random.Random(4)
    vals = interesting_integers(rng, 119)
    for _ in range(3000):   # 24-bit ties (the fp32 case) and their neighbours
        s = rng.randint(2, 119 - 25)
        m = rng.randint(1 << 23, (1 << 24) - 1)
        v = (m << s) + (1 << (s - 1)) + rng.choice((-1, 0, 1))
        vals.append(v if rng.random() < 0.5 else -v)
    for c in vals:
        c0, c1, c2 = split_limbs(c, 3, rng)
        got = lib.t_sum3_ro(float(c2) * 2.0 ** 80, float(c1) * 2.0 ** 40, float(c0))
        assert got == round_odd(c), c
        c0, c1 = split_limbs(c >> 40, 2, rng) if abs(c) < 1 << 90 else (0, 0)
        if abs(c) < 1 << 90:
            cc = c >> 40
            got = lib.t_sum_ro(float(c1) * 2.0 ** 40, float(c0))
            assert got == round_odd(cc), cc


@pytest.mark.parametrize("T,bits", [(2, 90), (3, 130), (4, 150), (5, 190), (6, 245)])
@pytest.mark.parametrize("fmt", ["f64", "f32"])
def test_multiword_rounding_into_format(lib, T, bits, fmt):
    """One rounding of c 2^sc into fp64 / fp32, subnormal results included,
    equals the oracle's pinned step-7 rounding."""
    rng = random.Random(10 * T + (fmt == "f32"))
    emin, prec = (-1022, 53) if fmt == "f64" else (-126, 24)
    for c in interesting_integers(rng, bits)[:2500]:
        limbs = split_limbs(c, T, rng)
        arr = np.array(limbs, dtype=np.int64)
        n = abs(c).bit_length()
        # normal, subnormal (quantum anywhere in c), and below half the least subnormal
        for sc in (rng.randint(-60, 60), emin - prec + 1 - rng.randint(0, n + 1), emin - n - rng.randint(0, 3)):
            got = narrow(lib.t_round_limbs_fmt(arr.ctypes.data, T, sc, int(fmt == "f32")), fmt)
            want = narrow(O.round_scaled(c, sc, fmt), fmt)
            assert np.float64(got).view(np.uint64) == np.float64(want).view(np.uint64), (c, sc, got, want)


def wild_limbs(c: int, T: int, rng: random.Random):
    """Limbs of c with |c_t| < 2^52 that are far from normalized: large limbs
    of opposite signs that cancel."""
    while True:
        limbs = [rng.randint(-(1 << 51), 1 << 51) for _ in range(T - 1)]
        top = (c - sum(l << (40 * t) for t, l in enumerate(limbs)))
        if top % (1 << (40 * (T - 1))) == 0 and abs(top >> (40 * (T - 1))) < 1 << 52:
            return limbs + [top >> (40 * (T - 1))]
        # fix the lowest limbs so that the remainder divides: adjust limb 0..T-2 exactly
        rest = c
        out = []
        for t in range(T - 1):
            lo = rest % (1 << 40) + rng.choice((0, -(1 << 40))) + (rng.randint(-(1 << 11), 1 << 11) << 40)
            out.append(lo)
            rest = (rest - lo) >> 40
        if abs(rest) < 1 << 52 and all(abs(x) < 1 << 52 for x in out):
            return out + [rest]


@pytest.mark.parametrize("T", [4, 5, 6])
@pytest.mark.parametrize("fmt", ["f64", "f32"])
def test_many_limb_rounding_via_three_terms(lib, T, fmt):
    """Four to six lifted limbs rounded through carry normalization and three
    terms (split on the top nonzero digit), against the oracle's rounding:
    values of every length, values just above and below each digit boundary
    2^(40 j) with a cancelling digit below, ties of 24- and 53-bit significands
    (+-1, exact, and with far-away low bits), small values held by large
    cancelling limbs, and subnormal results."""
    rng = random.Random(44 + 10 * T + (fmt == "f32"))
    emin, prec = (-1022, 53) if fmt == "f64" else (-126, 24)
    top = 40 * (T - 1) + 12
    vals = []
    for _ in range(1200):
        vals.append(rng.randint(-(1 << rng.randint(1, top)), 1 << rng.randint(1, top)))
    for jb in range(1, T):   # the top digit d_j = +-1 with the digit below of the opposite sign
        for _ in range(300):
            s_ = rng.choice((1, -1))
            vals.append(s_ * ((1 << (40 * jb)) - rng.randint(0, 1 << (40 * jb - 1)))
                        + rng.randint(-(1 << (40 * jb - 40)), 1 << (40 * jb - 40)))
    for _ in range(2500):
        p = rng.choice((24, 53))
        sh = rng.randint(2, top - p - 2)
        base = (rng.randint(1 << (p - 1), (1 << p) - 1) << sh) + (1 << (sh - 1))
        v = base + rng.choice((-1, 0, 1, rng.randint(-(1 << 40), 1 << 40)))
        vals.append(v if rng.random() < 0.5 else -v)
    for c in vals:
        limbs = wild_limbs(c, T, rng) if rng.random() < 0.5 else split_limbs(c, T, rng)
        arr = np.array(limbs, dtype=np.float64)
        assert sum(int(x) << (40 * t) for t, x in enumerate(limbs)) == c
        n = abs(c).bit_length()
        for sc in (rng.randint(-40, 40), emin - prec + 1 - rng.randint(0, n + 1)):
            got = lib.t_round_lifted(arr.ctypes.data, T, sc, int(fmt == "f32"))
            want = narrow(O.round_scaled(c, sc, fmt), fmt)
            assert np.float64(got).view(np.uint64) == np.float64(want).view(np.uint64), (c, limbs, sc)


@pytest.mark.parametrize("T", [2, 3, 4, 5, 6])
def test_normal_boundary_ties_round_once(lib, T):
    """c = 2^t - 2^(t-53) - 1 at 2^(-1022-t): c 2^sc lies just below 2^-1022
    and RN53(c) 2^sc = 2^-1022 - 2^-1075 ties on the subnormal grid, so the
    scaled 53-bit value rounds to 2^-1022; the one rounding of c 2^sc is the
    largest subnormal.  (Returning the scaled value whenever it is not below
    2^-1022 failed every case here.)"""
    top = 40 * T - 10
    for s in (1, -1):
        c = s * ((1 << top) - (1 << (top - 53)) - 1)
        sc = -1022 - top
        assert O.round_scaled(c, sc, "f64") == s * (2.0 ** -1022 - 2.0 ** -1074)
        rng = random.Random(T)
        limbs = split_limbs(c, T, rng)
        arr = np.array(limbs, dtype=np.float64)
        got = lib.t_round_lifted(arr.ctypes.data, T, sc, 0)
        assert np.float64(got).view(np.uint64) == np.float64(s * (2.0 ** -1022 - 2.0 ** -1074)).view(np.uint64)


@pytest.mark.parametrize("T", [2, 3, 4, 5, 6])
def test_rounding_near_format_boundaries(lib, T):
    """Values c 2^sc whose 24- or 53-bit patterns sit at or next to a tie,
    scaled to just below 2^-126, 2^-127, 2^-140, 2^-149, 2^-150 and 2^-1022
    (fp32's normal, subnormal and underflow boundaries, fp64's normal one)
    and 2^127, 2^128, 2^1023, 2^1024 (the largest binades and the overflow
    thresholds), into fp32 and fp64: one rounding each, as the oracle rounds."""
    top = 40 * T - 10
    for s in (1, -1):
        for p in (24, 53):
            for d in (-1, 0, 1, 2):
                c = s * ((1 << top) - (1 << (top - p)) + d)
                limbs = split_limbs(c, T, random.Random(top + p + d))
                arr = np.array(limbs, dtype=np.float64)
                for tgt in (-126, -127, -140, -149, -150, -1022, 127, 128, 1023, 1024):
                    for fmt in ("f32", "f64"):
                        got = lib.t_round_lifted(arr.ctypes.data, T, tgt - top, int(fmt == "f32"))
                        want = narrow(O.round_scaled(c, tgt - top, fmt), fmt)
                        assert np.float64(got).view(np.uint64) == np.float64(want).view(np.uint64), (c, tgt, fmt)


@pytest.mark.parametrize("T,bits", [(4, 150), (5, 190), (6, 245)])
def test_multiword_rounding(lib, T, bits):
    rng = random.Random(T)
    for c in interesting_integers(rng, bits):
        limbs = split_limbs(c, T, rng)
        arr = np.array(limbs, dtype=np.int64)
        for sc in (0, -1074 + 10, 200, -500):
            got = lib.t_round_limbs(arr.ctypes.data, T, sc)
            assert got == math.ldexp(float(c), sc) if c else got == 0.0, (c, sc)


@pytest.mark.parametrize("N", [4, 8, 12, 16, 17, 22, 23, 27, 28, 32])
@pytest.mark.parametrize("fmt", ["f64", "f32"])
def test_lift_round_with_crt_tables(lib, N, fmt):
    """Limb sums built the way the CRT kernel builds them (balanced base-2^40
    weights folded with 2^-1; plain weights for the 3M moduli of a hybrid set),
    lifted and rounded once into fp64 or fp32 (normal and subnormal results),
    equal the oracle's step-7 rounding of the exact symmetric lift computed
    with Python integers."""
    rng = random.Random(N + 100 * (fmt == "f32"))
    ms = O.moduli_set(N)
    M = O.product(ms)
    T = max(2, math.ceil((math.log2(M) + 1) / 40))

    def limbs(x):
        out = []
        for t in range(T - 1):
            d = x % (1 << 40)
            if d >= 1 << 39:
                d -= 1 << 40
            out.append(d)
            x = (x - d) >> 40
        out.append(x)
        return out

    W = []
    for q in ms:
        Ml = M // q
        fold = O.inv2(q) if O.is_2m_modulus(q) else 1
        g = (pow(Ml % q, -1, q) * fold) % q
        g = g - q if g > (q - 1) // 2 else g
        W.append(Ml * g)
    wl = [limbs(w) for w in W]
    ml = np.array(limbs(M), dtype=np.float64)
    h = (M - 1) // 2
    bound = h - (M >> 32)
    inv_m = 1.0 / float(M)
    emin, prec = (-1022, 53) if fmt == "f64" else (-126, 24)
    for it in range(600):
        c = rng.randint(-bound, bound)
        ps = [p for p in (24, 53) if bound.bit_length() - p - 2 >= 2]
        if it % 3 == 1 and ps:   # a tie of the output format's significand, +-1
            p = rng.choice(ps)
            s = rng.randint(2, bound.bit_length() - p - 2)
            c = (rng.randint(1 << (p - 1), (1 << p) - 1) << s) + (1 << (s - 1)) + rng.choice((-1, 0, 1))
            c = c if rng.random() < 0.5 else -c
        # residues of c mod each m, split as u = r- + r+ with symmetric parts
        u = []
        for q in ms:
            if O.is_2m_modulus(q):
                r = (c * 2) % q          # u = 2c mod q, since W folds in 2^-1
                r = r - q if r > (q - 1) // 2 else r
                rm = rng.randint(-(q - 1) // 2, (q - 1) // 2)
                rp = r - rm
                if abs(rp) > (q - 1) // 2:
                    rp = r
                    rm = 0
                u.append(rm + rp)
            else:                        # 3M: u = T1 - T2 with int8 residues
                r = c % q
                t2 = rng.randint(-(q // 2), (q - 1) // 2)
                t1 = (r + t2) % q
                t1 = t1 - q if t1 > (q - 1) // 2 else t1
                u.append(t1 - t2)
        S = np.array([sum(u[l] * wl[l][t] for l in range(N)) for t in range(T)], dtype=np.float64)
        assert all(abs(sum(u[l] * wl[l][t] for l in range(N))) < 1 << 53 for t in range(T))
        n = abs(c).bit_length()
        sc = rng.randint(-60, 60) if it % 2 == 0 else emin - prec + 1 - rng.randint(0, n + 1)
        got = lib.t_lift_round(S.ctypes.data, T, ml.ctypes.data, inv_m, sc, int(fmt == "f32"))
        want = narrow(O.round_scaled(c, sc, fmt), fmt)
        assert np.float64(got).view(np.uint64) == np.float64(want).view(np.uint64), (N, c, sc)
