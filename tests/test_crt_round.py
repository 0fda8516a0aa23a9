"""Host build of the CRT kernel's rounding (crt_round.h) against Python's
correctly rounded int -> float conversion: the three-term round-to-odd sum, the
multiword paths (192 and 256 bits), and the full lift with real CRT tables
built by the oracle (2M and hybrid sets)."""
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
    L.t_round_limbs.argtypes = [P, I, I]
    L.t_round_limbs.restype = D
    L.t_lift_round.argtypes = [P, I, P, D, I]
    L.t_lift_round.restype = D
    return L


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
def test_lift_round_with_crt_tables(lib, N):
    """Limb sums built the way the CRT kernel builds them (balanced base-2^40
    weights folded with 2^-1; plain weights for the 3M moduli of a hybrid set),
    lifted and rounded, equal RN of the exact symmetric lift computed with
    Python integers."""
    rng = random.Random(N)
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
    for _ in range(400):
        c = rng.randint(-bound, bound)
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
        sc = rng.randint(-60, 60)
        got = lib.t_lift_round(S.ctypes.data, T, ml.ctypes.data, inv_m, sc)
        assert got == math.ldexp(float(c), sc), (N, c)
