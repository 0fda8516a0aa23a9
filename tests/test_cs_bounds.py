"""Host build of the one-pass Cauchy-Schwarz bracket (cs_bounds.h).

The library settles the Cauchy-Schwarz exponent G = E - 20 + d of a row from
per-chunk records (S2 = sum y^2, S1 = sum y, n, with y = ceil(|v| 2^(20 - e))
against the chunk's own max exponent e), bracketing the rule's exact sum
U = sum ceil(|v| 2^(20 - E))^2 and summing again from the data only when the
bracket leaves d open.  Checked here against the definition in exact
integers: the bracket always holds U, and whenever it settles d, that d is
the definition's; d itself is the least d >= 0 with 4^d >= U.  The inputs
that leave d open (tests/cs_inputs.py) are checked to do so, and their
exponent against the oracle's exact-rational evaluation."""
import ctypes
import math
import os
import random
import subprocess

import numpy as np
import pytest

import oracle as O
from cs_inputs import exact_sum, frexp_exp, straddle_vector

HERE = os.path.dirname(os.path.abspath(__file__))
U64 = ctypes.c_uint64


@pytest.fixture(scope="module")
def lib(tmp_path_factory):
    out = tmp_path_factory.mktemp("cs") / "libcs_bounds_host.so"
    subprocess.run(["g++", "-O2", "-std=c++17", "-fPIC", "-shared", os.path.join(HERE, "cs_bounds_host.cpp"),
                    "-o", str(out)], check=True)
    L = ctypes.CDLL(str(out))
    L.t_cs_d_of.argtypes = [U64]
    L.t_cs_d_of.restype = ctypes.c_int
    L.t_cs_chunk_bounds.argtypes = [ctypes.c_int, U64, U64, U64, ctypes.POINTER(U64), ctypes.POINTER(U64)]
    return L


def d_def(U: int) -> int:
    d = 0
    while 4 ** d < U:
        d += 1
    return d


def record(parts):
    """(chunk max exponent e, S2, S1, n) of one chunk, in integers."""
    e = frexp_exp(parts)
    ys = []
    for v in parts:
        if v == 0:
            continue
        n, d = abs(float(v)).as_integer_ratio()
        if 20 - e >= 0:
            n <<= 20 - e
        else:
            d <<= e - 20
        ys.append(max(1, -((-n) // d)))
    return e, sum(y * y for y in ys), sum(ys), len(ys)


def bracket(lib, chunks):
    """(E, lo, hi) of the library's bracket over a row given as chunks of parts."""
    E = max(frexp_exp(c) for c in chunks)
    lo = hi = 0
    for c in chunks:
        e, s2, s1, n = record(c)
        if n == 0:
            continue
        l, h = U64(), U64()
        lib.t_cs_chunk_bounds(E - e, s2, s1, n, ctypes.byref(l), ctypes.byref(h))
        lo += l.value
        hi += h.value
    return E, lo, hi


def parts_of(x):
    x = np.asarray(x)
    if np.iscomplexobj(x):
        return [float(v) for pair in zip(x.real, x.imag) for v in pair]
    return [float(v) for v in x]


def test_d_of_is_the_least_power_of_four(lib):
    vals = [0, 1, 2, 3, 4, 5, 15, 16, 17, 63, 64, 65]
    for j in range(1, 30):
        vals += [4 ** j - 1, 4 ** j, 4 ** j + 1, 2 * 4 ** j]
    rng = random.Random(5)
    vals += [rng.randint(1, 1 << 62) for _ in range(2000)]
    for U in vals:
        assert lib.t_cs_d_of(U) == d_def(U), U


def test_chunk_bounds_closed_forms(lib):
    l, h = U64(), U64()
    # t = 0: the record is the share; t >= 21: every nonzero part counts 1
    lib.t_cs_chunk_bounds(0, 1234567, 999, 7, ctypes.byref(l), ctypes.byref(h))
    assert (l.value, h.value) == (1234567, 1234567)
    lib.t_cs_chunk_bounds(21, 2 ** 50, 2 ** 25, 33, ctypes.byref(l), ctypes.byref(h))
    assert (l.value, h.value) == (33, 33)
    # one part y = 2^19 + 1 one binade down: its share is ceil(y / 2)^2 = (2^18 + 1)^2
    y = 2 ** 19 + 1
    lib.t_cs_chunk_bounds(1, y * y, y, 1, ctypes.byref(l), ctypes.byref(h))
    assert l.value <= (2 ** 18 + 1) ** 2 <= h.value
    assert h.value == (2 ** 18 + 1) ** 2 and l.value == -((-y * y) // 4)
    # empty chunk
    lib.t_cs_chunk_bounds(3, 0, 0, 0, ctypes.byref(l), ctypes.byref(h))
    assert (l.value, h.value) == (0, 0)


def _random_row(rng, length, complex_):
    kind = rng.choice(["normal", "phi2", "dyadic", "edge", "sparse"])
    if kind == "normal":
        x = np.array([rng.gauss(0, 1) for _ in range(length)])
    elif kind == "phi2":
        x = np.array([(rng.random() - 0.5) * math.exp(2.0 * rng.gauss(0, 1)) for _ in range(length)])
    elif kind == "dyadic":     # small multiples of powers of two: ceilings land on integers
        x = np.array([rng.randint(-8, 8) * 2.0 ** rng.randint(-6, 2) for _ in range(length)])
    elif kind == "edge":       # values just below and at powers of two
        x = np.array([rng.choice([1.0, 1 - 2.0 ** -53, 0.5, 0.5 + 2.0 ** -30, 2.0 ** -1074, 0.0])
                      * rng.choice([1, -1]) for _ in range(length)])
    else:
        x = np.zeros(length)
        for _ in range(max(1, length // 10)):
            x[rng.randrange(length)] = rng.gauss(0, 1) * 2.0 ** rng.randint(-40, 40)
    if complex_:
        x = x + 1j * np.array([v * rng.choice([0.0, 1.0, 0.37]) for v in x[::-1]])
    return x


def test_bracket_holds_the_exact_sum_and_settles_correctly(lib):
    rng = random.Random(2024)
    settled = 0
    for it in range(400):
        length = rng.randint(1, 300)
        w = rng.choice([1, 2, 4, 8, 16, 32, 64])
        x = _random_row(rng, length, complex_=rng.random() < 0.7)
        cols = [x[c:c + w] for c in range(0, length, w)]
        chunks = [parts_of(c) for c in cols]
        parts = [v for c in chunks for v in c]
        if not any(parts):
            continue
        E, lo, hi = bracket(lib, chunks)
        U = exact_sum(parts, E)
        assert lo <= U <= hi, (it, lo, U, hi)
        if lib.t_cs_d_of(lo) == lib.t_cs_d_of(hi):
            settled += 1
            assert lib.t_cs_d_of(lo) == d_def(U)
    assert settled > 300


@pytest.mark.parametrize("kind", ["low", "high"])
@pytest.mark.parametrize("complex_", [True, False])
@pytest.mark.parametrize("w", [16, 32, 64, 128])
def test_straddle_rows_leave_d_open(lib, kind, complex_, w):
    x = straddle_vector(300, kind, complex_=complex_)
    chunks = [parts_of(x[c:c + w]) for c in range(0, len(x), w)]
    E, lo, hi = bracket(lib, chunks)
    parts = [v for c in chunks for v in c]
    U = exact_sum(parts, E)
    assert E == 1 and lo <= U <= hi
    assert lib.t_cs_d_of(lo) != lib.t_cs_d_of(hi)       # the data must be read again
    j = d_def(U)
    assert U == (4 ** (j - 1) + 1 if kind == "low" else 4 ** j)
    # and the exponent the rule gives, by the oracle's exact rationals
    vec = x if complex_ else x.astype(np.complex128)
    assert O.cs_exponent_exact(vec) == E - 20 + j


@pytest.mark.parametrize("kind", ["low", "high"])
def test_straddle_columns_leave_d_open(lib, kind):
    # column mode: chunks of 2048 entries along k
    x = straddle_vector(4200, kind, exact=(0, 2048), binade=(2048, 2112), stride=2048)
    chunks = [parts_of(x[c:c + 2048]) for c in range(0, len(x), 2048)]
    E, lo, hi = bracket(lib, chunks)
    U = exact_sum([v for c in chunks for v in c], E)
    assert lo <= U <= hi and lib.t_cs_d_of(lo) != lib.t_cs_d_of(hi)
    assert O.cs_exponent_exact(x) == E - 20 + d_def(U)


def test_straddle_vectors_are_exact_in_fp32():
    for kind in ("low", "high"):
        x = straddle_vector(300, kind)
        assert np.array_equal(x.astype(np.complex64).astype(np.complex128), x)
