"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (no GPU).

* The library's host code (moduli.cpp) and the header-only helpers shared by
  kernels and host (crt_round.h, cs_bounds.h, tile_schedule.h,
  sym_schedule.h) are built with g++ into tests/sanitize_host.cpp's driver:
  its step-7 rounding of limb integers is compared with the oracle's pinned
  rounding, its moduli tables with the oracle's, its Cauchy-Schwarz chunk
  brackets with the regular host build's (tests/cs_bounds_host.cpp, pinned
  against the rule's definition in tests/test_cs_bounds.py), and it checks the
  tile schedules' coverage itself.
* The C oracle (oracle/o2m_oracle.c) is built with gcc + OpenMP into
  tests/sanitize_oracle.c's driver and must give bit for bit the results of the
  regular oracle library on the same inputs.

Any sanitizer report aborts the driver (-fno-sanitize-recover=all), which
fails the test."""
import math
import os
import random
import shutil
import subprocess

import numpy as np
import pytest

import oracle as O
import workloads as W

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1", UBSAN_OPTIONS="print_stacktrace=1")


def _have(tool):
    return shutil.which(tool) is not None


pytestmark = pytest.mark.skipif(not (_have("g++") and _have("gcc")), reason="gcc / g++ not available")


@pytest.fixture(scope="module")
def host_driver(tmp_path_factory):
    exe = str(tmp_path_factory.mktemp("san") / "sanitize_host")
    csrc = os.path.join(ROOT, "paper_2609_05419_amd", "csrc")
    subprocess.run(["g++", "-std=c++17", *SAN, "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
                    "-I", os.path.join(ROOT, "include"), "-I", csrc, os.path.join(HERE, "sanitize_host.cpp"),
                    os.path.join(csrc, "moduli.cpp"), "-o", exe], check=True)
    return exe


def _limbs(c, T, rng):
    """Random non-normalized limbs with sum c_t 2^(40 t) = c and |c_t| < 2^53."""
    out, rest = [], c
    for _ in range(T - 1):
        lo = rest % (1 << 40)
        if rng.random() < 0.5:
            lo -= 1 << 40
        out.append(lo)
        rest = (rest - lo) >> 40
    out.append(rest)
    assert all(abs(x) < 1 << 53 for x in out)
    return out


def test_host_library_code_under_sanitizers(host_driver):
    rng = random.Random(17)
    cases, lines = [], []
    for _ in range(1500):
        T = rng.randint(2, 6)
        bits = 40 * (T - 1) + 12
        c = rng.randint(-(1 << bits), 1 << bits)
        if rng.random() < 0.3:   # a tie of a 24- or 53-bit significand, +-1
            p = rng.choice((24, 53))
            s = rng.randint(2, max(2, bits - p - 1))
            c = (rng.randint(1 << (p - 1), (1 << p) - 1) << s) + (1 << (s - 1)) + rng.choice((-1, 0, 1))
        f32 = rng.random() < 0.5
        emin, prec = (-126, 24) if f32 else (-1022, 53)
        n = abs(c).bit_length()
        sc = rng.choice((rng.randint(-80, 80), emin - prec + 1 - rng.randint(0, n + 1)))
        cases.append((c, sc, f32))
        lines.append(f"r {T} {sc} {int(f32)} " + " ".join(str(x) for x in _limbs(c, T, rng)))
    bcases = []
    for _ in range(3000):   # chunk records as the one-pass scan writes them (y <= 2^20, n <= 4096)
        n = rng.randint(0, 4096)
        ys = [rng.randint(1, 1 << 20) for _ in range(min(n, 8))]
        s1 = sum(ys) * n // max(1, len(ys)) if n else 0
        s2 = sum(y * y for y in ys) * n // max(1, len(ys)) if n else 0
        s2 = max(min(s2, n << 40), s1)
        bcases.append((rng.randint(0, 24), s2, s1, n, rng.randint(0, 1 << 58)))
    lines += [f"b {t} {s2} {s1} {n} {U}" for t, s2, s1, n, U in bcases]
    r = subprocess.run([host_driver], input="\n".join(lines) + "\n", capture_output=True, text=True, env=ENV)
    assert r.returncode == 0, r.stderr[-4000:]
    out = r.stdout.splitlines()
    got_b = [ln.split()[1:] for ln in out if ln.startswith("b ")]
    assert len(got_b) == len(bcases)
    ref = _cs_bounds_regular_build()
    for (t, s2, s1, n, U), (lo, hi, d) in zip(bcases, got_b):
        assert (int(lo), int(hi), int(d)) == ref(t, s2, s1, n, U)
    got = [ln for ln in out if ln.startswith("r ")]
    assert len(got) == len(cases)
    for (c, sc, f32), ln in zip(cases, got):
        want = O.round_scaled(c, sc, "f32" if f32 else "f64")
        assert int(ln.split()[1], 16) == int(np.float64(want).view(np.uint64)), (c, sc, f32)
    tables = [ln.split() for ln in out if ln.startswith("m ")]
    assert len(tables) == 32
    for t in tables:
        N, log2M, limbs, P1, P2, cs_ok, qa, qb = int(t[1]), float(t[2]), int(t[3]), int(t[4]), int(t[5]), \
            int(t[6]), int(t[7]), int(t[8])
        ms = O.moduli_set(N)
        assert [int(x) for x in t[9::2]] == ms
        assert [int(x) for x in t[10::2]] == [O.root_of(q) if O.is_2m_modulus(q) else 0 for q in ms]
        assert abs(log2M - math.log2(O.product(ms))) < 1e-6
        assert limbs == max(2, math.ceil((math.log2(O.product(ms)) + 1) / 40))
        assert (P1, P2) == (O.budget(ms, 1024), O.budget(ms, 65536))
        q = O.budget_cs(ms, 8192)
        assert bool(cs_ok) == (q is not None) and (q is None or (qa, qb) == tuple(q))
    assert any(ln.startswith("sched ") for ln in out)


def _cs_bounds_regular_build():
    """The chunk bracket and d of the regular (unsanitized) host build."""
    import ctypes
    import tempfile
    out = os.path.join(tempfile.mkdtemp(), "libcs_bounds_host.so")
    subprocess.run(["g++", "-O2", "-std=c++17", "-fPIC", "-shared", os.path.join(HERE, "cs_bounds_host.cpp"),
                    "-o", out], check=True)
    L = ctypes.CDLL(out)
    U64 = ctypes.c_uint64
    L.t_cs_d_of.argtypes = [U64]
    L.t_cs_d_of.restype = ctypes.c_int
    L.t_cs_chunk_bounds.argtypes = [ctypes.c_int, U64, U64, U64, ctypes.POINTER(U64), ctypes.POINTER(U64)]

    def f(t, s2, s1, n, U):
        lo, hi = U64(), U64()
        L.t_cs_chunk_bounds(t, s2, s1, n, ctypes.byref(lo), ctypes.byref(hi))
        return lo.value, hi.value, L.t_cs_d_of(U)
    return f


def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "sanitize_oracle")
    subprocess.run(["gcc", "-std=c11", *SAN, "-fopenmp", os.path.join(HERE, "sanitize_oracle.c"),
                    os.path.join(ROOT, "oracle", "o2m_oracle.c"), "-lm", "-o", exe], check=True)
    m, n, k, N = 23, 19, 37, 16
    a = W.complex_matrix(m, k, 5101, dist="phi", phi=2.0)
    b = W.complex_matrix(k, n, 5102, dist="phi", phi=2.0)
    a[4, :] = 0.0
    a[6, 3] = np.nan
    b[:, 2] *= 2.0 ** -1030
    ga = W.gauss_matrix(m, k, 5103, lo=-1000, hi=1000)
    gb = W.gauss_matrix(k, n, 5104, lo=-1000, hi=1000)
    for rule in ("max", "cs"):
        pA, pB = O.shifts(rule, O.moduli_set(N), k)
        inp = tmp_path / f"in_{rule}.bin"
        with open(inp, "wb") as f:
            f.write(np.array([m, n, k, pA, pB, 0 if rule == "max" else 1], dtype=np.int32).tobytes())
            f.write(np.asfortranarray(a).tobytes(order="F"))
            f.write(np.asfortranarray(b).tobytes(order="F"))
            f.write(np.ascontiguousarray(ga).tobytes())
            f.write(np.ascontiguousarray(gb).tobytes())
        outp = tmp_path / f"out_{rule}.bin"
        r = subprocess.run([exe, str(inp), str(outp)], capture_output=True, text=True,
                           env=dict(ENV, OMP_NUM_THREADS="4"))
        assert r.returncode == 0, r.stderr[-4000:]
        raw = open(outp, "rb").read()
        off = 0

        def take(dtype, count):
            nonlocal off
            x = np.frombuffer(raw, dtype=dtype, count=count, offset=off)
            off += x.nbytes
            return x

        C = take(np.complex128, m * n).reshape((n, m)).T
        C32 = take(np.complex64, m * n).reshape((n, m)).T
        hi = take(np.complex128, m * n).reshape((n, m)).T
        lo = take(np.complex128, m * n).reshape((n, m)).T
        G = take(np.int64, 2 * m * n).reshape((n, m, 2))
        E = take(np.int32, m)
        F = take(np.int32, n)
        rr = take(np.float64, 2)
        assert off == len(raw)
        same = lambda x, y: np.array_equal(np.ascontiguousarray(x).view(np.uint8), np.ascontiguousarray(y).view(np.uint8))
        assert same(C, O.oq_gemm_shifts(a, b, pA, pB, scaling=rule))
        assert same(C32, O.oq_gemm_shifts(a, b, pA, pB, scaling=rule, out_dtype=np.complex64))
        rhi, rlo = O.dd_gemm(a, b)
        assert same(hi, rhi) and same(lo, rlo)
        assert np.array_equal(G, O.gauss_4m(ga, gb))
        E0, _, F0, _ = O.exponents(a, b, rule)
        assert np.array_equal(E, E0) and np.array_equal(F, F0)
        assert rr[0] == 2.0 ** 60 + 2.0 ** 37 and rr[1] == 2.0 ** -1032 + 2.0 ** -1074
