"""Parity of the HIP path (through the C-ABI) with the CPU oracle.

Floating-point results are compared bit for bit with the oracle's exact output
of Algorithm 1 (the quantized product, rescaled, rounded once to the output type):
the GPU path computes that same number exactly, so any difference is a bug.
Accuracy against the unquantized product (double-double reference) is checked
separately with the tolerance 4 u k |A||B| (u = 2^-53 for ZGEMM, 2^-24 for
CGEMM)."""
import math
import os

import numpy as np
import pytest

import oracle as O
import workloads as W
from conftest import same_bits

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def o2m():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_05419_amd as lib
    return lib


DEV = "cuda:0"


def to_dev(x):
    """Host array (any order) -> device tensor with column-major storage."""
    return torch.from_numpy(np.ascontiguousarray(np.asarray(x).T)).to(DEV).t()


def host(t):
    torch.cuda.synchronize()
    return np.asfortranarray(t.cpu().numpy())


def report(name, **kw):
    print(f"[parity] {name} " + " ".join(f"{k}={v}" for k, v in kw.items()), flush=True)


# ------------------------------------------------------------------ gauss mode


def test_gauss_config1_bit_exact(o2m):
    sa, sb = W.config_seeds(1)
    A = W.gauss_matrix(64, 64, sa)
    B = W.gauss_matrix(64, 64, sb)
    ref = O.gauss_4m(A, B)
    ms, ss, _ = o2m.moduli(4)
    assert ms == [241, 233, 229, 221]
    assert all((s * s + 1) % q == 0 for q, s in zip(ms, ss))
    dA = torch.from_numpy(A).to(DEV).transpose(0, 1)
    dB = torch.from_numpy(B).to(DEV).transpose(0, 1)
    o2m.get_status()                                      # start clean
    C = o2m.gauss_gemm_2m(dA, dB, n_moduli=4)
    got = C.transpose(0, 1).cpu().numpy()
    assert o2m.get_status() == 0
    report("gauss 64^3 N=4", equal=bool(np.array_equal(got, ref)))
    assert np.array_equal(got, ref)


@pytest.mark.parametrize("shape,N,lo", [((100, 37, 77), 5, -3000), ((1, 1, 1), 1, -5), ((300, 260, 65), 8, -(2 ** 20))])
def test_gauss_ragged_bit_exact(o2m, shape, N, lo):
    m, n, k = shape
    A = W.gauss_matrix(m, k, 11, lo=lo, hi=-lo)
    B = W.gauss_matrix(k, n, 12, lo=lo, hi=-lo)
    ref = O.gauss_4m(A, B)
    C = o2m.gauss_gemm_2m(torch.from_numpy(A).to(DEV).transpose(0, 1),
                          torch.from_numpy(B).to(DEV).transpose(0, 1), n_moduli=N)
    got = C.transpose(0, 1).cpu().numpy()
    status = o2m.get_status()
    M = O.product(O.moduli_2m(N))
    need = 2 * k * max(abs(lo), abs(lo)) ** 2
    if need <= (M - 1) // 2:
        assert status == 0
        assert np.array_equal(got, ref)
    else:
        assert status & o2m.STATUS_OVERFLOW


def test_gauss_overflow_flag(o2m):
    A = W.gauss_matrix(8, 16, 1, lo=-(2 ** 30), hi=2 ** 30)
    B = W.gauss_matrix(16, 8, 2, lo=-(2 ** 30), hi=2 ** 30)
    o2m.gauss_gemm_2m(torch.from_numpy(A).to(DEV).transpose(0, 1),
                      torch.from_numpy(B).to(DEV).transpose(0, 1), n_moduli=2)
    assert o2m.get_status() & o2m.STATUS_OVERFLOW
    assert o2m.get_status() == 0   # cleared by the read


# ------------------------------------------------------------------ ZGEMM


ZCASES = [
    # m, n, k, dist, phi, N
    (64, 64, 64, "normal", 0.5, 16),
    (100, 77, 130, "phi", 0.5, 16),
    (257, 300, 200, "phi", 2.0, 16),
    (33, 290, 65, "normal", 0.5, 1),
    (128, 64, 513, "uniform", 0.5, 4),
    (70, 90, 300, "phi", 2.0, 8),
    (300, 33, 100, "normal", 0.5, 12),
    (65, 65, 1000, "phi", 0.5, 18),
    (40, 50, 96, "phi", 2.0, 20),
    (31, 47, 33, "normal", 0.5, 22),
    (5, 3, 1, "normal", 0.5, 22),
]


@pytest.mark.parametrize("case", ZCASES, ids=[f"{c[0]}x{c[1]}x{c[2]}-{c[3]}-N{c[5]}" for c in ZCASES])
def test_zgemm_bit_exact_vs_oracle(o2m, case):
    m, n, k, dist, phi, N = case
    a = W.complex_matrix(m, k, 1000 + m, dist=dist, phi=phi)
    b = W.complex_matrix(k, n, 2000 + n, dist=dist, phi=phi)
    ref = O.oq_zgemm(a, b, N)
    C = o2m.zgemm_2m(to_dev(a), to_dev(b), n_moduli=N)
    got = host(C)
    ok = same_bits(got, ref)
    report("zgemm", shape=(m, n, k), N=N, dist=dist, bitexact=ok,
           mismatches=int(np.sum(got != ref)))
    assert ok


def test_zgemm_edge_cases(o2m):
    rng = np.random.default_rng(3)
    m, n, k = 40, 36, 50
    a = W.complex_matrix(m, k, 31)
    b = W.complex_matrix(k, n, 32)
    a[3, :] = 0.0                       # zero row -> zero row of C
    b[:, 5] = 0.0                       # zero column
    a[7, :] *= 2.0 ** 900               # huge row
    a[8, :] *= 2.0 ** -1060             # subnormal row
    b[:, 9] *= 2.0 ** -600
    a[10, 4] = np.nan                   # non-finite row
    b[2, 11] = complex(np.inf, 0)       # non-finite column
    b[7, 20] = complex(0.5, np.nan)     # NaN in an imaginary part only
    a[12, :] = 2.0 ** 7                 # entries exactly at a power of two
    ref = O.oq_zgemm(a, b, 16)
    got = host(o2m.zgemm_2m(to_dev(a), to_dev(b), n_moduli=16))
    assert same_bits(got, ref)
    assert np.isnan(got[10, :]).all() and np.isnan(got[:, 11]).all() and np.isnan(got[:, 20]).all()
    assert (got[3, :][~np.isnan(got[3, :])] == 0).all()
    del rng


def test_zgemm_k_zero_and_empty(o2m):
    a = np.zeros((5, 0), dtype=np.complex128, order="F")
    b = np.zeros((0, 4), dtype=np.complex128, order="F")
    A = torch.zeros((0, 5), dtype=torch.complex128, device=DEV).t()
    B = torch.zeros((4, 0), dtype=torch.complex128, device=DEV).t()
    out = o2m.colmajor(torch.full((5, 4), 7.0 + 1j, dtype=torch.complex128, device=DEV))
    o2m.zgemm_2m(A, B, n_moduli=16, out=out)
    assert (host(out) == 0).all()
    del a, b


def test_zgemm_with_caller_workspace(o2m):
    a = W.complex_matrix(90, 70, 41)
    b = W.complex_matrix(70, 60, 42)
    need = o2m.workspace_bytes("z", 90, 60, 70, 16)
    ws = torch.empty(need, dtype=torch.uint8, device=DEV)
    o2m.set_workspace(ws)
    del ws                                  # the binding keeps the buffer alive
    try:
        got = host(o2m.zgemm_2m(to_dev(a), to_dev(b), n_moduli=16))
        with pytest.raises(o2m.O2MError):
            o2m.zgemm_2m(to_dev(W.complex_matrix(300, 70, 1)), to_dev(b), n_moduli=16)
    finally:
        o2m.set_workspace(None)
    assert same_bits(got, O.oq_zgemm(a, b, 16))


def test_residue_hook_matches_exact_integers(o2m):
    m, n, k, N = 37, 29, 90, 16
    a = W.complex_matrix(m, k, 51, dist="phi", phi=2.0)
    b = W.complex_matrix(k, n, 52, dist="phi", phi=2.0)
    res, E, F = o2m.zgemm_2m_residues(to_dev(a), to_dev(b), n_moduli=N)
    res = res.cpu().numpy()
    E0, _, F0, _ = O.exponents(a, b)
    assert np.array_equal(E.cpu().numpy(), E0) and np.array_equal(F.cpu().numpy(), F0)
    ms = O.moduli_2m(N)
    pA, pB = O.split_budget(O.budget(ms, k))
    ent = [(i, j) for i in range(0, m, 3) for j in range(0, n, 2)]
    cint = O.oq_cint(a, b, pA, pB, ent)
    for (i, j), (cr, ci) in zip(ent, cint):
        for l, q in enumerate(ms):
            assert int(res[l, 0, j, i]) == O.symmetric_lift(cr, q)
            assert int(res[l, 1, j, i]) == O.symmetric_lift(ci, q)


def test_zgemm_tolerance_vs_double_double(o2m):
    """Config 2 shape (1024^3, N(0,1)): the error against the unquantized
    product meets 4 u k |A||B| for N >= 14 (up to all 22 2M moduli) and
    shrinks ~3.7 bits per modulus."""
    m = n = k = 1024
    sa, sb = W.config_seeds(2)
    a = W.complex_matrix(m, k, sa)
    b = W.complex_matrix(k, n, sb)
    rng = np.random.default_rng(5)
    ent = [(int(i), int(j)) for i, j in zip(rng.integers(0, m, 2048), rng.integers(0, n, 2048))]
    hi, lo = O.dd_gemm(a, b, entries=ent)
    absab = np.array([np.sum(np.abs(a[i, :]) * np.abs(b[:, j])) for i, j in ent])
    A, B = to_dev(a), to_dev(b)
    curve = {}
    for N in (8, 10, 12, 14, 16, 18, 20, 22):
        C = host(o2m.zgemm_2m(A, B, n_moduli=N))
        c = np.array([C[i, j] for i, j in ent])
        curve[N] = O.error_vs_reference(c, absab, hi, lo, k, 2.0 ** -53)
        report("zgemm 1024^3 error", N=N, ratio=f"{curve[N]['ratio']:.3g}", maxrel=f"{curve[N]['maxrel']:.3g}")
    for N in (14, 16, 18, 20, 22):
        assert curve[N]["ratio"] <= 1.0
    seq = [curve[N]["maxrel"] for N in (8, 10, 12, 14, 16)]
    assert all(x > y for x, y in zip(seq, seq[1:]))


# ------------------------------------------------------------------ CGEMM


@pytest.mark.parametrize("shape,N", [((100, 90, 130), 8), ((257, 31, 300), 6), ((64, 64, 64), 16)])
def test_cgemm_bit_exact_vs_oracle(o2m, shape, N):
    m, n, k = shape
    a = W.complex_matrix(m, k, 61, dist="uniform", dtype=np.complex64)
    b = W.complex_matrix(k, n, 62, dist="uniform", dtype=np.complex64)
    ref = O.oq_cgemm(a, b, N)
    got = host(o2m.cgemm_2m(to_dev(a), to_dev(b), n_moduli=N))
    assert same_bits(got, ref)


def test_cgemm_tolerance(o2m):
    m, n, k = 256, 256, 2048
    a = W.complex_matrix(m, k, 71, dist="uniform", dtype=np.complex64)
    b = W.complex_matrix(k, n, 72, dist="uniform", dtype=np.complex64)
    got = host(o2m.cgemm_2m(to_dev(a), to_dev(b), n_moduli=8)).astype(np.complex128)
    hi, lo = O.dd_gemm(a.astype(np.complex128), b.astype(np.complex128))
    absab = np.abs(a.astype(np.complex128)) @ np.abs(b.astype(np.complex128))
    err = O.error_vs_reference(got, absab, hi, lo, k, 2.0 ** -24)
    report("cgemm error", ratio=err["ratio"], maxrel=err["maxrel"])
    assert err["ratio"] <= 1.0


# ------------------------------------------------------------------ HERK / SYRK


@pytest.mark.parametrize("shape,N", [((100, 130), 16), ((257, 64), 8), ((33, 500), 20), ((1, 3), 16), ((161, 90), 13),
                                     ((96, 40), 3)])
def test_zherk_bit_exact_lower_triangle(o2m, shape, N):
    n, k = shape
    a = W.complex_matrix(n, k, 81 + n, dist="phi", phi=1.0)
    ref = O.oq_zherk(a, N)
    sentinel = 3.25 - 1.5j
    out = o2m.colmajor(torch.full((n, n), sentinel, dtype=torch.complex128, device=DEV))
    o2m.zherk_2m(to_dev(a), n_moduli=N, out=out)
    got = host(out)
    low = np.tril(np.ones((n, n), dtype=bool))
    assert same_bits(got[low], ref[low])
    assert (got[~low] == sentinel).all()
    assert (np.diag(got).imag == 0).all()


@pytest.mark.parametrize("shape,N", [((100, 130), 16), ((70, 65), 16), ((257, 1), 8), ((40, 300), 22), ((130, 77), 9)])
def test_dsyrk_bit_exact_lower_triangle(o2m, shape, N):
    n, k = shape
    a = W.real_matrix(n, k, 91 + k)
    ref = O.oq_dsyrk(a, N)
    out = o2m.colmajor(torch.full((n, n), -7.0, dtype=torch.float64, device=DEV))
    o2m.dsyrk_2m(to_dev(a), n_moduli=N, out=out)
    got = host(out)
    low = np.tril(np.ones((n, n), dtype=bool))
    assert same_bits(got[low], ref[low])
    assert (got[~low] == -7.0).all()


# ------------------------------------------------------------------ full size, sampled


@pytest.mark.slow
def test_zgemm_8192_sampled_vs_oracle(o2m):
    """The benchmark workload (8192^3, U(-0.5,0.5) exp(0.5 N(0,1)), N = 16), in
    the benchmark's launch configuration, on sampled entries."""
    m = n = k = 8192
    N = 16
    sa, sb = W.config_seeds(3)
    a = W.complex_matrix(m, k, sa, dist="phi", phi=0.5)
    b = W.complex_matrix(k, n, sb, dist="phi", phi=0.5)
    C = host(o2m.zgemm_2m(to_dev(a), to_dev(b), n_moduli=N))
    rng = np.random.default_rng(8)
    ent = [(0, 0), (m - 1, n - 1), (m - 1, 0), (0, n - 1)]
    ent += [(int(i), int(j)) for i, j in zip(rng.integers(0, m, 60), rng.integers(0, n, 60))]
    ref = O.oq_zgemm(a, b, N, entries=ent)
    got = np.array([C[i, j] for i, j in ent])
    assert same_bits(got, ref)
    hi, lo = O.dd_gemm(a, b, entries=ent)
    absab = np.array([np.sum(np.abs(a[i, :]) * np.abs(b[:, j])) for i, j in ent])
    err = O.error_vs_reference(got, absab, hi, lo, k, 2.0 ** -53)
    report("zgemm 8192^3 sampled", ratio=err["ratio"], maxrel=err["maxrel"])
    assert err["ratio"] <= 1.0


def _sample(rng, m, n, count, lower=False):
    ent = [(0, 0), (m - 1, n - 1), (m - 1, 0)] + ([] if lower else [(0, n - 1)])
    while len(ent) < count:
        i, j = int(rng.integers(0, m)), int(rng.integers(0, n))
        if lower and i < j:
            i, j = j, i
        ent.append((i, j))
    return ent


@pytest.mark.slow
def test_zgemm_8192_phi2_sampled(o2m):
    """8192^3 with the wide exponent spread phi = 2 (N = 16)."""
    m = n = k = 8192
    sa, sb = W.config_seeds(3)
    a = W.complex_matrix(m, k, sa + 10, dist="phi", phi=2.0)
    b = W.complex_matrix(k, n, sb + 10, dist="phi", phi=2.0)
    C = host(o2m.zgemm_2m(to_dev(a), to_dev(b), n_moduli=16))
    ent = _sample(np.random.default_rng(9), m, n, 48)
    got = np.array([C[i, j] for i, j in ent])
    assert same_bits(got, O.oq_zgemm(a, b, 16, entries=ent))
    hi, lo = O.dd_gemm(a, b, entries=ent)
    absab = np.array([np.sum(np.abs(a[i, :]) * np.abs(b[:, j])) for i, j in ent])
    err = O.error_vs_reference(got, absab, hi, lo, k, 2.0 ** -53)
    report("zgemm 8192^3 phi=2 sampled", ratio=err["ratio"], maxrel=err["maxrel"])
    assert err["ratio"] <= 1.0


@pytest.mark.slow
def test_cgemm_16384_sampled(o2m):
    """CGEMM 16384^3, U(-1,1) fp32, N = 8, on sampled entries."""
    m = n = k = 16384
    sa, sb = W.config_seeds(4)
    a = W.complex_matrix(m, k, sa, dist="uniform", dtype=np.complex64)
    b = W.complex_matrix(k, n, sb, dist="uniform", dtype=np.complex64)
    C = host(o2m.cgemm_2m(to_dev(a), to_dev(b), n_moduli=8))
    ent = _sample(np.random.default_rng(10), m, n, 32)
    got = np.array([C[i, j] for i, j in ent])
    assert same_bits(got, O.oq_cgemm(a, b, 8, entries=ent))
    a64, b64 = a.astype(np.complex128), b.astype(np.complex128)
    hi, lo = O.dd_gemm(a64, b64, entries=ent)
    absab = np.array([np.sum(np.abs(a64[i, :]) * np.abs(b64[:, j])) for i, j in ent])
    err = O.error_vs_reference(got.astype(np.complex128), absab, hi, lo, k, 2.0 ** -24)
    report("cgemm 16384^3 sampled", ratio=err["ratio"], maxrel=err["maxrel"])
    assert err["ratio"] <= 1.0


@pytest.mark.slow
def test_zherk_8192_sampled(o2m):
    """HERK n = k = 8192, N(0,1), N = 16: sampled lower-triangle entries."""
    n = k = 8192
    sa, _ = W.config_seeds(5)
    a = W.complex_matrix(n, k, sa)
    C = host(o2m.zherk_2m(to_dev(a), n_moduli=16))
    ent = _sample(np.random.default_rng(11), n, n, 48, lower=True)
    got = np.array([C[i, j] for i, j in ent])
    ref = O.oq_zherk(a, 16, entries=ent)
    assert same_bits(got, ref)
    assert all(C[i, i].imag == 0 for i in (0, 17, n - 1))


@pytest.mark.slow
def test_zgemm_dealt_windows_ragged_sampled(o2m):
    """22 x 23 tiles of 256 (16 windows of 32, the last one partial) with
    k = 24000, so that one product's planes outgrow the Infinity Cache and the
    int8 GEMM deals its tile windows to the XCDs round-robin; sampled entries,
    among them the first and last tile rows and columns, are bit-exact."""
    m, n, k = 22 * 256 - 37, 23 * 256 - 5, 24000
    a = W.complex_matrix(m, k, 9101)
    b = W.complex_matrix(k, n, 9102)
    C = host(o2m.zgemm_2m(to_dev(a), to_dev(b), n_moduli=16))
    rng = np.random.default_rng(13)
    ent = [(0, 0), (m - 1, n - 1), (m - 1, 0), (0, n - 1), (5375, 5631), (5376, 5632)]
    ent += [(int(i), int(j)) for i, j in zip(rng.integers(0, m, 30), rng.integers(0, n, 30))]
    ent += [(int(i), int(j)) for i, j in zip(rng.integers(m - 219, m, 8), rng.integers(n - 251, n, 8))]
    got = np.array([C[i, j] for i, j in ent])
    assert same_bits(got, O.oq_zgemm(a, b, 16, entries=ent))


MANY_TILES = [
    # m, n, k, N: many tiles per product, ragged edges; k = 250: one ring of 4
    # k-stages per tile; N = 22: 44 products of 16 tiles each.
    (8 * 256 - 13, 4 * 256 - 7, 250, 16),
    (4 * 256 - 13, 4 * 256 - 7, 500, 22),
]


@pytest.mark.parametrize("case", MANY_TILES, ids=[f"{c[0]}x{c[1]}x{c[2]}-N{c[3]}" for c in MANY_TILES])
def test_zgemm_many_tiles_bit_exact(o2m, case):
    """Whole outputs bit-exact against the oracle over many output tiles."""
    m, n, k, N = case
    a = W.complex_matrix(m, k, 9201 + N, dist="phi", phi=2.0)
    b = W.complex_matrix(k, n, 9202 + N, dist="phi", phi=2.0)
    print(f"[parity] many tiles {m}x{n}x{k} N={N}", flush=True)
    got = host(o2m.zgemm_2m(to_dev(a), to_dev(b), n_moduli=N))
    assert same_bits(got, O.oq_zgemm(a, b, N))


def test_zgemm_pooled_tiles_sampled(o2m):
    """129 k-stages and 8 x 8 tiles per product, 32 products: 256 slots per
    XCD, so the int8 GEMM leaves the last eighth of every XCD's slots to a
    pool that workgroups claim at run time (with spares that take slots of
    other XCDs' pools).  Two sampled entries in every 256 x 256 output tile,
    each depending on that tile of all 32 products, are bit-exact: a tile
    skipped or computed twice by the claims would show."""
    m, n, k = 8 * 256 - 21, 8 * 256 - 3, 8200
    a = W.complex_matrix(m, k, 9301)
    b = W.complex_matrix(k, n, 9302)
    print(f"[parity] pooled tiles {m}x{n}x{k} N=16", flush=True)
    C = host(o2m.zgemm_2m(to_dev(a), to_dev(b), n_moduli=16))
    rng = np.random.default_rng(31)
    ent = [(m - 1, n - 1)]
    for ti in range(8):
        for tj in range(8):
            hi_i, hi_j = min(256, m - 256 * ti), min(256, n - 256 * tj)
            for _ in range(2):
                ent.append((256 * ti + int(rng.integers(0, hi_i)), 256 * tj + int(rng.integers(0, hi_j))))
    got = np.array([C[i, j] for i, j in ent])
    assert same_bits(got, O.oq_zgemm(a, b, 16, entries=ent))


@pytest.mark.slow
def test_zgemm_pooled_with_idle_slots_sampled(o2m):
    """19 x 3 = 57 tiles per product (not a multiple of the 8 XCDs, so every
    product leaves 7 idle slots, some of them in the pools) with 129 k-stages
    and 32 products: pooled launch.  Two sampled entries in each of the 57
    output tiles, bit-exact."""
    m, n, k = 19 * 256 - 5, 3 * 256 - 9, 8200
    a = W.complex_matrix(m, k, 9501)
    b = W.complex_matrix(k, n, 9502)
    print(f"[parity] pooled with idle slots {m}x{n}x{k} N=16", flush=True)
    C = host(o2m.zgemm_2m(to_dev(a), to_dev(b), n_moduli=16))
    rng = np.random.default_rng(51)
    ent = [(m - 1, n - 1)]
    for ti in range(19):
        for tj in range(3):
            for _ in range(2):
                ent.append((256 * ti + int(rng.integers(0, min(256, m - 256 * ti))),
                            256 * tj + int(rng.integers(0, min(256, n - 256 * tj)))))
    got = np.array([C[i, j] for i, j in ent])
    assert same_bits(got, O.oq_zgemm(a, b, 16, entries=ent))


@pytest.mark.slow
def test_zgemm_pooled_random_shapes(o2m):
    """Random ragged shapes with k >= 8129 (the int8 GEMM's claimed pool in
    use), moduli counts 8..22 and both scaling rules; two sampled entries in
    every output tile and the corners, bit-exact.  O2M_POOLED_CASES and
    O2M_POOLED_SEED widen the sweep (default: 4 cases, seed 777)."""
    rng = np.random.default_rng(int(os.environ.get("O2M_POOLED_SEED", "777")))
    for case in range(int(os.environ.get("O2M_POOLED_CASES", "4"))):
        m, n = (int(x) for x in rng.integers(256, 2600, 2))
        k = int(rng.choice([8200, 9001, 10240, 12000]))
        N = int(rng.integers(8, 23))
        rule = "cs" if rng.random() < 0.3 else "max"
        if rule == "cs" and O.budget_cs(O.moduli_set(N), k, False) is None:
            rule = "max"
        a = W.complex_matrix(m, k, 20000 + case, dist="phi", phi=float(rng.choice([0.5, 2.0])))
        b = W.complex_matrix(k, n, 30000 + case)
        print(f"[parity] pooled random case {case}: {m}x{n}x{k} N={N} {rule}", flush=True)
        C = host(o2m.zgemm_2m(to_dev(a), to_dev(b), n_moduli=N, scaling=rule))
        ent = [(m - 1, n - 1), (0, 0)]
        for ti in range(-(-m // 256)):
            for tj in range(-(-n // 256)):
                for _ in range(2):
                    ent.append((256 * ti + int(rng.integers(0, min(256, m - 256 * ti))),
                                256 * tj + int(rng.integers(0, min(256, n - 256 * tj)))))
        got = np.array([C[i, j] for i, j in ent])
        assert same_bits(got, O.oq_zgemm(a, b, N, entries=ent, scaling=rule)), case


@pytest.mark.slow
def test_zgemm_tall_skinny_sampled(o2m):
    """m = n = 4096, k = 65536 (N = 16): int32 headroom and the long k-loop."""
    m, n, k = 4096, 4096, 65536
    sa, sb = W.config_seeds(6)
    a = W.complex_matrix(m, k, sa)
    b = W.complex_matrix(k, n, sb)
    C = host(o2m.zgemm_2m(to_dev(a), to_dev(b), n_moduli=16))
    ent = _sample(np.random.default_rng(12), m, n, 32)
    got = np.array([C[i, j] for i, j in ent])
    assert same_bits(got, O.oq_zgemm(a, b, 16, entries=ent))
    hi, lo = O.dd_gemm(a, b, entries=ent)
    absab = np.array([np.sum(np.abs(a[i, :]) * np.abs(b[:, j])) for i, j in ent])
    err = O.error_vs_reference(got, absab, hi, lo, k, 2.0 ** -53)
    report("zgemm 4096x4096x65536 sampled", ratio=err["ratio"], maxrel=err["maxrel"])
    assert err["ratio"] <= 1.0


@pytest.mark.slow
def test_dsyrk_4096_sampled(o2m):
    """SYRK n = 4096, k = 8191 (odd: the zero-padded half-k HERK)."""
    n, k = 4096, 8191
    a = W.real_matrix(n, k, 701)
    C = host(o2m.dsyrk_2m(to_dev(a), n_moduli=16))
    ent = _sample(np.random.default_rng(13), n, n, 48, lower=True)
    got = np.array([C[i, j] for i, j in ent])
    assert same_bits(got, O.oq_dsyrk(a, 16, entries=ent))


# ------------------------------------------------------------------ layouts and streams


def _padded_view(x, pad_rows):
    """Device view of host matrix x inside a larger column-major buffer
    (leading dimension rows + pad_rows), the padding filled with NaN so that a
    read outside the view would poison the result."""
    rows, cols = x.shape
    big = np.full((rows + pad_rows, cols), np.nan, dtype=x.dtype)
    big[:rows, :] = x
    return to_dev(big)[:rows, :]


def test_zgemm_strided_operands_and_output(o2m):
    m, n, k = 70, 50, 90
    a = W.complex_matrix(m, k, 401)
    b = W.complex_matrix(k, n, 402)
    A, B = _padded_view(a, 13), _padded_view(b, 7)
    assert A.stride(1) == m + 13 and B.stride(1) == k + 7
    Cbig = o2m.colmajor(torch.full((m + 5, n), 9.0 + 9j, dtype=torch.complex128, device=DEV))
    C = Cbig[:m, :]
    o2m.zgemm_2m(A, B, n_moduli=16, out=C)
    got = host(Cbig)
    assert same_bits(np.asfortranarray(got[:m, :]), O.oq_zgemm(a, b, 16))
    assert (got[m:, :] == 9.0 + 9j).all()           # rows beyond m untouched



# the CRT stores whole lines: complex fp64 results leave each wave in row
# order (a lane stores rows computed by other lanes), HERK/SYRK threads own
# rows r, r + 8, r + 16, r + 24 of a tile column.  Row counts around the wave
# (256 rows) and tile (32, 128) boundaries, with a padded ldc whose extra rows
# (and, for HERK/SYRK, the upper triangle) must stay untouched.
@pytest.mark.parametrize("m", [1, 63, 64, 65, 255, 256, 257, 1023, 1025, 1100])
def test_zgemm_ragged_rows_padded_ldc(o2m, m):
    n, k, pad = 3, 40, 37
    a = W.complex_matrix(m, k, 430 + m)
    b = W.complex_matrix(k, n, 431)
    Cbig = o2m.colmajor(torch.full((m + pad, n), -5.0 + 2j, dtype=torch.complex128, device=DEV))
    o2m.zgemm_2m(to_dev(a), to_dev(b), n_moduli=16, out=Cbig[:m, :])
    got = host(Cbig)
    assert same_bits(np.asfortranarray(got[:m, :]), O.oq_zgemm(a, b, 16))
    assert (got[m:, :] == -5.0 + 2j).all()


@pytest.mark.parametrize("m", [65, 257, 1025])
def test_cgemm_ragged_rows_padded_ldc(o2m, m):
    n, k, pad = 2, 33, 11
    a = W.complex_matrix(m, k, 440 + m, dist="uniform", dtype=np.complex64)
    b = W.complex_matrix(k, n, 441, dist="uniform", dtype=np.complex64)
    Cbig = o2m.colmajor(torch.full((m + pad, n), 3.0 - 1j, dtype=torch.complex64, device=DEV))
    o2m.cgemm_2m(to_dev(a), to_dev(b), n_moduli=8, out=Cbig[:m, :])
    got = host(Cbig)
    assert same_bits(np.asfortranarray(got[:m, :]), O.oq_cgemm(a, b, 8))
    assert (got[m:, :] == 3.0 - 1j).all()


@pytest.mark.parametrize("n,N", [(1, 16), (31, 16), (33, 7), (127, 16), (129, 13), (200, 16)])
def test_zherk_dsyrk_ragged_padded_ldc(o2m, n, N):
    k, pad = 20, 9
    a = W.complex_matrix(n, k, 450 + n)
    Cbig = o2m.colmajor(torch.full((n + pad, n), 6.5 - 0.5j, dtype=torch.complex128, device=DEV))
    o2m.zherk_2m(to_dev(a), n_moduli=N, out=Cbig[:n, :])
    got = host(Cbig)
    low = np.tril(np.ones((n, n), dtype=bool))
    assert same_bits(got[:n, :][low], O.oq_zherk(a, N)[low])
    assert (got[:n, :][~low] == 6.5 - 0.5j).all() and (got[n:, :] == 6.5 - 0.5j).all()
    r = W.real_matrix(n, 2 * k + 1, 460 + n)
    Rbig = o2m.colmajor(torch.full((n + pad, n), -4.25, dtype=torch.float64, device=DEV))
    o2m.dsyrk_2m(to_dev(r), n_moduli=N, out=Rbig[:n, :])
    gotr = host(Rbig)
    assert same_bits(gotr[:n, :][low], O.oq_dsyrk(r, N)[low])
    assert (gotr[:n, :][~low] == -4.25).all() and (gotr[n:, :] == -4.25).all()

def _offset_view(x, pad_rows, offset):
    """As _padded_view, with the view starting `offset` elements into the
    buffer (a base address off the 16-byte grid for offset 1 in fp32)."""
    rows, cols = x.shape
    big = np.full((rows + pad_rows, cols), np.nan, dtype=x.dtype)
    big[offset:offset + rows, :] = x
    return to_dev(big)[offset:offset + rows, :]


# complex fp32 entries are read two per 16-byte load when every pair is
# aligned (even leading dimension, aligned base): consecutive entries of a
# column of B, rows 2i, 2i + 1 of A; one entry per load otherwise
PAIR_CASES = [(41, 33, 11, 0), (41, 33, 10, 0), (40, 33, 11, 1), (41, 4101, 3, 0), (40, 4101, 4, 1), (257, 300, 5, 0)]


@pytest.mark.parametrize("rule", ["max", "cs"])
@pytest.mark.parametrize("m,k,pad,offset", PAIR_CASES, ids=[f"m{m}-k{k}-pad{p}-off{o}" for m, k, p, o in PAIR_CASES])
def test_cgemm_paired_and_single_loads(o2m, m, k, pad, offset, rule):
    a = W.complex_matrix(m, k, 415, dist="uniform", dtype=np.complex64)
    b = W.complex_matrix(k, 21, 416, dist="uniform", dtype=np.complex64)
    B = _offset_view(b, pad, offset)
    assert B.stride(1) == k + pad
    got = host(o2m.cgemm_2m(to_dev(a), B, n_moduli=8, scaling=rule))
    ref = O.oq_cgemm(a, b, 8, scaling=rule)
    assert same_bits(got, ref)
    A = _offset_view(a, pad, offset)                  # A's rows in pairs (or not), B plain
    assert A.stride(1) == m + pad
    got = host(o2m.cgemm_2m(A, to_dev(b), n_moduli=8, scaling=rule))
    assert same_bits(got, ref)


def test_cgemm_and_zherk_strided(o2m):
    a = W.complex_matrix(40, 33, 411, dist="uniform", dtype=np.complex64)
    b = W.complex_matrix(33, 21, 412, dist="uniform", dtype=np.complex64)
    got = host(o2m.cgemm_2m(_padded_view(a, 3), _padded_view(b, 11), n_moduli=8))
    assert same_bits(got, O.oq_cgemm(a, b, 8))
    h = W.complex_matrix(45, 60, 413)
    Cbig = o2m.colmajor(torch.zeros((45 + 6, 45), dtype=torch.complex128, device=DEV))
    o2m.zherk_2m(_padded_view(h, 9), n_moduli=16, out=Cbig[:45, :])
    got = host(Cbig)[:45, :]
    ref = O.oq_zherk(h, 16)
    low = np.tril(np.ones((45, 45), dtype=bool))
    assert same_bits(got[low], ref[low])


def test_zgemm_caller_workspace_is_per_stream(o2m):
    a = W.complex_matrix(90, 70, 43)
    b = W.complex_matrix(70, 60, 44)
    need = o2m.workspace_bytes("z", 90, 60, 70, 16)
    s = torch.cuda.Stream()
    ws = torch.empty(need, dtype=torch.uint8, device=DEV)
    o2m.set_workspace(ws, stream=s)            # only calls on s use (and are limited by) it
    try:
        big = W.complex_matrix(300, 70, 2)
        got_big = host(o2m.zgemm_2m(to_dev(big), to_dev(b), n_moduli=16))   # current stream: library memory
        with torch.cuda.stream(s):
            got = o2m.zgemm_2m(to_dev(a), to_dev(b), n_moduli=16)
            with pytest.raises(o2m.O2MError):
                o2m.zgemm_2m(to_dev(big), to_dev(b), n_moduli=16)
        s.synchronize()
        got = host(got)
    finally:
        o2m.set_workspace(None, stream=s)
    assert same_bits(got, O.oq_zgemm(a, b, 16))
    assert same_bits(got_big, O.oq_zgemm(big, b, 16))
    with pytest.raises(ValueError):
        o2m.set_workspace(torch.empty(need, dtype=torch.uint8))               # host memory
    with pytest.raises(ValueError):
        o2m.set_workspace(torch.empty((need, 2), dtype=torch.uint8, device=DEV)[:, 0])  # strided
    o2m.release_workspace(s)


def test_concurrent_calls_on_two_streams(o2m):
    """Calls that overlap on two streams have workspaces of their own: two
    different-shape ZGEMMs enqueued back to back on two streams, several
    times over, are bit-identical to the oracle at sampled entries and to the
    same calls run one after another."""
    shapes = [(1536, 1280, 1088, 16, 811), (1024, 1792, 1600, 12, 823)]
    ops = []
    for m, n, k, N, seed in shapes:
        a = W.complex_matrix(m, k, seed, dist="phi", phi=0.5)
        b = W.complex_matrix(k, n, seed + 1, dist="phi", phi=0.5)
        ops.append((a, b, to_dev(a), to_dev(b), N))
    serial = [host(o2m.zgemm_2m(A, B, n_moduli=N)) for _, _, A, B, N in ops]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    outs = []
    for rep in range(3):
        for (a, b, A, B, N), s in zip(ops, streams):
            with torch.cuda.stream(s):
                outs.append((rep, o2m.zgemm_2m(A, B, n_moduli=N)))
    torch.cuda.synchronize()
    rng = np.random.default_rng(5)
    for t, (rep, C) in enumerate(outs):
        a, b, _, _, N = ops[t % 2]
        got = host(C)
        assert same_bits(got, serial[t % 2]), (rep, t % 2)
        ent = _sample(rng, a.shape[0], b.shape[1], 300)
        ref = O.oq_zgemm(a, b, N, entries=ent)
        assert same_bits(np.array([got[i, j] for i, j in ent]), ref)
    for s in streams:
        o2m.release_workspace(s)


def test_nonfinite_status_bit(o2m):
    a = W.complex_matrix(70, 50, 71)
    b = W.complex_matrix(50, 40, 72)
    o2m.get_status()                                      # start clean
    got = host(o2m.zgemm_2m(to_dev(a), to_dev(b), n_moduli=16))
    assert np.isfinite(got).all() and o2m.get_status() == 0
    a[13, 7] = complex(np.nan, 0.0)                       # a NaN row of A
    got = host(o2m.zgemm_2m(to_dev(a), to_dev(b), n_moduli=16))
    assert np.isnan(got[13, :]).all()
    assert o2m.get_status() == o2m.STATUS_NONFINITE
    assert o2m.get_status() == 0                          # cleared by the read
    b2 = b.copy()
    b2[3, 39] = complex(0.0, -np.inf)                     # an Inf column of B (last column)
    host(o2m.cgemm_2m(to_dev(a.astype(np.complex64)), to_dev(b2.astype(np.complex64)), n_moduli=8))
    assert o2m.get_status() == o2m.STATUS_NONFINITE
    h = W.complex_matrix(60, 30, 73)
    h[59, 0] = np.inf                                     # the last row of a HERK operand
    o2m.zherk_2m(to_dev(h), n_moduli=16)
    assert o2m.get_status() == o2m.STATUS_NONFINITE
    o2m.zherk_2m(to_dev(W.complex_matrix(60, 30, 74)), n_moduli=16, scaling="cs")
    assert o2m.get_status() == 0
    # the Cauchy-Schwarz rule finds non-finite rows and columns in its one pass
    got = host(o2m.zgemm_2m(to_dev(a), to_dev(b), n_moduli=16, scaling="cs"))
    assert np.isnan(got[13, :]).all() and o2m.get_status() == o2m.STATUS_NONFINITE
    host(o2m.cgemm_2m(to_dev(a.astype(np.complex64) * 0 + 1), to_dev(b2.astype(np.complex64)), n_moduli=8,
                      scaling="cs"))
    assert o2m.get_status() == o2m.STATUS_NONFINITE
    o2m.zherk_2m(to_dev(h), n_moduli=16, scaling="cs")
    assert o2m.get_status() == o2m.STATUS_NONFINITE
    host(o2m.zgemm_2m(to_dev(W.complex_matrix(70, 50, 75)), to_dev(b), n_moduli=16, scaling="cs"))
    assert o2m.get_status() == 0


def test_calls_on_a_side_stream(o2m):
    a = W.complex_matrix(120, 100, 421)
    b = W.complex_matrix(100, 80, 422)
    A, B = to_dev(a), to_dev(b)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        C1 = o2m.zgemm_2m(A, B, n_moduli=16)                 # current stream = s
        C2 = o2m.zgemm_2m(A, B, n_moduli=12, stream=s)
    s.synchronize()
    assert same_bits(np.asfortranarray(C1.cpu().numpy()), O.oq_zgemm(a, b, 16))
    assert same_bits(np.asfortranarray(C2.cpu().numpy()), O.oq_zgemm(a, b, 12))


def _graph_replays(o2m, m, n, k, N, seeds, entries=None, scaling="max", edit=None):
    """Capture one zgemm_2m call into a HIP graph and replay it on fresh
    inputs copied into the captured buffers (eager copies and a sync between
    replays); each replay must equal the oracle for the inputs it saw.
    ``edit(seed, a)`` may change A's rows before a replay."""
    A = o2m.colmajor(torch.zeros((m, k), dtype=torch.complex128, device=DEV))
    B = o2m.colmajor(torch.zeros((k, n), dtype=torch.complex128, device=DEV))
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        o2m.zgemm_2m(A, B, n_moduli=N, scaling=scaling)  # sizes the capture stream's workspace outside the capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        C = o2m.zgemm_2m(A, B, n_moduli=N, scaling=scaling)
    for seed in seeds:
        a = W.complex_matrix(m, k, seed, dist="phi", phi=2.0)
        b = W.complex_matrix(k, n, seed + 1, dist="phi", phi=2.0)
        if edit:
            edit(seed, a)
        A.copy_(to_dev(a))
        B.copy_(to_dev(b))
        g.replay()
        got = host(C)
        if entries is None:
            assert same_bits(got, O.oq_zgemm(a, b, N, scaling=scaling)), seed
        else:
            ref = O.oq_zgemm(a, b, N, entries=entries, scaling=scaling)
            assert same_bits(np.array([got[i, j] for i, j in entries]), ref), seed
    del g
    o2m.release_workspace(s)


def test_capture_without_a_sized_workspace_is_refused(o2m):
    """A capture on a stream whose workspace is too small fails with
    O2M_ERR_WORKSPACE and leaves the capture intact (nothing allocated or
    synchronized inside it)."""
    A = o2m.colmajor(torch.zeros((64, 64), dtype=torch.complex128, device=DEV))
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        with pytest.raises(o2m.O2MError) as e:
            o2m.zgemm_2m(A, A, n_moduli=16)
        C = A * 2                                          # the capture still works
    assert e.value.status == -22
    g.replay()
    torch.cuda.synchronize()
    assert (C == 0).all()


def test_zgemm_in_a_hip_graph(o2m):
    """The call is capturable: no host synchronisation, allocation or memset
    once the workspace is sized; three replays on three inputs, bit-exact."""
    print("[parity] graph replays 300x270x520 N=16", flush=True)
    _graph_replays(o2m, 300, 270, 520, 16, seeds=(9401, 9403, 9405))


def test_zgemm_cs_in_a_hip_graph(o2m):
    """The Cauchy-Schwarz rule's one-pass scaling is capturable too, including
    the rows its chunk records leave open (summed again inside the graph): the
    second replay holds two such rows, the third none."""
    from cs_inputs import straddle_vector

    def edit(seed, a):
        if seed == 9423:
            a[5, :] = straddle_vector(a.shape[1], "low")
            a[200, :] = straddle_vector(a.shape[1], "high")
    print("[parity] graph replays 300x270x520 N=16, Cauchy-Schwarz rule", flush=True)
    _graph_replays(o2m, 300, 270, 520, 16, seeds=(9421, 9423, 9425), scaling="cs", edit=edit)


@pytest.mark.slow
def test_zgemm_pooled_in_a_hip_graph(o2m):
    """As above at a shape whose int8 GEMM pools the last slots of each XCD:
    the pool counters are cleared inside the graph (by the first kernel's
    fill), so every replay claims from fresh pools; sampled entries in every
    output tile, bit-exact."""
    m, n, k = 8 * 256 - 21, 8 * 256 - 3, 8200
    rng = np.random.default_rng(41)
    ent = [(256 * ti + int(rng.integers(0, min(256, m - 256 * ti))),
            256 * tj + int(rng.integers(0, min(256, n - 256 * tj)))) for ti in range(8) for tj in range(8)]
    print(f"[parity] graph replays {m}x{n}x{k} N=16 (pooled)", flush=True)
    _graph_replays(o2m, m, n, k, 16, seeds=(9411, 9413), entries=ent)


def test_phase_timing(o2m):
    """The per-phase HIP events: four positive phase times averaged over the
    calls since enabling, a restart on re-enabling, nothing while disabled,
    and results unchanged by the timing."""
    a = W.complex_matrix(300, 200, 441)
    b = W.complex_matrix(200, 260, 442)
    A, B = to_dev(a), to_dev(b)
    o2m.phase_timing(True)
    try:
        for _ in range(3):
            C = o2m.zgemm_2m(A, B, n_moduli=16)
        t = o2m.phase_times()
        assert list(t) == ["scale", "residues", "int8_gemm", "crt"]
        assert all(v > 0.0 for v in t.values()), t
        o2m.phase_timing(True)                      # restart: no call timed yet
        assert o2m.phase_times() == {}
    finally:
        o2m.phase_timing(False)
    o2m.zgemm_2m(A, B, n_moduli=16)
    assert o2m.phase_times() == {}
    assert same_bits(host(C), O.oq_zgemm(a, b, 16))


@pytest.mark.slow
def test_zgemm_k_at_the_int32_limit_sampled(o2m):
    """k = 149130, the largest k whose int32 accumulation is exact with 2M
    residues (|r| <= 120): the longest k-loop of the plain calls."""
    m, n, k = 256, 300, 149130
    a = W.complex_matrix(m, k, 431)
    b = W.complex_matrix(k, n, 432)
    C = host(o2m.zgemm_2m(to_dev(a), to_dev(b), n_moduli=16))
    rng = np.random.default_rng(26)
    ent = [(0, 0), (m - 1, n - 1)] + [(int(i), int(j)) for i, j in zip(rng.integers(0, m, 30), rng.integers(0, n, 30))]
    got = np.array([C[i, j] for i, j in ent])
    assert same_bits(got, O.oq_zgemm(a, b, 16, entries=ent))


# The residue kernel reduces quantized values below 2^44 without splitting them
# into base-2^26 digits; above that they are split.  Shapes whose shifts sit on
# either side of that bound (operands on different sides in one call), with
# entries that quantize to exactly +-2^p.
DIGIT_CASES = [("max", 13, 64), ("max", 13, 128), ("max", 13, 256), ("max", 14, 8192), ("cs", 11, 100),
               ("cs", 12, 100)]


@pytest.mark.parametrize("rule,N,k", DIGIT_CASES, ids=[f"{r}-N{n}-k{k}" for r, n, k in DIGIT_CASES])
def test_residue_digit_boundaries(o2m, rule, N, k):
    m, n = 40, 24
    a = W.complex_matrix(m, k, 8800 + k, dist="phi", phi=2.0)
    b = W.complex_matrix(k, n, 8900 + k, dist="phi", phi=2.0)
    below = np.nextafter(1.0, 0.0)           # just below 2^0: quantizes to 2^p under the max rule
    a[3, :] = 0.5
    a[3, 0] = complex(below, -below)
    b[:, 4] = -0.25
    b[7, 4] = complex(-below / 2, below / 2)
    pA, pB = O.shifts(rule, O.moduli_set(N), k)
    ref = O.oq_zgemm(a, b, N, scaling=rule)
    got = host(o2m.zgemm_2m(to_dev(a), to_dev(b), n_moduli=N, scaling=rule))
    ok = same_bits(got, ref)
    report("digit boundary", rule=rule, N=N, k=k, pA=pA, pB=pB, bitexact=ok)
    assert ok


# --------------------------------------------- transposed and conjugated operands
# C = op(A) op(B), op = 'N', 'T' or 'C': the library reads rows of op(A) as
# columns of the stored A when transposed and negates imaginary parts when
# conjugated; the result must equal the oracle's exact output on the explicitly
# formed op(A), op(B).

OPS = [(ta, tb) for ta in "NTC" for tb in "NTC"]


def _stored(op_x, t):
    """The matrix a caller stores so that op(stored) = op_x."""
    return op_x if t == "N" else (op_x.T if t == "T" else op_x.conj().T)


@pytest.mark.parametrize("rule", ["max", "cs"])
@pytest.mark.parametrize("ta,tb", OPS, ids=[a + b for a, b in OPS])
def test_zgemm_op_bit_exact(o2m, ta, tb, rule):
    m, n, k, N = 70, 50, 90, 16
    opa = W.complex_matrix(m, k, 4701, dist="phi", phi=2.0)
    opb = W.complex_matrix(k, n, 4702, dist="phi", phi=2.0)
    A = _padded_view(np.ascontiguousarray(_stored(opa, ta)), 5)
    B = _padded_view(np.ascontiguousarray(_stored(opb, tb)), 3)
    got = host(o2m.zgemm_2m_op(A, B, ta, tb, n_moduli=N, scaling=rule))
    ok = same_bits(got, O.oq_zgemm(opa, opb, N, scaling=rule))
    report("zgemm op", ops=ta + tb, rule=rule, bitexact=ok)
    assert ok


@pytest.mark.parametrize("rule", ["max", "cs"])
@pytest.mark.parametrize("ta,tb,pad", [("T", "N", 4), ("C", "T", 3), ("N", "C", 2), ("C", "C", 1)])
def test_cgemm_op_bit_exact(o2m, ta, tb, pad, rule):
    m, n, k = 41, 30, 67
    opa = W.complex_matrix(m, k, 4711, dist="uniform", dtype=np.complex64)
    opb = W.complex_matrix(k, n, 4712, dist="uniform", dtype=np.complex64)
    A = _padded_view(np.ascontiguousarray(_stored(opa, ta)), pad)
    B = _padded_view(np.ascontiguousarray(_stored(opb, tb)), pad + 1)
    got = host(o2m.cgemm_2m_op(A, B, ta, tb, n_moduli=8, scaling=rule))
    assert same_bits(got, O.oq_cgemm(opa, opb, 8, scaling=rule))


def test_zgemm_op_matches_plain_call_and_hybrid(o2m):
    """'N','N' is the plain call; a hybrid set (N = 26) with both operands
    conjugate-transposed; k = 0 zeroes C."""
    m, n, k = 33, 29, 300
    a = W.complex_matrix(m, k, 4721)
    b = W.complex_matrix(k, n, 4722)
    plain = host(o2m.zgemm_2m(to_dev(a), to_dev(b), n_moduli=16))
    assert same_bits(host(o2m.zgemm_2m_op(to_dev(a), to_dev(b), "n", "n", n_moduli=16)), plain)
    got = host(o2m.zgemm_2m_op(to_dev(a.conj().T), to_dev(b.conj().T), "C", "C", n_moduli=26, scaling="cs"))
    assert same_bits(got, O.oq_zgemm(a, b, 26, scaling="cs"))
    z = o2m.zgemm_2m_op(to_dev(np.zeros((0, m), np.complex128)), to_dev(np.zeros((n, 0), np.complex128)),
                        "T", "T", n_moduli=16)
    assert z.shape == (m, n) and (host(z) == 0).all()


@pytest.mark.slow
@pytest.mark.parametrize("rule", ["max", "cs"])
@pytest.mark.parametrize("ta,tb", [("C", "T"), ("T", "N")])
def test_zgemm_op_4096_sampled(o2m, ta, tb, rule):
    """Transposed and conjugated operands of 256 MiB each, large enough for the
    scaling pass's streaming loads in both scan layouts: sampled entries
    bit-exact against the oracle on the explicitly formed op(A), op(B)."""
    m = n = k = 4096
    N = 16
    opa = W.complex_matrix(m, k, 4711, dist="phi", phi=0.5)
    opb = W.complex_matrix(k, n, 4712, dist="phi", phi=0.5)
    A = to_dev(np.ascontiguousarray(_stored(opa, ta)))
    B = to_dev(np.ascontiguousarray(_stored(opb, tb)))
    C = host(o2m.zgemm_2m_op(A, B, ta, tb, n_moduli=N, scaling=rule))
    ent = _sample(np.random.default_rng(47), m, n, 48)
    got = np.array([C[i, j] for i, j in ent])
    ok = same_bits(got, O.oq_zgemm(opa, opb, N, entries=ent, scaling=rule))
    report("zgemm op 4096^3 sampled", ops=ta + tb, rule=rule, bitexact=ok)
    assert ok


def test_cs_resummed_entries_transposed_operands(o2m):
    """Rows of op(A) read as columns of the stored A, columns of op(B) read as
    rows of the stored B, among them ones whose chunk records leave the
    Cauchy-Schwarz exponent open (summed again from the data)."""
    from cs_inputs import straddle_vector
    m, n, k, N = 24, 20, 4096, 16
    opa = W.complex_matrix(m, k, 4731, dist="phi", phi=0.5)
    opb = W.complex_matrix(k, n, 4732, dist="phi", phi=0.5)
    for i, kind in ((2, "low"), (m - 1, "high")):      # a column of the stored A: chunks of 2048
        opa[i, :] = straddle_vector(k, kind, exact=(0, 2048), binade=(2048, 2112), stride=2048)
    for j, kind in ((0, "high"), (11, "low")):         # a row of the stored B: chunks of 16..128 columns
        opb[:, j] = straddle_vector(k, kind)
    for ta, tb in (("T", "T"), ("C", "C"), ("C", "T")):
        A = to_dev(np.ascontiguousarray(_stored(opa, ta)))
        B = to_dev(np.ascontiguousarray(_stored(opb, tb)))
        got = host(o2m.zgemm_2m_op(A, B, ta, tb, n_moduli=N, scaling="cs"))
        ok = same_bits(got, O.oq_zgemm(opa, opb, N, scaling="cs"))
        report("cs re-summed, transposed", ops=ta + tb, bitexact=ok)
        assert ok
