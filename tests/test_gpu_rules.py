"""GPU parity of the Cauchy-Schwarz scaling rule and of the rank-2k updates
(HER2K / SYR2K, Section 5) with the CPU oracle, through the C-ABI.

As for the plain calls, the HIP path computes Algorithm 1's exact output, so
results are compared bit for bit; accuracy against the unquantized product is
checked separately with the tolerance 4 u k |A||B|."""
import numpy as np
import pytest

import oracle as O
import workloads as W
from conftest import same_bits

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

DEV = "cuda:0"


@pytest.fixture(scope="module")
def o2m():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_05419_amd as lib
    return lib


def to_dev(x):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(x).T)).to(DEV).t()


def host(t):
    torch.cuda.synchronize()
    return np.asfortranarray(t.cpu().numpy())


def report(name, **kw):
    print(f"[rules] {name} " + " ".join(f"{k}={v}" for k, v in kw.items()), flush=True)


LOW = lambda n: np.tril(np.ones((n, n), dtype=bool))


# ------------------------------------------------------------ Cauchy-Schwarz


CS_CASES = [
    # m, n, k, dist, phi, N
    (64, 64, 64, "normal", 0.5, 16),
    (100, 77, 130, "phi", 2.0, 16),
    (257, 300, 200, "phi", 0.5, 16),
    (70, 90, 300, "phi", 2.0, 8),
    (33, 47, 65, "normal", 0.5, 3),
    (40, 50, 96, "phi", 2.0, 22),      # shifts above 62: the three-way split
    (65, 65, 1000, "uniform", 0.5, 20),
    (5, 3, 1, "normal", 0.5, 2),
]


@pytest.mark.parametrize("case", CS_CASES, ids=[f"{c[0]}x{c[1]}x{c[2]}-{c[3]}-N{c[5]}" for c in CS_CASES])
def test_zgemm_cs_bit_exact(o2m, case):
    m, n, k, dist, phi, N = case
    a = W.complex_matrix(m, k, 3000 + m, dist=dist, phi=phi)
    b = W.complex_matrix(k, n, 4000 + n, dist=dist, phi=phi)
    ref = O.oq_zgemm(a, b, N, scaling="cs")
    got = host(o2m.zgemm_2m(to_dev(a), to_dev(b), n_moduli=N, scaling="cs"))
    ok = same_bits(got, ref)
    report("zgemm cs", shape=(m, n, k), N=N, bitexact=ok, mismatches=int(np.sum(got != ref)))
    assert ok


def test_zgemm_cs_edge_cases(o2m):
    m, n, k = 40, 36, 50
    a = W.complex_matrix(m, k, 131)
    b = W.complex_matrix(k, n, 132)
    a[3, :] = 0.0
    b[:, 5] = 0.0
    a[7, :] *= 2.0 ** 900
    a[8, :] *= 2.0 ** -1060          # subnormal row: the sum of squares counts underflowed parts as 1
    a[9, :] = 0.0
    a[9, 2] = 2.0 ** -1074           # one smallest subnormal
    b[:, 9] *= 2.0 ** -600
    a[10, 4] = np.nan
    b[2, 11] = complex(np.inf, 0)
    a[12, :] = 2.0 ** 7              # the norm is exactly a power of two
    a[13, ::3] = 1e300               # huge entries next to ordinary ones
    ref = O.oq_zgemm(a, b, 16, scaling="cs")
    o2m.get_status()                                      # start clean
    got = host(o2m.zgemm_2m(to_dev(a), to_dev(b), n_moduli=16, scaling="cs"))
    assert same_bits(got, ref)
    assert np.isnan(got[10, :]).all() and np.isnan(got[:, 11]).all()
    assert o2m.get_status() == o2m.STATUS_NONFINITE       # read and cleared


def test_residue_hook_cs_exponents_and_residues(o2m):
    m, n, k, N = 37, 29, 90, 16
    a = W.complex_matrix(m, k, 151, dist="phi", phi=2.0)
    b = W.complex_matrix(k, n, 152, dist="phi", phi=2.0)
    res, E, F = o2m.zgemm_2m_residues(to_dev(a), to_dev(b), n_moduli=N, scaling="cs")
    res = res.cpu().numpy()
    E0, _, F0, _ = O.exponents(a, b, "cs")
    assert np.array_equal(E.cpu().numpy(), E0) and np.array_equal(F.cpu().numpy(), F0)
    ms = O.moduli_2m(N)
    pA, pB = O.shifts("cs", ms, k)
    ent = [(i, j) for i in range(0, m, 3) for j in range(0, n, 2)]
    for (i, j), (cr, ci) in zip(ent, O.oq_cint(a, b, pA, pB, ent, scaling="cs")):
        for l, q in enumerate(ms):
            assert int(res[l, 0, j, i]) == O.symmetric_lift(cr, q)
            assert int(res[l, 1, j, i]) == O.symmetric_lift(ci, q)


def test_cgemm_cs_bit_exact(o2m):
    a = W.complex_matrix(100, 130, 161, dist="uniform", dtype=np.complex64)
    b = W.complex_matrix(130, 90, 162, dist="uniform", dtype=np.complex64)
    ref = O.oq_cgemm(a, b, 8, scaling="cs")
    assert same_bits(host(o2m.cgemm_2m(to_dev(a), to_dev(b), n_moduli=8, scaling="cs")), ref)


@pytest.mark.parametrize("shape,N", [((100, 130), 16), ((33, 500), 22), ((257, 64), 8)])
def test_zherk_cs_bit_exact(o2m, shape, N):
    n, k = shape
    a = W.complex_matrix(n, k, 171 + n, dist="phi", phi=2.0)
    ref = O.oq_zherk(a, N, scaling="cs")
    got = host(o2m.zherk_2m(to_dev(a), n_moduli=N, scaling="cs"))
    assert same_bits(got[LOW(n)], ref[LOW(n)])


@pytest.mark.parametrize("shape,N", [((70, 65), 16), ((40, 301), 22)])
def test_dsyrk_cs_bit_exact(o2m, shape, N):
    n, k = shape
    a = W.real_matrix(n, k, 181 + k, dist="phi", phi=2.0)
    ref = O.oq_dsyrk(a, N, scaling="cs")
    got = host(o2m.dsyrk_2m(to_dev(a), n_moduli=N, scaling="cs"))
    assert same_bits(got[LOW(n)], ref[LOW(n)])


def test_cs_rule_rejected_without_valid_shifts(o2m):
    a = to_dev(W.complex_matrix(4, 8192, 1))
    b = to_dev(W.complex_matrix(8192, 4, 2))
    with pytest.raises(o2m.O2MError) as e:
        o2m.zgemm_2m(a, b, n_moduli=1, scaling="cs")
    assert e.value.status == -26


def test_cs_accuracy_curve_phi2(o2m):
    """1024^3 with phi = 2 (rows dominated by a few entries): the Cauchy-Schwarz
    rule meets 4 u k |A||B| at N = 16 and beats the max rule at every N."""
    m = n = k = 1024
    a = W.complex_matrix(m, k, 201, dist="phi", phi=2.0)
    b = W.complex_matrix(k, n, 202, dist="phi", phi=2.0)
    rng = np.random.default_rng(15)
    ent = [(int(i), int(j)) for i, j in zip(rng.integers(0, m, 1024), rng.integers(0, n, 1024))]
    hi, lo = O.dd_gemm(a, b, entries=ent)
    absab = np.array([np.sum(np.abs(a[i, :]) * np.abs(b[:, j])) for i, j in ent])
    A, B = to_dev(a), to_dev(b)
    for N in (12, 14, 16, 18):
        err = {}
        for rule in ("max", "cs"):
            C = host(o2m.zgemm_2m(A, B, n_moduli=N, scaling=rule))
            c = np.array([C[i, j] for i, j in ent])
            err[rule] = O.error_vs_reference(c, absab, hi, lo, k, 2.0 ** -53)
        report("phi=2 1024^3", N=N, max_rel=f"{err['max']['maxrel']:.3g}", cs_rel=f"{err['cs']['maxrel']:.3g}",
               cs_ratio=f"{err['cs']['ratio']:.3g}")
        assert err["cs"]["maxrel"] < err["max"]["maxrel"]
        if N >= 16:
            assert err["cs"]["ratio"] <= 1.0


# ------------------------------------------------------------ HER2K / SYR2K


H2_CASES = [((100, 130), 16, "max"), ((257, 64), 8, "max"), ((33, 500), 22, "max"), ((1, 3), 16, "max"),
            ((300, 70), 16, "cs"), ((65, 129), 20, "cs"), ((129, 66), 15, "max"), ((70, 33), 21, "cs")]


@pytest.mark.parametrize("shape,N,rule", H2_CASES, ids=[f"{c[0][0]}x{c[0][1]}-N{c[1]}-{c[2]}" for c in H2_CASES])
def test_zher2k_bit_exact_lower_triangle(o2m, shape, N, rule):
    n, k = shape
    a = W.complex_matrix(n, k, 211 + n, dist="phi", phi=1.0)
    b = W.complex_matrix(n, k, 212 + k, dist="phi", phi=1.0)
    ref = O.oq_zher2k(a, b, N, scaling=rule)
    sentinel = 3.25 - 1.5j
    out = o2m.colmajor(torch.full((n, n), sentinel, dtype=torch.complex128, device=DEV))
    o2m.zher2k_2m(to_dev(a), to_dev(b), n_moduli=N, out=out, scaling=rule)
    got = host(out)
    ok = same_bits(got[LOW(n)], ref[LOW(n)])
    report("zher2k", shape=shape, N=N, rule=rule, bitexact=ok)
    assert ok
    assert (got[~LOW(n)] == sentinel).all()
    assert (np.diag(got).imag == 0).all()


@pytest.mark.parametrize("shape,N,rule", [((100, 130), 16, "max"), ((70, 65), 16, "max"), ((257, 1), 8, "max"),
                                          ((40, 301), 22, "cs"), ((90, 64), 16, "cs")])
def test_dsyr2k_bit_exact_lower_triangle(o2m, shape, N, rule):
    n, k = shape
    a = W.real_matrix(n, k, 221 + k)
    b = W.real_matrix(n, k, 222 + n)
    ref = O.oq_dsyr2k(a, b, N, scaling=rule)
    out = o2m.colmajor(torch.full((n, n), -7.0, dtype=torch.float64, device=DEV))
    o2m.dsyr2k_2m(to_dev(a), to_dev(b), n_moduli=N, out=out, scaling=rule)
    got = host(out)
    assert same_bits(got[LOW(n)], ref[LOW(n)])
    assert (got[~LOW(n)] == -7.0).all()


def test_zher2k_edge_cases(o2m):
    n, k = 50, 70
    a = W.complex_matrix(n, k, 231)
    b = W.complex_matrix(n, k, 232)
    a[3, :] = 0.0
    b[3, :] = 0.0                    # zero row in both: zero row and column of C
    b[5, :] *= 2.0 ** 700            # the shared scale follows the larger row
    a[6, 2] = np.nan                 # non-finite in A's row 6 only
    ref = O.oq_zher2k(a, b, 16)
    got = host(o2m.zher2k_2m(to_dev(a), to_dev(b), n_moduli=16))
    low = LOW(n)
    assert same_bits(got[low], ref[low])
    assert np.isnan(got[6, :7]).all() and np.isnan(got[6:, 6]).all()


def test_zher2k_accuracy(o2m):
    n, k = 512, 1024
    a = W.complex_matrix(n, k, 241)
    b = W.complex_matrix(n, k, 242)
    got = host(o2m.zher2k_2m(to_dev(a), to_dev(b), n_moduli=16))
    rng = np.random.default_rng(16)
    ent = []
    while len(ent) < 512:
        i, j = sorted(int(x) for x in rng.integers(0, n, 2))
        ent.append((j, i))
    z = np.asfortranarray(np.hstack([a, b]))
    wh = np.asfortranarray(np.conj(np.hstack([b, a])).T)
    hi, lo = O.dd_gemm(z, wh, entries=ent)
    absab = np.array([np.sum(np.abs(z[i, :]) * np.abs(wh[:, j])) for i, j in ent])
    c = np.array([got[i, j] for i, j in ent])
    err = O.error_vs_reference(c, absab, hi, lo, 2 * k, 2.0 ** -53)
    report("zher2k 512x1024", ratio=err["ratio"], maxrel=err["maxrel"])
    assert err["ratio"] <= 1.0


# ------------------------------------------------------------ full size, sampled


def _sample(rng, m, n, count, lower=False):
    ent = [(0, 0), (m - 1, n - 1), (m - 1, 0)] + ([] if lower else [(0, n - 1)])
    while len(ent) < count:
        i, j = int(rng.integers(0, m)), int(rng.integers(0, n))
        if lower and i < j:
            i, j = j, i
        ent.append((i, j))
    return ent


@pytest.mark.slow
def test_zgemm_8192_phi2_cs_sampled(o2m):
    """8192^3, phi = 2, N = 16 under the Cauchy-Schwarz rule: sampled entries
    bit-exact and within 4 u k |A||B|."""
    m = n = k = 8192
    sa, sb = W.config_seeds(3)
    a = W.complex_matrix(m, k, sa + 10, dist="phi", phi=2.0)
    b = W.complex_matrix(k, n, sb + 10, dist="phi", phi=2.0)
    C = host(o2m.zgemm_2m(to_dev(a), to_dev(b), n_moduli=16, scaling="cs"))
    ent = _sample(np.random.default_rng(19), m, n, 40)
    got = np.array([C[i, j] for i, j in ent])
    assert same_bits(got, O.oq_zgemm(a, b, 16, entries=ent, scaling="cs"))
    hi, lo = O.dd_gemm(a, b, entries=ent)
    absab = np.array([np.sum(np.abs(a[i, :]) * np.abs(b[:, j])) for i, j in ent])
    err = O.error_vs_reference(got, absab, hi, lo, k, 2.0 ** -53)
    report("zgemm 8192^3 phi=2 cs sampled", ratio=err["ratio"], maxrel=err["maxrel"])
    assert err["ratio"] <= 1.0


@pytest.mark.slow
def test_zher2k_4096_sampled(o2m):
    """HER2K n = 4096, k = 4096 (GEMMs over k' = 8192), N = 16."""
    n = k = 4096
    a = W.complex_matrix(n, k, 251)
    b = W.complex_matrix(n, k, 252)
    C = host(o2m.zher2k_2m(to_dev(a), to_dev(b), n_moduli=16))
    ent = _sample(np.random.default_rng(20), n, n, 32, lower=True)
    got = np.array([C[i, j] for i, j in ent])
    assert same_bits(got, O.oq_zher2k(a, b, 16, entries=ent))


# ------------------------------- one pass over each operand: re-summed entries
# Rows (columns) built so that the per-chunk records of the one-pass scan do
# not settle the exponent (tests/cs_inputs.py): the library sums them again
# from the data, and everything must still equal the oracle bit for bit.


def _straddle_operands(m, n, k, dtype=np.complex128):
    from cs_inputs import straddle_vector
    a = W.complex_matrix(m, k, 191, dist="phi", phi=0.5)
    b = W.complex_matrix(k, n, 192, dist="phi", phi=0.5)
    rows = {1: "low", 4: "high", m - 1: "low"}
    cols = {0: "high", 3: "low", n - 1: "high"}
    for i, kind in rows.items():
        a[i, :] = straddle_vector(k, kind)
    for j, kind in cols.items():
        b[:, j] = straddle_vector(k, kind, exact=(0, 2048), binade=(2048, 2112), stride=2048)
    return a.astype(dtype), b.astype(dtype), rows, cols


def test_cs_resummed_entries_exponents_and_zgemm(o2m):
    m, n, k, N = 40, 36, 4096, 16
    a, b, rows, cols = _straddle_operands(m, n, k)
    _, E, F = o2m.zgemm_2m_residues(to_dev(a), to_dev(b), n_moduli=N, scaling="cs")
    E0, _, F0, _ = O.exponents(a, b, "cs")
    E, F = E.cpu().numpy(), F.cpu().numpy()
    for i in rows:
        assert E0[i] == O.cs_exponent_exact(a[i, :])
    for j in cols:
        assert F0[j] == O.cs_exponent_exact(b[:, j])
    ok_e = np.array_equal(E, E0) and np.array_equal(F, F0)
    ref = O.oq_zgemm(a, b, N, scaling="cs")
    got = host(o2m.zgemm_2m(to_dev(a), to_dev(b), n_moduli=N, scaling="cs"))
    ok = same_bits(got, ref)
    report("cs re-summed zgemm", shape=(m, n, k), exponents=ok_e, bitexact=ok)
    assert ok_e and ok


def test_cs_resummed_entries_cgemm(o2m):
    a, b, _, _ = _straddle_operands(24, 20, 4096, np.complex64)
    ref = O.oq_cgemm(a, b, 8, scaling="cs")
    assert same_bits(host(o2m.cgemm_2m(to_dev(a), to_dev(b), n_moduli=8, scaling="cs")), ref)


def test_cs_resummed_rows_symmetric_calls(o2m):
    from cs_inputs import straddle_vector
    n, k, N = 30, 700, 16
    a = W.complex_matrix(n, k, 193, dist="phi", phi=2.0)
    b = W.complex_matrix(n, k, 194, dist="phi", phi=2.0)
    for i, kind in ((0, "low"), (7, "high"), (n - 1, "high")):
        a[i, :] = straddle_vector(k, kind)
        b[i, :] = 0.0                 # rank-2k: the row of [A | B] is A's
    ref = O.oq_zherk(a, N, scaling="cs")
    got = host(o2m.zherk_2m(to_dev(a), n_moduli=N, scaling="cs"))
    assert same_bits(got[LOW(n)], ref[LOW(n)])
    ref = O.oq_zher2k(a, b, N, scaling="cs")
    got = host(o2m.zher2k_2m(to_dev(a), to_dev(b), n_moduli=N, scaling="cs"))
    assert same_bits(got[LOW(n)], ref[LOW(n)])
    r = W.real_matrix(n, k, 195, dist="phi", phi=2.0)
    for i, kind in ((2, "low"), (5, "high")):
        r[i, :] = straddle_vector(k, kind, complex_=False)
    ref = O.oq_dsyrk(r, N, scaling="cs")
    got = host(o2m.dsyrk_2m(to_dev(r), n_moduli=N, scaling="cs"))
    assert same_bits(got[LOW(n)], ref[LOW(n)])


@pytest.mark.slow
def test_cs_k_at_the_int32_limit_sampled(o2m):
    """k = 149130 under the Cauchy-Schwarz rule: 1166 chunk records per row of
    A, 73 per column of B, rows and columns among them that the records leave
    open; exponents equal the oracle's, sampled entries bit-exact."""
    from cs_inputs import straddle_vector
    m, n, k, N = 256, 300, 149130, 16
    a = W.complex_matrix(m, k, 441, dist="phi", phi=2.0)
    b = W.complex_matrix(k, n, 442, dist="phi", phi=2.0)
    a[17, :] = straddle_vector(k, "low")
    a[m - 1, :] = straddle_vector(k, "high")
    b[:, 5] = straddle_vector(k, "high", exact=(0, 2048), binade=(2048, 2112), stride=2048)
    _, E, F = o2m.zgemm_2m_residues(to_dev(a), to_dev(b), n_moduli=N, scaling="cs")
    E0, _, F0, _ = O.exponents(a, b, "cs")
    assert np.array_equal(E.cpu().numpy(), E0) and np.array_equal(F.cpu().numpy(), F0)
    C = host(o2m.zgemm_2m(to_dev(a), to_dev(b), n_moduli=N, scaling="cs"))
    rng = np.random.default_rng(27)
    ent = [(0, 0), (m - 1, n - 1), (17, 5), (m - 1, 5)]
    ent += [(int(i), int(j)) for i, j in zip(rng.integers(0, m, 28), rng.integers(0, n, 28))]
    got = np.array([C[i, j] for i, j in ent])
    ok = same_bits(got, O.oq_zgemm(a, b, N, entries=ent, scaling="cs"))
    report("cs k=149130", bitexact=ok)
    assert ok


# ------------------------------------------------------------ upper triangles
# uplo 'U': the symmetric calls write the upper triangle (the mirrored tile
# pairs of the CRT kernel), leave the strictly lower one untouched, and give
# the same exact values as the lower triangle (c_ji = conj(c_ij)).

UP = lambda n: np.triu(np.ones((n, n), dtype=bool))


@pytest.mark.parametrize("rule", ["max", "cs"])
@pytest.mark.parametrize("n,k", [(77, 130), (300, 65)])
def test_symmetric_calls_upper_triangle(o2m, n, k, rule):
    N = 16
    a = W.complex_matrix(n, k, 5301 + n, dist="phi", phi=2.0)
    b = W.complex_matrix(n, k, 5302 + n, dist="phi", phi=2.0)
    r, s = W.real_matrix(n, k, 5303 + n, dist="phi", phi=2.0), W.real_matrix(n, k, 5304 + n)
    up, low = UP(n), ~UP(n)
    zc = 7.5 - 2.5j

    def check(name, call, ref, sentinel, dtype):
        C = o2m.colmajor(torch.full((n, n), sentinel, dtype=dtype, device=DEV))
        call(C, "U")
        got = host(C)
        ok = same_bits(got[up], ref[up]) and bool((got[low] == sentinel).all())
        lower = host(call(o2m.colmajor(torch.zeros((n, n), dtype=dtype, device=DEV)), "L"))
        mirror = np.array_equal(np.conj(lower.T)[up], got[up])      # values: -0 and +0 compare equal
        report("upper", op=name, n=n, k=k, rule=rule, bitexact=ok, mirror=mirror)
        assert ok and mirror
        if np.iscomplexobj(got):
            assert (np.diag(got).imag == 0).all()

    check("zherk", lambda C, u: o2m.zherk_2m(to_dev(a), n_moduli=N, out=C, scaling=rule, uplo=u),
          O.oq_zherk(a, N, scaling=rule), zc, torch.complex128)
    check("zher2k", lambda C, u: o2m.zher2k_2m(to_dev(a), to_dev(b), n_moduli=N, out=C, scaling=rule, uplo=u),
          O.oq_zher2k(a, b, N, scaling=rule), zc, torch.complex128)
    check("dsyrk", lambda C, u: o2m.dsyrk_2m(to_dev(r), n_moduli=N, out=C, scaling=rule, uplo=u),
          O.oq_dsyrk(r, N, scaling=rule), -3.25, torch.float64)
    check("dsyr2k", lambda C, u: o2m.dsyr2k_2m(to_dev(r), to_dev(s), n_moduli=N, out=C, scaling=rule, uplo=u),
          O.oq_dsyr2k(r, s, N, scaling=rule), -3.25, torch.float64)
