"""GPU parity of hybrid 2M/3M moduli sets (Section 3.2: beyond the 22 2M moduli,
3M per modulus) with the CPU oracle, through the C-ABI: bit-exact results,
exact per-modulus residues, and the accuracy the extra moduli buy."""
import os

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
    print(f"[hybrid] {name} " + " ".join(f"{k}={v}" for k, v in kw.items()), flush=True)


CASES = [
    # m, n, k, dist, phi, N, rule
    (64, 64, 64, "normal", 0.5, 23, "max"),
    (100, 77, 130, "phi", 2.0, 24, "max"),
    (257, 300, 200, "phi", 4.0, 27, "max"),
    (33, 47, 65, "normal", 0.5, 32, "max"),
    (70, 90, 300, "phi", 2.0, 25, "cs"),
    (5, 3, 1, "normal", 0.5, 32, "cs"),
    # quantized values beyond 2^88: four base-2^26 digits (pA, pB 98..106),
    # then five (pA 110); their residues are computed by two waves per fragment
    (257, 130, 300, "phi", 2.0, 29, "max"),
    (130, 301, 1000, "normal", 0.5, 31, "max"),
    (200, 150, 130, "phi", 2.0, 32, "max"),
]


@pytest.mark.parametrize("case", CASES, ids=[f"{c[0]}x{c[1]}x{c[2]}-N{c[5]}-{c[6]}" for c in CASES])
def test_zgemm_hybrid_bit_exact(o2m, case):
    m, n, k, dist, phi, N, rule = case
    a = W.complex_matrix(m, k, 5000 + m, dist=dist, phi=phi)
    b = W.complex_matrix(k, n, 6000 + n, dist=dist, phi=phi)
    ref = O.oq_zgemm(a, b, N, scaling=rule)
    got = host(o2m.zgemm_2m(to_dev(a), to_dev(b), n_moduli=N, scaling=rule))
    ok = same_bits(got, ref)
    report("zgemm", shape=(m, n, k), N=N, rule=rule, bitexact=ok, mismatches=int(np.sum(got != ref)))
    assert ok


def test_moduli_reported(o2m):
    ms, ss, l2 = o2m.moduli(32)
    assert ms == O.moduli_set(32)
    assert ss[22:] == [0] * 10
    assert abs(l2 - np.log2(float(O.product(ms)))) < 1e-6


def test_residue_hook_hybrid(o2m):
    m, n, k, N = 37, 29, 90, 26
    a = W.complex_matrix(m, k, 301, dist="phi", phi=2.0)
    b = W.complex_matrix(k, n, 302, dist="phi", phi=2.0)
    res, E, F = o2m.zgemm_2m_residues(to_dev(a), to_dev(b), n_moduli=N)
    res = res.cpu().numpy()
    ms = O.moduli_set(N)
    pA, pB = O.shifts("max", ms, k)
    ent = [(i, j) for i in range(0, m, 3) for j in range(0, n, 2)]

    def sym(v, q):  # the symmetric representative, [-(q-1)/2, (q-1)/2] or [-q/2, q/2 - 1]
        r = v % q
        return r - q if r > (q - 1) // 2 else r

    for (i, j), (cr, ci) in zip(ent, O.oq_cint(a, b, pA, pB, ent)):
        for l, q in enumerate(ms):
            assert int(res[l, 0, j, i]) == sym(cr, q), (l, q)
            assert int(res[l, 1, j, i]) == sym(ci, q), (l, q)


def test_cgemm_hybrid_bit_exact(o2m):
    a = W.complex_matrix(100, 130, 311, dist="uniform", dtype=np.complex64)
    b = W.complex_matrix(130, 90, 312, dist="uniform", dtype=np.complex64)
    ref = O.oq_cgemm(a, b, 24)
    assert same_bits(host(o2m.cgemm_2m(to_dev(a), to_dev(b), n_moduli=24)), ref)


def test_symmetric_calls_reject_hybrid_sets(o2m):
    a = to_dev(W.complex_matrix(8, 8, 1))
    with pytest.raises(o2m.O2MError) as e:
        o2m.zherk_2m(a, n_moduli=23)
    assert e.value.status == -20


def test_hybrid_recovers_wide_exponent_span(o2m):
    """Rows of A hold one entry 2^40 times the others, facing a zero row of B:
    22 moduli leave the small entries too few bits for the tolerance, the 3M
    extension to 30 moduli restores it (as the oracle predicts)."""
    m, n, k = 256, 256, 512
    a = W.complex_matrix(m, k, 321)
    b = W.complex_matrix(k, n, 322)
    a[:, 0] = 2.0 ** 40
    b[0, :] = 0.0
    rng = np.random.default_rng(23)
    ent = [(int(i), int(j)) for i, j in zip(rng.integers(0, m, 512), rng.integers(0, n, 512))]
    hi, lo = O.dd_gemm(a, b, entries=ent)
    absab = np.array([np.sum(np.abs(a[i, :]) * np.abs(b[:, j])) for i, j in ent])
    A, B = to_dev(a), to_dev(b)
    err = {}
    for N in (22, 26, 30):
        C = host(o2m.zgemm_2m(A, B, n_moduli=N))
        c = np.array([C[i, j] for i, j in ent])
        assert same_bits(c, O.oq_zgemm(a, b, N, entries=ent))
        err[N] = O.error_vs_reference(c, absab, hi, lo, k, 2.0 ** -53)
        report("wide span", N=N, ratio=f"{err[N]['ratio']:.3g}", maxrel=f"{err[N]['maxrel']:.3g}")
    assert err[22]["ratio"] > 1.0 and err[30]["ratio"] <= 1.0
    assert err[22]["maxrel"] > err[26]["maxrel"] > err[30]["maxrel"]


@pytest.mark.slow
def test_hybrid_k_limit_sampled(o2m):
    """k = 131071 (the largest k with residues mod 256), N = 23: the longest
    k-loop with the widest residues, on sampled entries."""
    m, n, k = 256, 512, 131071
    a = W.complex_matrix(m, k, 331)
    b = W.complex_matrix(k, n, 332)
    C = host(o2m.zgemm_2m(to_dev(a), to_dev(b), n_moduli=23))
    rng = np.random.default_rng(24)
    ent = [(0, 0), (m - 1, n - 1)] + [(int(i), int(j)) for i, j in zip(rng.integers(0, m, 30), rng.integers(0, n, 30))]
    got = np.array([C[i, j] for i, j in ent])
    assert same_bits(got, O.oq_zgemm(a, b, 23, entries=ent))


@pytest.mark.slow
def test_zgemm_8192_hybrid_sampled(o2m):
    """The benchmark shape with N = 26 (hybrid): sampled entries bit-exact."""
    m = n = k = 8192
    sa, sb = W.config_seeds(3)
    a = W.complex_matrix(m, k, sa, dist="phi", phi=2.0)
    b = W.complex_matrix(k, n, sb, dist="phi", phi=2.0)
    C = host(o2m.zgemm_2m(to_dev(a), to_dev(b), n_moduli=26))
    rng = np.random.default_rng(25)
    ent = [(0, 0), (m - 1, n - 1), (m - 1, 0), (0, n - 1)]
    ent += [(int(i), int(j)) for i, j in zip(rng.integers(0, m, 28), rng.integers(0, n, 28))]
    got = np.array([C[i, j] for i, j in ent])
    assert same_bits(got, O.oq_zgemm(a, b, 26, entries=ent))


@pytest.mark.slow
def test_randomized_configurations(o2m):
    """Seeded random combinations of call, shape, moduli count, scaling rule and
    input distribution, each bit-exact against the oracle (a sweep over the
    corners the fixed cases do not combine).  O2M_RANDOM_CASES and
    O2M_RANDOM_SEED widen the sweep (default: 36 cases, seed 2609);
    O2M_RANDOM_TALL=1 draws m up to 1300 (several 256-row waves of the CRT's
    row-order stores, several 128 x 128 super-tiles of the symmetric CRT) with
    n and k up to 200 instead of all three up to 300.  A second generator
    draws the operand layout (op(A), op(B) of the GEMMs, the triangle of the
    symmetric calls), so the first one's cases stay those of earlier sweeps."""
    seed0 = int(os.environ.get("O2M_RANDOM_SEED", "2609"))
    rng = np.random.default_rng(seed0)
    lay = np.random.default_rng(seed0 + 1)
    tall = os.environ.get("O2M_RANDOM_TALL") == "1"
    ops = ["zgemm", "cgemm", "zherk", "dsyrk", "zher2k", "dsyr2k"]
    tri = lambda n, u: np.triu(np.ones((n, n), dtype=bool)) if u == "U" else np.tril(np.ones((n, n), dtype=bool))
    stored = lambda x, t: x if t == "N" else (x.T if t == "T" else x.conj().T)
    for case in range(int(os.environ.get("O2M_RANDOM_CASES", "36"))):
        op = ops[case % len(ops)]
        sym = op not in ("zgemm", "cgemm")
        N = int(rng.integers(1, 23 if sym else 33))
        rule = "cs" if rng.random() < 0.5 else "max"
        if tall:
            m = int(rng.integers(1, 1300))
            n, k = (int(x) for x in rng.integers(1, 200, 2))
        else:
            m, n, k = (int(x) for x in rng.integers(1, 300, 3))
        k = max(1, k)
        if rule == "cs" and O.budget_cs(O.moduli_set(N), 2 * k if op in ("zher2k", "dsyr2k") else k, sym) is None:
            rule = "max"
        dist = ["normal", "uniform", "phi"][int(rng.integers(0, 3))]
        phi = float(rng.choice([0.5, 2.0, 4.0]))
        seed = 9000 + case
        ta, tb = (str(x) for x in lay.choice(list("NTC"), 2))
        up = str(lay.choice(["L", "U"]))
        print(f"[hybrid] random case {case}: {op} m={m} n={n} k={k} N={N} {rule} {dist} "
              + (f"op={ta}{tb}" if not sym else f"uplo={up}"), flush=True)
        if op in ("zgemm", "cgemm"):
            dt = np.complex128 if op == "zgemm" else np.complex64
            a = W.complex_matrix(m, k, seed, dist=dist, phi=phi, dtype=dt)
            b = W.complex_matrix(k, n, seed + 1, dist=dist, phi=phi, dtype=dt)
            fn = o2m.zgemm_2m_op if op == "zgemm" else o2m.cgemm_2m_op
            ofn = O.oq_zgemm if op == "zgemm" else O.oq_cgemm
            A = to_dev(np.ascontiguousarray(stored(a, ta)))
            B = to_dev(np.ascontiguousarray(stored(b, tb)))
            got = host(fn(A, B, ta, tb, n_moduli=N, scaling=rule))
            assert same_bits(got, ofn(a, b, N, scaling=rule)), case
        elif op in ("zherk", "zher2k"):
            a = W.complex_matrix(m, k, seed, dist=dist, phi=phi)
            if op == "zherk":
                got = host(o2m.zherk_2m(to_dev(a), n_moduli=N, scaling=rule, uplo=up))
                ref = O.oq_zherk(a, N, scaling=rule)
            else:
                b = W.complex_matrix(m, k, seed + 1, dist=dist, phi=phi)
                got = host(o2m.zher2k_2m(to_dev(a), to_dev(b), n_moduli=N, scaling=rule, uplo=up))
                ref = O.oq_zher2k(a, b, N, scaling=rule)
            assert same_bits(got[tri(m, up)], ref[tri(m, up)]), case
        else:
            a = W.real_matrix(m, k, seed, dist=dist, phi=phi)
            if op == "dsyrk":
                got = host(o2m.dsyrk_2m(to_dev(a), n_moduli=N, scaling=rule, uplo=up))
                ref = O.oq_dsyrk(a, N, scaling=rule)
            else:
                b = W.real_matrix(m, k, seed + 1, dist=dist, phi=phi)
                got = host(o2m.dsyr2k_2m(to_dev(a), to_dev(b), n_moduli=N, scaling=rule, uplo=up))
                ref = O.oq_dsyr2k(a, b, N, scaling=rule)
            assert same_bits(got[tri(m, up)], ref[tri(m, up)]), case
