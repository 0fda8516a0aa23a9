"""Step 7 on the GPU (through the C-ABI): each output component is the exact
scaled integer product rounded once into the output type.  Inputs hold rows
and columns whose quantized product is a double-rounding tie (rounding to fp64
first, then to fp32 or to the fp64 subnormal grid, would give another value),
embedded in random matrices; whole outputs are compared bit for bit with the
oracle, and the tie entries with their hand-derived values."""
import numpy as np
import pytest

import oracle as O
import workloads as W
from conftest import same_bits
from test_oracle_rounding import subnormal_f32_exponents, tie_operands

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


def embed(m, n, k, seed, dtype, ties):
    """Random m x k and k x n matrices with tie rows / columns planted:
    ties = [(row, col, a_row, b_col)]."""
    a = W.complex_matrix(m, k, seed, dist="uniform", dtype=dtype)
    b = W.complex_matrix(k, n, seed + 1, dist="uniform", dtype=dtype)
    for i, j, ar, bc in ties:
        a[i, :] = ar[0, :]
        b[:, j] = bc[:, 0]
    return np.asfortranarray(a), np.asfortranarray(b)


@pytest.mark.parametrize("N,k", [(8, 4), (8, 300), (12, 64), (20, 16), (26, 8)])
def test_cgemm_rounds_ties_once(o2m, N, k):
    pA, pB = O.shifts("max", O.moduli_set(N), k)
    L, j = pA + pB - 1, 24
    sc = 4 - pA - pB
    a1, b1 = tie_operands(pA, pB, 2, 2, j, k)
    a2, _ = tie_operands(pA, pB, 2, 2, j, k, imag=True, negate=True)
    ties = [(5, 7, a1, b1), (9, 7, a2, b1)]
    sub = pA + pB <= 149 + 20            # an fp32-subnormal tie has representable inputs
    if sub:
        ps, pf = subnormal_f32_exponents(pA, pB, 20)
        a3, b3 = tie_operands(pA, pB, ps, pf, 20, k)
        ties.append((30, 33, a3, b3))
    a, b = embed(70, 40, k, 900 + N, np.complex64, ties)
    print(f"[rounding] cgemm ties N={N} k={k}", flush=True)
    got = host(o2m.cgemm_2m(to_dev(a), to_dev(b), n_moduli=N))
    ref = O.oq_cgemm(a, b, N)
    assert same_bits(got, ref)
    want = 2.0 ** (L + sc) + 2.0 ** (L - j + 1 + sc)
    assert float(got[5, 7].real) == want and float(got[9, 7].imag) == -want
    if sub:
        assert float(got[30, 33].real) == 2.0 ** -130 + 2.0 ** -149


@pytest.mark.parametrize("N,k", [(8, 4), (16, 64), (22, 10), (26, 8)])
def test_zgemm_subnormal_ties_once(o2m, N, k):
    pA, pB = O.shifts("max", O.moduli_set(N), k)
    j, E = 30, -522
    F = j - 1074 - E
    a1, b1 = tie_operands(pA, pB, E, F, j, k, negate=True)
    a, b = embed(50, 40, k, 700 + N, np.complex128, [(3, 11, a1, b1)])
    a[7, :] *= 2.0 ** -1000               # more subnormal outputs in row 7
    print(f"[rounding] zgemm subnormal ties N={N} k={k}", flush=True)
    got = host(o2m.zgemm_2m(to_dev(a), to_dev(b), n_moduli=N))
    assert same_bits(got, O.oq_zgemm(a, b, N))
    assert got[3, 11].real == -(2.0 ** (j - 1075) + 2.0 ** -1074)
    assert (np.abs(got[7, :].real) < 2.0 ** -1022).any()


@pytest.mark.parametrize("N", [16, 22])
@pytest.mark.parametrize("sign", [1.0, -1.0])
def test_zgemm_normal_boundary_rounds_once(o2m, N, sign):
    """An exact product just below 2^-1022, (2^57 - 17) 2^-1079, whose 53-bit
    rounding (2^53 - 1) 2^-1075 ties on the subnormal grid: scaling that value
    would give 2^-1022, the one rounding gives the largest subnormal."""
    k = 2
    pA, _ = O.shifts("max", O.moduli_set(N), k)
    assert pA >= 57                         # every entry below quantizes exactly
    ar = np.array([[sign * (2 ** 53 - 1) * 2.0 ** -540, -sign * 2.0 ** -544]], dtype=np.complex128)
    bc = np.array([[2.0 ** -535], [2.0 ** -535]], dtype=np.complex128)
    a, b = embed(40, 30, k, 900 + N, np.complex128, [(5, 7, ar, bc)])
    print(f"[rounding] zgemm normal boundary N={N} sign={sign}", flush=True)
    got = host(o2m.zgemm_2m(to_dev(a), to_dev(b), n_moduli=N))
    assert same_bits(got, O.oq_zgemm(a, b, N))
    assert got[5, 7].real == sign * (2.0 ** -1022 - 2.0 ** -1074)


@pytest.mark.parametrize("N", [16, 22])
def test_symmetric_normal_boundary_rounds_once(o2m, N):
    """The same tie through the symmetric CRT: with row 0 = [b, b] and row 1 =
    [a1, a2], entry (1, 0) of A A^H (and of the real A A^T, whose half-k
    complex form has z_i = a_i0 + i a_i1) is (a1 + a2) b."""
    rng = np.random.default_rng(950 + N)
    a = rng.standard_normal((6, 2))
    a[0, :] = 2.0 ** -535
    a[1, 0], a[1, 1] = (2 ** 53 - 1) * 2.0 ** -540, -(2.0 ** -544)
    a = np.asfortranarray(a)
    low = np.tril(np.ones((6, 6), dtype=bool))
    want = 2.0 ** -1022 - 2.0 ** -1074
    print(f"[rounding] zherk / dsyrk normal boundary N={N}", flush=True)
    ac = np.asfortranarray(a.astype(np.complex128))
    got = host(o2m.zherk_2m(to_dev(ac), n_moduli=N))
    assert same_bits(got[low], O.oq_zherk(ac, N)[low])
    assert got[1, 0].real == want
    got = host(o2m.dsyrk_2m(to_dev(a), n_moduli=N))
    assert same_bits(got[low], O.oq_dsyrk(a, N)[low])
    assert got[1, 0] == want


@pytest.mark.parametrize("N", [8, 16, 20])
def test_zherk_subnormal_outputs(o2m, N):
    n, k = 60, 40
    a = W.complex_matrix(n, k, 555 + N)
    a[4, :] *= 2.0 ** -540                # rows 4 x 5: products near 2^-1080..2^-1060
    a[5, :] *= 2.0 ** -525
    print(f"[rounding] zherk subnormal N={N}", flush=True)
    out = host(o2m.zherk_2m(to_dev(a), n_moduli=N))
    ref = O.oq_zherk(a, N)
    low = np.tril(np.ones((n, n), dtype=bool))
    assert same_bits(out[low], ref[low])
    assert 0 < abs(out[5, 4].real) < 2.0 ** -1022
