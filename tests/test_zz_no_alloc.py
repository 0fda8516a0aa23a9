"""zgemm_2m_noalloc: the ZGEMM entry point that allocates no device memory
(its scratch buffers live in a static device array per GPU), called through
the C-ABI and compared bit for bit with zgemm_2m_ex on the same inputs, on
two calls in a row (the second smaller, so it runs on what the first left in
the array), against sampled oracle entries, under graph capture on a stream
that never had a workspace, and with a size beyond the array."""
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


def nan_out(o2m, m, n):
    return o2m.colmajor(torch.full((m, n), complex(np.nan, np.nan), dtype=torch.complex128, device=DEV))


def sample(rng, m, n, count):
    ent = [(0, 0), (m - 1, n - 1), (m - 1, 0), (0, n - 1)]
    while len(ent) < count:
        ent.append((int(rng.integers(0, m)), int(rng.integers(0, n))))
    return ent


def test_noalloc_equals_zgemm_2m_ex_on_two_calls(o2m):
    rng = np.random.default_rng(77)
    cases = [(1000, 900, 1100, 16, "max", 6101), (300, 200, 500, 12, "cs", 6103)]   # second call smaller
    for m, n, k, N, rule, seed in cases:
        print(f"[noalloc] zgemm_2m_noalloc {m}x{n}x{k} N={N} rule={rule}", flush=True)
        assert o2m.workspace_bytes("z", m, n, k, N) <= o2m.NOALLOC_SCRATCH_BYTES
        a = W.complex_matrix(m, k, seed, dist="phi", phi=0.5)
        b = W.complex_matrix(k, n, seed + 1, dist="phi", phi=0.5)
        A, B = to_dev(a), to_dev(b)
        C = nan_out(o2m, m, n)
        o2m.zgemm_2m_noalloc(A, B, C, n_moduli=N, scaling=rule)
        got = host(C)
        ref = host(o2m.zgemm_2m(A, B, n_moduli=N, scaling=rule))
        assert same_bits(got, ref)
        ent = sample(rng, m, n, 200)
        assert same_bits(np.array([got[i, j] for i, j in ent]), O.oq_zgemm(a, b, N, entries=ent, scaling=rule))


def test_noalloc_in_a_graph_on_a_fresh_stream(o2m):
    """Captured on a stream that never had a workspace (a zgemm_2m call there
    would be refused under capture): the call needs no allocation and no
    synchronisation.  Three replays on fresh inputs, eager work and a
    synchronisation between them, each bit-identical to zgemm_2m_ex."""
    m, n, k, N = 260, 300, 333, 16
    A = o2m.colmajor(torch.zeros((m, k), dtype=torch.complex128, device=DEV))
    B = o2m.colmajor(torch.zeros((k, n), dtype=torch.complex128, device=DEV))
    C = nan_out(o2m, m, n)
    o2m.zgemm_2m_noalloc(A, B, C, n_moduli=N)         # the device's scratch address is known
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        o2m.zgemm_2m_noalloc(A, B, C, n_moduli=N)
    for seed in (6201, 6203, 6205):
        print(f"[noalloc] graph replay seed={seed}", flush=True)
        a = W.complex_matrix(m, k, seed, dist="phi", phi=2.0)
        b = W.complex_matrix(k, n, seed + 1, dist="phi", phi=2.0)
        A.copy_(to_dev(a))
        B.copy_(to_dev(b))
        torch.cuda.synchronize()
        g.replay()
        got = host(C)
        assert same_bits(got, host(o2m.zgemm_2m(A, B, n_moduli=N)))
    del g


def test_noalloc_rejects_calls_beyond_the_array(o2m):
    m = n = k = 2048
    N = 16
    assert o2m.workspace_bytes("z", m, n, k, N) > o2m.NOALLOC_SCRATCH_BYTES
    A = o2m.colmajor(torch.zeros((m, k), dtype=torch.complex128, device=DEV))
    C = nan_out(o2m, m, n)
    with pytest.raises(o2m.O2MError) as e:
        o2m.zgemm_2m_noalloc(A, A, C, n_moduli=N)
    assert e.value.status == -27
    assert torch.isnan(C).all()                           # nothing was enqueued
    # argument errors come first, as for zgemm_2m
    with pytest.raises(o2m.O2MError) as e:
        o2m.zgemm_2m_noalloc(A, A, C, n_moduli=33)
    assert e.value.status == -20
