"""The C-ABI library loads, exports every symbol include/o2m.h declares, and
its host-only parts (tables, budget, workspace sizes, argument checks) agree
with the oracle and the header (no GPU: no compute call is made)."""
import ctypes
import os
import re

import pytest

import oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "o2m.h")
LIB = os.path.join(ROOT, "paper_2609_05419_amd", "libo2m.so")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:o2m_status|size_t|int|const char \*)\s*(\w+)\s*\(", text, flags=re.M)
    return sorted(set(names))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        pytest.skip("libo2m.so not built")
    return ctypes.CDLL(LIB)


def test_header_declares_the_entry_points():
    names = declared_functions()
    for f in ("zgemm_2m", "cgemm_2m", "zherk_2m", "dsyrk_2m", "gauss_gemm_2m", "zgemm_2m_residues",
              "o2m_moduli", "o2m_budget", "o2m_workspace_bytes", "o2m_set_workspace",
              "o2m_release_workspace", "o2m_get_status", "o2m_phase_timing", "o2m_phase_times", "o2m_status_string"):
        assert f in names


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_package_binding_loads():
    import paper_2609_05419_amd as o2m
    assert os.path.samefile(o2m.LIB_PATH, LIB)


def test_moduli_table_matches_oracle():
    import paper_2609_05419_amd as o2m
    for n in (1, 4, 8, 16, 22, 23, 27, 32):
        ms, ss, l2 = o2m.moduli(n)
        assert ms == O.moduli_set(n)
        assert ss == [O.root_of(q) if O.is_2m_modulus(q) else 0 for q in ms]
        assert abs(l2 - __import__("math").log2(O.product(ms))) < 1e-9
    with pytest.raises(o2m.O2MError):
        o2m.moduli(33)


def test_budget_matches_oracle():
    import paper_2609_05419_amd as o2m
    for n in (1, 2, 3, 4, 5, 8, 12, 16, 17, 20, 22, 23, 26, 29, 32):
        for k in (0, 1, 2, 7, 64, 1000, 1024, 8192, 16384, 65536, 131071, 149130):
            assert o2m.budget(n, k) == O.budget(O.moduli_set(n), k), (n, k)


def test_workspace_bytes_grow_with_the_problem():
    import paper_2609_05419_amd as o2m
    z = o2m.workspace_bytes("z", 8192, 8192, 8192, 16)
    # planes: 2N (m + n) k + 2N m n bytes, plus exponents and the
    # Cauchy-Schwarz chunk records: 24 bytes per operand row and chunk, with
    # room for either layout of each GEMM operand (rows of a column-major
    # matrix: chunks of 128 columns; columns: chunks of 2048 rows)
    records = 24 * (8192 * (8192 // 128) + 8192 * (8192 // 128))
    assert z >= 32 * (8192 * 8192 * 3) + records
    assert z < 32 * (8192 * 8192 * 3) + records + (1 << 20)
    h = o2m.workspace_bytes("h", 8192, 8192, 8192, 16)
    assert h < z
    s = o2m.workspace_bytes("s", 8192, 8192, 8192, 16)
    assert s < h
    assert o2m.workspace_bytes("z", 8192, 8192, 8192, 33) == 0
    assert o2m.workspace_bytes("h", 8192, 8192, 8192, 23) == 0
    # hybrid: 2 planes per 2M modulus and 3 per 3M modulus, on each side
    z24 = o2m.workspace_bytes("z", 8192, 8192, 8192, 24)
    assert z24 >= (2 * 22 + 3 * 2) * (8192 * 8192 * 3)


def test_argument_errors_are_reported_before_any_gpu_work(lib):
    P = ctypes.c_void_p
    lib.zgemm_2m.argtypes = [ctypes.c_int] * 3 + [P, ctypes.c_int, P, ctypes.c_int, P, ctypes.c_int, ctypes.c_int, P]
    fake = P(0x1000)
    call = lambda *a: lib.zgemm_2m(*a)
    assert call(-1, 4, 4, fake, 4, fake, 4, fake, 4, 16, None) == -1
    assert call(4, -1, 4, fake, 4, fake, 4, fake, 4, 16, None) == -2
    assert call(4, 4, -1, fake, 4, fake, 4, fake, 4, 16, None) == -3
    assert call(4, 4, 4, None, 4, fake, 4, fake, 4, 16, None) == -4
    assert call(4, 4, 4, fake, 3, fake, 4, fake, 4, 16, None) == -5
    assert call(4, 4, 4, fake, 4, None, 4, fake, 4, 16, None) == -6
    assert call(4, 4, 4, fake, 4, fake, 3, fake, 4, 16, None) == -7
    assert call(4, 4, 4, fake, 4, fake, 4, None, 4, 16, None) == -8
    assert call(4, 4, 4, fake, 4, fake, 4, fake, 3, 16, None) == -9
    assert call(4, 4, 4, fake, 4, fake, 4, fake, 4, 0, None) == -20
    assert call(4, 4, 4, fake, 4, fake, 4, fake, 4, 33, None) == -20
    assert call(4, 4, 149131, fake, 4, fake, 149131, fake, 4, 16, None) == -21
    assert call(4, 4, 131072, fake, 4, fake, 131072, fake, 4, 23, None) == -21   # hybrid k limit
    # empty outputs are a no-op that touches nothing
    assert call(0, 4, 4, None, 1, fake, 4, fake, 1, 16, None) == 0
    assert call(4, 0, 4, fake, 4, fake, 4, None, 4, 16, None) == 0
    lib.gauss_gemm_2m.argtypes = lib.zgemm_2m.argtypes
    assert lib.gauss_gemm_2m(4, 4, 4, fake, 4, fake, 4, fake, 4, 9, None) == -20
    lib.zherk_2m.argtypes = [ctypes.c_char, ctypes.c_int, ctypes.c_int, P, ctypes.c_int, P, ctypes.c_int, ctypes.c_int, P]
    assert lib.zherk_2m(b"X", 4, 4, fake, 4, fake, 4, 16, None) == -1
    assert lib.zherk_2m(b"L", 4, 4, fake, 4, fake, 4, 23, None) == -20    # symmetric calls: 2M only
    assert lib.zherk_2m(b"L", 4, 4, fake, 3, fake, 4, 16, None) == -5
    assert lib.zherk_2m(b"L", 0, 4, None, 1, None, 1, 16, None) == 0
    lib.o2m_status_string.restype = ctypes.c_char_p
    assert b"n_moduli" in lib.o2m_status_string(-20)


def test_new_entry_points_declared():
    names = declared_functions()
    for f in ("zher2k_2m", "dsyr2k_2m", "zgemm_2m_ex", "cgemm_2m_ex", "zherk_2m_ex", "dsyrk_2m_ex",
              "zher2k_2m_ex", "dsyr2k_2m_ex", "zgemm_2m_residues_ex", "o2m_shifts", "zgemm_2m_op", "cgemm_2m_op"):
        assert f in names


@pytest.mark.parametrize("scaling", ["max", "cs"])
def test_shifts_match_oracle(scaling):
    import paper_2609_05419_amd as o2m
    for n in (1, 2, 3, 4, 8, 12, 16, 17, 20, 22, 23, 28, 32):
        ms = O.moduli_set(n)
        for k in (0, 1, 2, 7, 64, 1000, 8192, 16384, 65536, 74565, 149130):
            cases = {"z": (k, False), "c": (k, False), "r": (k, False), "h": (k, True),
                     "s": ((k + 1) // 2, True), "x": (2 * k, True), "y": (2 * ((k + 1) // 2), True)}
            for op, (kin, sym) in cases.items():
                if sym and n > 22:
                    with pytest.raises(o2m.O2MError) as e:
                        o2m.shifts(op, n, k, scaling)
                    assert e.value.status == -20
                    continue
                try:
                    want = O.shifts(scaling, ms, kin, sym)
                except ValueError:
                    want = None
                if want is None:
                    with pytest.raises(o2m.O2MError) as e:
                        o2m.shifts(op, n, k, scaling)
                    assert e.value.status == -26
                else:
                    assert o2m.shifts(op, n, k, scaling) == want, (op, n, k)


def test_rank2k_and_scaling_argument_errors(lib):
    P, I, C = ctypes.c_void_p, ctypes.c_int, ctypes.c_char
    fake = P(0x1000)
    lib.zher2k_2m.argtypes = [C, I, I, P, I, P, I, P, I, I, P]
    f = lib.zher2k_2m
    assert f(b"X", 4, 4, fake, 4, fake, 4, fake, 4, 16, None) == -1
    assert f(b"L", -1, 4, fake, 4, fake, 4, fake, 4, 16, None) == -2
    assert f(b"L", 4, -1, fake, 4, fake, 4, fake, 4, 16, None) == -3
    assert f(b"L", 4, 4, None, 4, fake, 4, fake, 4, 16, None) == -4
    assert f(b"L", 4, 4, fake, 3, fake, 4, fake, 4, 16, None) == -5
    assert f(b"L", 4, 4, fake, 4, None, 4, fake, 4, 16, None) == -6
    assert f(b"L", 4, 4, fake, 4, fake, 3, fake, 4, 16, None) == -7
    assert f(b"L", 4, 4, fake, 4, fake, 4, None, 4, 16, None) == -8
    assert f(b"L", 4, 4, fake, 4, fake, 4, fake, 3, 16, None) == -9
    assert f(b"L", 4, 4, fake, 4, fake, 4, fake, 4, 23, None) == -20
    assert f(b"L", 4, 74566, fake, 4, fake, 4, fake, 4, 16, None) == -21   # 2k > 149130
    assert f(b"L", 0, 4, None, 1, None, 1, None, 1, 16, None) == 0
    lib.dsyr2k_2m.argtypes = lib.zher2k_2m.argtypes
    assert lib.dsyr2k_2m(b"L", 4, 149132, fake, 4, fake, 4, fake, 4, 16, None) == -21
    lib.zgemm_2m_ex.argtypes = [I, I, I, P, I, P, I, P, I, I, I, P]
    assert lib.zgemm_2m_ex(4, 4, 4, fake, 4, fake, 4, fake, 4, 16, 2, None) == -26
    assert lib.zgemm_2m_ex(4, 4, 8192, fake, 4, fake, 8192, fake, 4, 1, 1, None) == -26  # no CS shifts
    lib.o2m_status_string.restype = ctypes.c_char_p
    assert b"scaling" in lib.o2m_status_string(-26)


def test_transposed_gemm_argument_errors(lib):
    P, I, C = ctypes.c_void_p, ctypes.c_int, ctypes.c_char
    fake = P(0x1000)
    for f in (lib.zgemm_2m_op, lib.cgemm_2m_op):
        f.argtypes = [C, C, I, I, I, P, I, P, I, P, I, I, I, P]
        # op(A) 6 x 5 (stored 5 x 6 when transposed), op(B) 5 x 7 (stored 7 x 5)
        assert f(b"X", b"N", 6, 7, 5, fake, 6, fake, 5, fake, 6, 16, 0, None) == -1
        assert f(b"N", b"H", 6, 7, 5, fake, 6, fake, 5, fake, 6, 16, 0, None) == -2
        assert f(b"N", b"N", -1, 7, 5, fake, 6, fake, 5, fake, 6, 16, 0, None) == -3
        assert f(b"N", b"N", 6, -1, 5, fake, 6, fake, 5, fake, 6, 16, 0, None) == -4
        assert f(b"N", b"N", 6, 7, -1, fake, 6, fake, 5, fake, 6, 16, 0, None) == -5
        assert f(b"N", b"N", 6, 7, 5, None, 6, fake, 5, fake, 6, 16, 0, None) == -6
        assert f(b"N", b"N", 6, 7, 5, fake, 5, fake, 5, fake, 6, 16, 0, None) == -7    # lda < m
        assert f(b"T", b"N", 6, 7, 5, fake, 4, fake, 5, fake, 6, 16, 0, None) == -7    # lda < k
        assert f(b"c", b"N", 6, 7, 5, fake, 4, fake, 5, fake, 6, 16, 0, None) == -7
        assert f(b"N", b"N", 6, 7, 5, fake, 6, None, 5, fake, 6, 16, 0, None) == -8
        assert f(b"N", b"N", 6, 7, 5, fake, 6, fake, 4, fake, 6, 16, 0, None) == -9    # ldb < k
        assert f(b"N", b"T", 6, 7, 5, fake, 6, fake, 6, fake, 6, 16, 0, None) == -9    # ldb < n
        assert f(b"N", b"N", 6, 7, 5, fake, 6, fake, 5, None, 6, 16, 0, None) == -10
        assert f(b"N", b"N", 6, 7, 5, fake, 6, fake, 5, fake, 5, 16, 0, None) == -11
        assert f(b"N", b"N", 6, 7, 5, fake, 6, fake, 5, fake, 6, 33, 0, None) == -20
        assert f(b"N", b"N", 6, 7, 5, fake, 6, fake, 5, fake, 6, 16, 5, None) == -26
        assert f(b"t", b"c", 0, 7, 5, None, 5, fake, 7, None, 1, 16, 1, None) == 0   # empty: no-op


def test_probe_library_exports_its_header():
    path = os.path.join(ROOT, "paper_2609_05419_amd", "libo2m_probe.so")
    if not os.path.exists(path):
        pytest.skip("libo2m_probe.so not built")
    text = re.sub(r"/\*.*?\*/", "", open(os.path.join(ROOT, "include", "o2m_probe.h")).read(), flags=re.S)
    names = re.findall(r"^\s*(?:double|int|void)\s*(\w+)\s*\(", text, flags=re.M)
    assert names == ["o2m_probe_int8_mfma", "o2m_probe_int8_mfma_residues", "o2m_probe_hbm"]
    L = ctypes.CDLL(path)
    for n in names:
        assert hasattr(L, n)
    L.o2m_probe_int8_mfma.restype = ctypes.c_double
    L.o2m_probe_int8_mfma.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    # bad arguments are refused before any GPU call
    assert L.o2m_probe_int8_mfma(3, 1, 1, ctypes.c_void_p(0x1000), None) < 0
    assert L.o2m_probe_int8_mfma(0, 0, 1, ctypes.c_void_p(0x1000), None) < 0
    assert L.o2m_probe_int8_mfma(0, 1, 1, None, None) < 0
    L.o2m_probe_int8_mfma_residues.restype = ctypes.c_double
    L.o2m_probe_int8_mfma_residues.argtypes = [ctypes.c_int] * 3 + [ctypes.c_void_p] * 3
    assert L.o2m_probe_int8_mfma_residues(2, 1, 1, ctypes.c_void_p(0x1000), None, None) < 0     # modulus
    assert L.o2m_probe_int8_mfma_residues(257, 1, 1, ctypes.c_void_p(0x1000), None, None) < 0
    assert L.o2m_probe_int8_mfma_residues(241, 1, 1, None, None, None) < 0
    L.o2m_probe_hbm.restype = ctypes.c_double
    L.o2m_probe_hbm.argtypes = [ctypes.c_int] + [ctypes.c_void_p] * 4 + [ctypes.c_size_t, ctypes.c_int] + \
        [ctypes.c_void_p] * 2
    fake = ctypes.c_void_p(0x1000)
    assert L.o2m_probe_hbm(5, fake, fake, fake, fake, 1 << 20, 1, fake, None) < 0       # kind
    assert L.o2m_probe_hbm(0, fake, None, None, None, 1 << 20, 1, None, None) < 0       # read needs a sink
    assert L.o2m_probe_hbm(3, fake, None, fake, None, 1 << 20, 1, None, None) < 0       # 1R:2W needs d
    assert L.o2m_probe_hbm(4, fake, None, fake, None, 1 << 20, 1, None, None) < 0       # 2R:1W needs b
    assert L.o2m_probe_hbm(2, fake, None, fake, None, 8, 1, None, None) < 0              # below 16 bytes
    assert L.o2m_probe_hbm(2, fake, None, fake, None, 1 << 20, 3, None, None) < 0        # chunks
