"""Host build of the int8 GEMM's tile schedule (tile_schedule.h): every slot
maps to a distinct tile or idles, every tile of every product has a slot, the
launch parameters keep their invariants, and a model of the run-time claims
(fixed slots by workgroup index, per-XCD pools with stealing, spare
workgroups; random XCD speeds) computes every tile exactly once.  And of the
symmetric CRT's (sym_schedule.h): every lower-triangle tile has exactly one
workgroup, and the four tiles that share a column line of either operand tile
run on one XCD."""
import ctypes
import math
import os
import subprocess

import numpy as np
import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
STAGE_BYTES = 256 * 64  # one k-stage of one 256-row operand tile


@pytest.fixture(scope="module")
def lib(tmp_path_factory):
    out = tmp_path_factory.mktemp("sched") / "libtile_schedule_host.so"
    subprocess.run(["g++", "-O2", "-std=c++17", "-fPIC", "-shared", os.path.join(HERE, "tile_schedule_host.cpp"),
                    "-o", str(out)], check=True)
    L = ctypes.CDLL(str(out))
    I, Lg, P = ctypes.c_int, ctypes.c_long, ctypes.c_void_p
    L.t_schedule.argtypes = [I, I, I, I, Lg, P]
    L.t_tile_of.argtypes = [I, I, I, I, I, I, P]
    L.t_all_tiles.argtypes = [I, I, I, I, Lg, P]
    L.t_sym_grid.argtypes = [I]
    L.t_sym_grid.restype = Lg
    L.t_sym_tiles.argtypes = [I, Lg, P]
    L.t_sym_tile_of.argtypes = [Lg, I, P]
    return L


def schedule(lib, mt, nt, kb, batch):
    out = np.zeros(5, dtype=np.int64)
    lib.t_schedule(mt, nt, kb, batch, STAGE_BYTES, out.ctypes.data)
    return dict(zip(("deal", "chunk", "slots", "fixed", "grid"), (int(v) for v in out)))


def all_tiles(lib, mt, nt, s):
    t = np.zeros((8, s["slots"], 4), dtype=np.int32)
    lib.t_all_tiles(mt, nt, s["chunk"], s["deal"], s["slots"], t.ctypes.data)
    return t


SHAPES = [  # mt, nt, k-stages, products
    (1, 1, 1, 1), (1, 1, 4, 32), (3, 5, 7, 2), (4, 4, 16, 32), (8, 4, 4, 32),
    (32, 32, 128, 32),            # 8192^3, N = 16: pooled
    (64, 64, 256, 16),            # 16384^3, N = 8: pooled, windows dealt
    (22, 23, 375, 32),            # ragged and dealt, last window partial
    (8, 8, 129, 32),              # pooled at the smallest slot count
    (8, 8, 128, 31), (7, 9, 200, 44), (16, 16, 512, 1), (2, 130, 128, 74), (130, 2, 130, 9),
]


def test_shared_constants(lib):
    assert lib.t_xcds() == 8 and lib.t_slot_bits() == 28


@pytest.mark.parametrize("shape", SHAPES, ids=[f"{s[0]}x{s[1]}-kb{s[2]}-b{s[3]}" for s in SHAPES])
def test_slots_cover_every_tile_once(lib, shape):
    mt, nt, kb, batch = shape
    s = schedule(lib, mt, nt, kb, batch)
    t = all_tiles(lib, mt, nt, s)
    valid = t[..., 0].astype(bool)
    keys = t[valid][:, 1:]
    assert len(keys) == mt * nt * batch
    assert len({tuple(k) for k in keys}) == mt * nt * batch       # distinct
    assert keys[:, 0].min() >= 0 and keys[:, 0].max() < batch
    assert keys[:, 1].max() < mt and keys[:, 2].max() < nt and keys.min() >= 0
    # product-major: slot s of every XCD belongs to product s // chunk
    slot_p = np.arange(s["slots"]) // s["chunk"]
    assert (t[..., 1][valid] == np.broadcast_to(slot_p, (8, s["slots"]))[valid]).all()


@pytest.mark.parametrize("shape", SHAPES, ids=[f"{s[0]}x{s[1]}-kb{s[2]}-b{s[3]}" for s in SHAPES])
def test_launch_parameters(lib, shape):
    mt, nt, kb, batch = shape
    s = schedule(lib, mt, nt, kb, batch)
    tiles = mt * nt
    windows = -(-tiles // 32)
    assert s["deal"] == int(windows >= 16 and (mt + nt) * STAGE_BYTES * kb > 256 << 20)
    assert s["chunk"] * 8 >= tiles and s["slots"] == s["chunk"] * batch
    pooled = kb >= 128 and s["slots"] >= 256
    pool = s["slots"] - s["fixed"]
    assert pool == (s["slots"] // 8 if pooled else 0)
    spare = s["grid"] // 8 - s["slots"]
    assert s["grid"] % 8 == 0 and spare == (-(-s["slots"] // 12) if pooled else 0)
    assert s["slots"] < 1 << 28


def test_empty_problem(lib):
    for shape in [(0, 4, 4, 4), (4, 0, 4, 4), (4, 4, 0, 4), (4, 4, 4, 0)]:
        assert schedule(lib, *shape)["grid"] == 0


def claim(counters, x, fixed, slots):
    """The pool claim of one workgroup on XCD x (a model of the kernel's
    claim: its own pool first, then the pools that still look open, in turn)."""
    pool = slots - fixed
    t = counters[x]
    counters[x] += 1
    if t < pool:
        return x, fixed + t
    open_ = [i for i in range(1, 8) if counters[(x + i) % 8] < pool]
    for i in open_:
        z = (x + i) % 8
        t = counters[z]
        counters[z] += 1
        if t < pool:
            return z, fixed + t
    return None


@pytest.mark.parametrize("shape", [(32, 32, 128, 32), (64, 64, 256, 16), (22, 23, 375, 32), (8, 8, 129, 32),
                                   (8, 8, 128, 31), (4, 4, 16, 32)])
def test_claimed_run_computes_every_tile_once(lib, shape):
    mt, nt, kb, batch = shape
    s = schedule(lib, mt, nt, kb, batch)
    t = all_tiles(lib, mt, nt, s)
    rng = np.random.default_rng(mt * 1000 + nt)
    for trial in range(3):
        speed = rng.uniform(0.8, 1.2, 8) if trial else np.ones(8)
        queue = [list(range(x, s["grid"], 8)) for x in range(8)]   # dispatch order per XCD
        pos, clock = [0] * 8, np.zeros(8)
        counters = [0] * 8
        done = np.zeros((batch, mt, nt), dtype=np.int64)
        empty = 0
        while True:
            live = [x for x in range(8) if pos[x] < len(queue[x])]
            if not live:
                break
            x = min(live, key=lambda i: clock[i] + rng.uniform(0, 1e-3))  # the XCD whose CU frees first
            b = queue[x][pos[x]]
            pos[x] += 1
            if b // 8 < s["fixed"]:
                z, slot = x, b // 8
            else:
                got = claim(counters, x, s["fixed"], s["slots"])
                if got is None:
                    empty += 1
                    continue
                z, slot = got
            valid, p, ti, tj = t[z, slot]
            if valid:
                done[p, ti, tj] += 1
                clock[x] += 1.0 / speed[x]
        assert (done == 1).all(), (trial, int((done == 0).sum()), int((done > 1).sum()))
        # every slot went to exactly one workgroup, so exactly the spares came away empty
        assert empty == s["grid"] - 8 * s["slots"]


SYM_NB = [0, 1, 2, 3, 4, 5, 7, 8, 9, 31, 32, 33, 63, 64, 65, 127, 255, 256, 257, 1000]


@pytest.mark.parametrize("nb", SYM_NB)
def test_sym_tiles_cover_lower_triangle_once(lib, nb):
    grid = lib.t_sym_grid(nb)
    S = 16  # tiles per super-tile side
    ns = -(-nb // S)
    assert grid == 8 * S * S * -(-(ns * (ns + 1) // 2) // 8)
    t = np.zeros((max(grid, 1), 3), dtype=np.int32)
    lib.t_sym_tiles(nb, grid, t.ctypes.data)
    t = t[:grid]
    v = t[:, 0].astype(bool)
    I, J = t[v, 1], t[v, 2]
    assert len(I) == nb * (nb + 1) // 2
    assert (I < nb).all() and (J >= 0).all() and (I >= J).all()
    assert len(set(zip(I.tolist(), J.tolist()))) == len(I)
    # the tiles sharing a line: same J, I // 4 (own tile) and same I, J // 4
    # (mirrored tile) -- all in one super-tile on one XCD, in S * S consecutive slots
    b = np.nonzero(v)[0]
    key = (I // S) * (ns + 1) + J // S
    for k in np.unique(key):
        members = b[key == k]
        assert len(set((members % 8).tolist())) == 1
        slots = members // 8
        assert slots.max() - slots.min() < S * S and len(set((slots // (S * S)).tolist())) == 1


def test_sym_tile_of_large_grids(lib):
    # super-tile rows near triangular numbers, where a float square root could round
    # the row index the wrong way
    nb = 1 << 24
    out = np.zeros(3, dtype=np.int32)
    for k in (1, 2, 3, 1000, 46340, 46341, 1 << 19, (1 << 20) - 1):
        for s in (k * (k + 1) // 2 - 1, k * (k + 1) // 2, k * (k + 1) // 2 + 1):
            b = (s // 8) * 8 * 256 + s % 8  # the first workgroup (sub-tile 0) of super-tile s
            lib.t_sym_tile_of(b, nb, out.ctypes.data)
            si = (math.isqrt(8 * s + 1) - 1) // 2  # exact integer square root
            assert (out[1], out[2]) == (16 * si, 16 * (s - si * (si + 1) // 2)), (k, s)
            assert out[0] == 1
