// Tile schedule of the symmetric CRT (K4 for HERK / SYRK / HER2K / SYR2K
// outputs): which workgroup computes which output tile.  Shared by the kernel
// and the host-compiled test of its invariants; nothing here touches memory.
//
// Each workgroup owns a 32 x 32 output tile (I, J) with I >= J and reads, per
// modulus, its own tile of the int8 residue plane and the mirrored tile
// (J, I).  A tile column is a 32-byte piece of a 128-byte line (int8,
// column-major), shared with the three neighbouring tiles of the same column
// strip, and each XCD fetches into its own L2.  Dispatched in index order the
// four tiles that share a line run on four XCDs, and the line crosses the
// fabric four times.  Instead, super-tiles of 16 x 16 tiles (512 x 512, the
// lower triangle in row-major order) are dealt round-robin to the XCDs, and
// the 256 workgroups of one super-tile take 256 consecutive slots of the same
// XCD (about as many as it holds at once), so that a line is fetched once and
// serves all four tiles from L2, and the workgroups of a super-tile read each
// column of the plane in 512-byte runs.  Tiles above the diagonal (in
// diagonal super-tiles) and beyond nb idle.
#pragma once

#include <cmath>

#ifndef O2M_HD
#define O2M_HD __host__ __device__
#endif

namespace o2m {

constexpr int kSymXcds = 8;   // workgroup b is dispatched to XCD b % 8
constexpr int kSymSuper = 16;  // tiles per super-tile side

struct SymTile {
    int I, J;  // tile-row and tile-column of the output tile
    bool valid;
};

// lower-triangle super-tiles of an nb x nb tile grid
O2M_HD inline long sym_supers(int nb) {
    const long ns = (nb + kSymSuper - 1) / kSymSuper;
    return ns * (ns + 1) / 2;
}

// workgroups of the symmetric CRT launch (0 for nb = 0)
O2M_HD inline long sym_grid(int nb) {
    return (long)kSymXcds * kSymSuper * kSymSuper * ((sym_supers(nb) + kSymXcds - 1) / kSymXcds);
}

// workgroup b (on XCD b % 8, slot b / 8) -> its output tile, or idle
O2M_HD inline SymTile sym_tile_of(long b, int nb) {
    constexpr int per = kSymSuper * kSymSuper;
    SymTile t = {0, 0, false};
    const long slot = b / kSymXcds;
    const long s = (slot / per) * kSymXcds + b % kSymXcds;  // super-tile index
    if (s >= sym_supers(nb)) return t;
    // super-tile row si: si (si + 1) / 2 <= s < (si + 1) (si + 2) / 2
    long si = (long)((sqrt(8.0 * (double)s + 1.0) - 1.0) * 0.5);
    while (si > 0 && si * (si + 1) / 2 > s) --si;
    while ((si + 1) * (si + 2) / 2 <= s) ++si;
    const long sj = s - si * (si + 1) / 2;
    const int sub = (int)(slot % per);
    t.I = (int)(si * kSymSuper + sub % kSymSuper);
    t.J = (int)(sj * kSymSuper + sub / kSymSuper);
    t.valid = t.I < nb && t.I >= t.J;
    return t;
}

}  // namespace o2m
