// Host build of the int8 GEMM's and the symmetric CRT's tile schedules, for
// tests/test_tile_schedule.py.
#define O2M_HD
#include "../paper_2609_05419_amd/csrc/tile_schedule.h"
#include "../paper_2609_05419_amd/csrc/sym_schedule.h"

extern "C" {
// deal, chunk, slots, fixed, grid
void t_schedule(int mt, int nt, int kblocks, int batch, long stage_bytes, long *out) {
    const o2m::GemmSchedule s = o2m::gemm_schedule(mt, nt, kblocks, batch, stage_bytes);
    out[0] = s.deal;
    out[1] = s.chunk;
    out[2] = s.slots;
    out[3] = s.fixed;
    out[4] = s.grid;
}
// valid, p, ti, tj
void t_tile_of(int x, int slot, int mt, int nt, int chunk, int deal, int *out) {
    const o2m::TileCoord c = o2m::tile_of(x, slot, mt, nt, chunk, deal);
    out[0] = c.valid;
    out[1] = c.p;
    out[2] = c.ti;
    out[3] = c.tj;
}
// The tiles of all slots of all XCDs: tiles[4 * (x * slots + slot) + {valid, p, ti, tj}].
void t_all_tiles(int mt, int nt, int chunk, int deal, long slots, int *tiles) {
    for (int x = 0; x < o2m::kXcds; ++x)
        for (long s = 0; s < slots; ++s) {
            const o2m::TileCoord c = o2m::tile_of(x, (int)s, mt, nt, chunk, deal);
            int *o = tiles + 4 * (x * slots + s);
            o[0] = c.valid;
            o[1] = c.p;
            o[2] = c.ti;
            o[3] = c.tj;
        }
}
int t_xcds() { return o2m::kXcds; }
int t_slot_bits() { return o2m::kSlotBits; }
// Symmetric CRT: the launch's workgroup count, and tiles[3 * b + {valid, I, J}]
// for each of its workgroups.
long t_sym_grid(int nb) { return o2m::sym_grid(nb); }
void t_sym_tiles(int nb, long grid, int *tiles) {
    for (long b = 0; b < grid; ++b) {
        const o2m::SymTile t = o2m::sym_tile_of(b, nb);
        tiles[3 * b] = t.valid;
        tiles[3 * b + 1] = t.I;
        tiles[3 * b + 2] = t.J;
    }
}
void t_sym_tile_of(long b, int nb, int *out) {
    const o2m::SymTile t = o2m::sym_tile_of(b, nb);
    out[0] = t.valid;
    out[1] = t.I;
    out[2] = t.J;
}
}
