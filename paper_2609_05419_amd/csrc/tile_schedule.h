// Tile schedule of the int8 GEMM (K3): which workgroup computes which output
// tile.  Shared by the kernel and the host-compiled test of its invariants;
// nothing here touches memory.
//
// Each XCD has a queue of slots, and within a product the slots follow a
// grouped order of the tiles (groups of 8 tile-rows, column-major inside a
// group), cut into windows of 32 tiles (8 tile-rows x 4 tile-columns): the
// tiles resident on one XCD at a time share their A and B stages in that
// XCD's L2.  All XCDs sweep the batch items (one int8 GEMM each) in the same
// order, so at any time the whole chip works on one product.  Products whose
// planes fit in the 256 MB Infinity Cache give each XCD one contiguous chunk
// of the order.  Larger ones (2 x 256 MB at 16384^2) deal the windows
// round-robin (window w -> XCD w % 8), so that all XCDs work in the same
// group of 8 tile-rows at once and its A strip is read once from HBM and
// shared through the Infinity Cache.  Slots beyond a product's tiles idle.
//
// The XCDs of the part do not run at one clock (up to a tenth apart under
// this load), so a fixed share of tiles per XCD would leave the fast ones idle
// while the slowest finishes.  In long launches the first 7/8 of each XCD's
// slots therefore go to workgroups by index, as dispatched (workgroup b runs
// on XCD b % 8 and takes its slot b / 8), and the last 1/8 form a pool that
// workgroups claim at run time: the next slot of the pool of their own XCD,
// and once that is empty, the next slot of the first other pool that still
// has one.  The launch carries spare workgroups for those extra claims; a
// workgroup that finds every pool empty exits.  Only the pool's workgroups
// wait for an atomic round trip before their first stage copy, and the spares
// cost a few microseconds at the end, so short launches (fewer than 128
// k-stages or 256 slots per XCD, where that cost outweighs the balance) keep
// every slot fixed.  Each pool slot is handed out once (atomic counters,
// which start at zero), and every one is claimed: a workgroup only finds all
// pools empty when all their slots are taken, and the pools have more
// workgroups than slots.
#pragma once

#ifndef O2M_HD
#define O2M_HD __host__ __device__
#endif

namespace o2m {

constexpr int kXcds = 8;
constexpr int kGroupRows = 8;     // tile-rows per group of the grouped order
constexpr int kWindowTiles = 32;  // tiles per window (8 tile-rows x 4 tile-columns)
constexpr int kSlotBits = 28;     // a claimed slot travels as x << 28 | slot

struct TileCoord {
    int p, ti, tj;
    bool valid;
};

// Slot `slot` of XCD x's queue -> product p, tile (ti, tj), or an idle slot.
O2M_HD inline TileCoord tile_of(int x, int slot, int mt, int nt, int chunk, int deal) {
    TileCoord c;
    c.p = slot / chunk;
    const int s = slot - c.p * chunk;  // the slot within the product
    const int t = deal ? (kXcds * (s / kWindowTiles) + x) * kWindowTiles + s % kWindowTiles
                       : x * chunk + s;  // index in the grouped order
    c.valid = t < mt * nt;
    c.ti = c.tj = 0;
    if (!c.valid) return c;  // idle slot (its group arithmetic would divide by zero)
    const int group = t / (kGroupRows * nt);
    const int first = group * kGroupRows;
    const int gsize = mt - first < kGroupRows ? mt - first : kGroupRows;
    const int within = t - group * kGroupRows * nt;
    c.ti = first + within % gsize;
    c.tj = within / gsize;
    return c;
}

// Launch parameters of one batched int8 GEMM.
struct GemmSchedule {
    int deal;    // 1: windows dealt round-robin to the XCDs
    int chunk;   // slots per XCD and product
    long slots;  // slots per XCD over the batch
    long fixed;  // of those, taken by workgroup index; the rest are pooled
    long grid;   // workgroups: kXcds * slots plus the spares (0 when nothing to do)
};

// mt x nt tiles per product, kblocks k-stages of stage_bytes per operand
// tile, batch products.  grid stays 0 for an empty problem; the caller
// rejects grids beyond the launch limit.
O2M_HD inline GemmSchedule gemm_schedule(int mt, int nt, int kblocks, int batch, long stage_bytes) {
    GemmSchedule s = {0, 0, 0, 0, 0};
    const long tiles = (long)mt * nt;
    if (tiles <= 0 || batch <= 0 || kblocks <= 0) return s;
    // deal windows when each XCD gets at least two and one product's operand
    // planes outgrow the 256 MB Infinity Cache
    const long windows = (tiles + kWindowTiles - 1) / kWindowTiles;
    const long plane_bytes = (long)(mt + nt) * stage_bytes * kblocks;
    s.deal = windows >= 2 * kXcds && plane_bytes > (256L << 20) ? 1 : 0;
    s.chunk = (int)(s.deal ? kWindowTiles * ((windows + kXcds - 1) / kXcds) : (tiles + kXcds - 1) / kXcds);
    s.slots = (long)s.chunk * batch;
    // pooled: the last 1/8 of each XCD's slots, plus one spare workgroup per
    // 12 slots, so that a faster XCD can take slots of a slower one's pool
    const bool pool = kblocks >= 128 && s.slots >= 256;
    s.fixed = pool ? s.slots - s.slots / 8 : s.slots;
    s.grid = kXcds * (s.slots + (pool ? (s.slots + 11) / 12 : 0));
    return s;
}

}  // namespace o2m
