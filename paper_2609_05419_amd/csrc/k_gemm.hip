// K3: the int8 GEMMs of 2M (eq. 2m-mul), batched over moduli and signs.
//
//   C_p = A_p B_p^T   (A_p: m_pad x k_pad, B_p: n_pad x k_pad, both K-major
//                      int8 planes in fragment order, see o2m_internal.h)
//
// with exact int32 accumulation: |entries| <= 120 for the 2M moduli, so
// |C| <= 14400 k < 2^31 for k <= 149130 (<= 128 and k <= 131071 once the 3M
// modulus 256 of a hybrid set is in).  The epilogue reduces C_p modulo the
// product's modulus m_p to the symmetric residue and stores it as int8,
// column-major with leading dimension ldc (= m_pad), so the CRT kernel reads
// 1 byte per product per output entry instead of 4.
//
// Tiling for gfx950: a 256 x 256 output tile per workgroup of 4 waves (one
// per SIMD, 2 x 2), each wave owning 128 x 128 = 8 x 8 accumulators of
// v_mfma_i32_16x16x64_i8 held in the 256 accumulation registers (AGPRs).  On
// random int8 data this instruction sustains a markedly higher clock than
// v_mfma_i32_32x32x32_i8 at the same MAC rate.  A k-stage of 64 is 16 KB per
// operand, one contiguous chunk of the plane, copied by direct buffer->LDS
// loads (buffer_load_dwordx4 ... lds, no register staging) into a ring of 4
// stages (128 KB of the 160 KB LDS), so loads run 3 stages ahead of the
// MFMAs.  Each wave reads an operand fragment with one ds_read_b128 (64 lanes
// x 16 contiguous bytes: no bank conflicts); with 128 x 128 wave tiles that is
// 16 reads per 64 MFMAs, a third fewer than with 128 x 64, which also lets the
// part hold a higher clock.  With one wave per SIMD nothing else feeds the
// MFMA pipe, so each stage issues its 16 fragment reads after every other one
// of its first 32 MFMAs and its 8 stage copies after every fourth of the last
// 32: a memory instruction never waits behind another one in front of an
// MFMA.  The residues leave straight from the accumulators.
//
// Which workgroup computes which tile is set out in tile_schedule.h: fixed
// slots by workgroup index, and on long launches a pool of slots per XCD
// that workgroups claim at run time (claim_slot below), so that XCDs running
// at different clocks finish together.

// Bound: int8 MFMA.  Algorithmic work per launch = 2 m n k int8 ops per
// product (counting the padded-free m, n, k of the problem).
#include "o2m_internal.h"
#include "tile_schedule.h"

namespace o2m {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;                    // 4 waves: one per SIMD
constexpr int kStages = 4;                       // LDS ring of k-stages (32 KB each)
constexpr int kStageBuf = 2 * kStageBytes;       // A and B of one stage
constexpr int kLoadsPerStage = 8;                // 16-byte direct loads per thread per stage
constexpr int kPipeBytes = kStages * kStageBuf;
constexpr double kMagic = 6755399441055744.0;  // 1.5 * 2^52

typedef __attribute__((address_space(3))) void lds_void;

__device__ inline uint32_t lo32(double d) { return (uint32_t)__double2loint(d); }

// a * b + c on the low 24 bits of a and b (v_mad_u32_u24)
__device__ inline uint32_t mad24(uint32_t a, uint32_t b, uint32_t c) { return __umul24(a, b) + c; }

__device__ inline uint32_t pack4(uint32_t b0, uint32_t b1, uint32_t b2, uint32_t b3) {
    const uint32_t lo = __builtin_amdgcn_perm(b1, b0, 0x0c0c0400u);
    const uint32_t hi = __builtin_amdgcn_perm(b3, b2, 0x0c0c0400u);
    return __builtin_amdgcn_perm(hi, lo, 0x05040100u);
}

// The tile schedule (tile_of, gemm_schedule) is in tile_schedule.h; the pool
// of claimed slots is worked here.
constexpr int kHwRegXccId = (31 << 11) | 20;  // s_getreg operand: all 32 bits of XCC_ID

__device__ inline unsigned claim_next(unsigned *q) {
    return __hip_atomic_fetch_add(q, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Run by all lanes of one wave; returns x << kSlotBits | slot, or -1
// (wave-uniform).
// Pool x holds slots [S, slots) of XCD x; its counter counts the claims.
__device__ inline int claim_slot(unsigned *queue, unsigned S, unsigned slots, int lane) {
    const int x = __builtin_amdgcn_s_getreg(kHwRegXccId) & 7;
    unsigned t = lane == 0 ? claim_next(queue + x * kQueueStride) : 0u;
    t = __builtin_amdgcn_readfirstlane(t);
    if (t < slots - S) return (x << kSlotBits) | (int)(S + t);
    // own pool empty: look at the others all at once, then claim in turn
    const int y = (x + lane) & 7;
    const unsigned used =
        lane >= 1 && lane < 8 ? __hip_atomic_load(queue + y * kQueueStride, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                              : slots;
    unsigned long long open = __ballot(used < slots - S);
    while (open) {
        const int i = __builtin_ctzll(open);
        open &= open - 1;
        const int z = (x + i) & 7;
        t = lane == 0 ? claim_next(queue + z * kQueueStride) : 0u;
        t = __builtin_amdgcn_readfirstlane(t);
        if (t < slots - S) return (z << kSlotBits) | (int)(S + t);
    }
    return -1;
}

// s_waitcnt on the vector-memory counter only (gfx9 encoding), n <= 63
template <int N>
__device__ inline void wait_vm() {
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (0xF << 8));
}

// Keep the machine scheduler from moving instructions across this point: the
// fragment reads of the next stage must stay ahead of the current MFMAs.
__device__ inline void sched_fence() { __builtin_amdgcn_sched_barrier(0); }

// lgkmcnt(0): all LDS reads of this wave have returned.  At most 8 fragment
// reads are ever in flight, which the compiler tracks exactly (the counter
// holds 15), so MFMAs never wait on reads they do not consume.
__device__ inline void wait_lds() { __builtin_amdgcn_s_waitcnt(0xC07F); }

// Workgroup barrier without a memory fence: the stage data arrives by direct
// buffer->LDS loads that each thread has already waited for (vmcnt), and the
// LDS reads of the stage being recycled have completed (lgkmcnt(0)).
__device__ inline void stage_barrier() {
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Raw buffer descriptor over one tile's K-major operand rows (all its
// k-stages): the copies then take their stage offset from a scalar register
// and a fixed per-lane offset, with no 64-bit address arithmetic per copy, and
// a copy beyond the extent would read zeros instead of faulting.
constexpr int kBufferWord3 = 0x00020000;  // raw 32-bit buffer (gfx9 family)

__device__ inline __amdgpu_buffer_rsrc_t tile_rsrc(const int8_t *base, int kblocks) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<int8_t *>(base), (short)0, kblocks * kStageBytes,
                                             kBufferWord3);
}

// Direct copy q (0..7) of k-stage `stage` into LDS buffer `buf`: even q copy
// 4 KB of A, odd q 4 KB of B; each wave copies 1 KB contiguous.
__device__ inline void load_part(__amdgpu_buffer_rsrc_t rA, __amdgpu_buffer_rsrc_t rB, int stage, int8_t *buf,
                                 int tid, int wave, int q) {
    const int off = (q >> 1) * 4096;
    const int soff = stage * kStageBytes + off;
    if ((q & 1) == 0)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rA, (lds_void *)(buf + off + wave * 1024), 16, tid * 16, soff, 0, 0);
    else
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rB, (lds_void *)(buf + kStageBytes + off + wave * 1024), 16,
                                                 tid * 16, soff, 0, 0);
}

__device__ inline void load_stage(__amdgpu_buffer_rsrc_t rA, __amdgpu_buffer_rsrc_t rB, int stage, int8_t *buf,
                                  int tid, int wave) {
#pragma unroll
    for (int q = 0; q < kLoadsPerStage; ++q) load_part(rA, rB, stage, buf, tid, wave, q);
}

// Fragment f (0..15) of a stage: A rows 16 f of the wave for f < 8, B rows
// 16 (f - 8) of the wave after that.
__device__ inline v4i read_frag(const int8_t *buf, int aoff, int boff, int lane, int f) {
    const int off = f < 8 ? aoff + f * kFragBytes : boff + (f - 8) * kFragBytes;
    return *reinterpret_cast<const v4i *>(buf + off + lane * 16);
}

// acc += a b^T on one 16 x 16 block.  Written as inline assembly so that the
// accumulator stays in its AGPRs: with the builtin the compiler copies the
// 256 accumulators between AGPRs and VGPRs in every stage.  The compiler does
// not see this as an MFMA, so the hazards it would otherwise cover are
// handled where they arise: fragment reads are waited for (lgkmcnt) before a
// stage's MFMAs, and acc_after_fill() / acc_after_mfma() separate
// accumulator writes from reads.
__device__ inline void mfma(v4i &acc, const v4i &a, const v4i &b) {
    asm volatile("v_mfma_i32_16x16x64_i8 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b) : "memory");
}

// Wait states between the accumulator registers' last writer and their next
// reader.  Each asm takes a row of accumulators as operands, so no access to
// them can move across it.
//   acc_after_fill: the zero fill (VALU writes) before the first MFMA reads them
//   acc_after_mfma: the last MFMAs (16 passes) before the epilogue reads them
__device__ inline void acc_after_fill(v4i (&acc)[8][8]) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
        asm volatile("s_nop 4" : "+a"(acc[i][0]), "+a"(acc[i][1]), "+a"(acc[i][2]), "+a"(acc[i][3]),
                     "+a"(acc[i][4]), "+a"(acc[i][5]), "+a"(acc[i][6]), "+a"(acc[i][7]));
}
__device__ inline void acc_after_mfma(v4i (&acc)[8][8]) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
        asm volatile("s_nop 7\n s_nop 7\n s_nop 7" : "+a"(acc[i][0]), "+a"(acc[i][1]), "+a"(acc[i][2]),
                     "+a"(acc[i][3]), "+a"(acc[i][4]), "+a"(acc[i][5]), "+a"(acc[i][6]), "+a"(acc[i][7]));
}

// 4 x 4 transpose of dwords across the four 16-lane rows of a wave: on entry
// row r of d[q] holds X[r][q], on exit row r of d[q] holds X[q][r].
// v_permlane32_swap exchanges the upper 32 lanes of its first operand with the
// lower 32 lanes of its second, v_permlane16_swap the odd rows of its first
// operand with the even rows of its second.
__device__ inline void transpose_rows(uint32_t (&d)[4]) {
    auto t02 = __builtin_amdgcn_permlane32_swap(d[0], d[2], false, false);
    auto t13 = __builtin_amdgcn_permlane32_swap(d[1], d[3], false, false);
    auto t01 = __builtin_amdgcn_permlane16_swap(t02[0], t13[0], false, false);
    auto t23 = __builtin_amdgcn_permlane16_swap(t02[1], t13[1], false, false);
    d[0] = t01[0];
    d[1] = t01[1];
    d[2] = t23[0];
    d[3] = t23[1];
}

// Epilogue: C mod m -> int8, stored from the accumulators.
// v_mfma_i32_16x16x64_i8 leaves column (lane % 16), rows 4 (lane / 16) + e of
// its 16 x 16 block in element e: 4 consecutive rows of the column-major
// output make one dword.  A transpose across the lane rows of four row blocks
// gives each lane 16 consecutive rows of one block, so one 16-byte store per
// lane writes 64 contiguous bytes of each of 16 columns, and the two halves of
// the wave tile fill whole 128-byte column segments.
__device__ inline void store_tile(const v4i (&acc)[8][8], int8_t *C, int ldc, int m, double inv) {
    const uint32_t negm = (uint32_t)(-m) & 0xFFFFFFu;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            uint32_t d[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                uint32_t by[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int v = acc[4 * h + q][j][e];
                    const double qm = fma((double)v, inv, kMagic);  // 1.5 2^52 + rint(v / m)
                    by[e] = mad24(lo32(qm), negm, (uint32_t)v);    // v - q m (low byte)
                }
                d[q] = pack4(by[0], by[1], by[2], by[3]);
            }
            transpose_rows(d);
            *reinterpret_cast<uint4 *>(C + (size_t)(j * 16) * ldc + h * 64) = uint4{d[0], d[1], d[2], d[3]};
        }
    }
}

// One wave's place in the workgroup's pipeline.
struct Wave {
    int8_t *lds;     // the ring of kStages stage buffers
    int tid, lane;
    int wave;        // wave-uniform
    int aoff, boff;  // this wave's A and B fragments within a stage buffer
};

__device__ inline Wave wave_of(int8_t *lds) {
    Wave w;
    w.lds = lds;
    w.tid = threadIdx.x;
    w.lane = w.tid & 63;
    w.wave = __builtin_amdgcn_readfirstlane(w.tid >> 6);  // wave-uniform (SGPR)
    const int wr = w.wave >> 1, wc = w.wave & 1;          // 2 x 2 waves of 128 x 128
    w.aoff = wr * 8 * kFragBytes;
    w.boff = kStageBytes + wc * 8 * kFragBytes;
    return w;
}

__device__ inline void zero_acc(v4i (&acc)[8][8]) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[i][j] = v4i{};
    acc_after_fill(acc);
}

// Fill the ring with the first min(KB, kStages) stages of one tile.
__device__ inline void prologue_copies(const Wave &w, __amdgpu_buffer_rsrc_t rA, __amdgpu_buffer_rsrc_t rB,
                                       int KB) {
    const int pre = KB < kStages ? KB : kStages;
    for (int s = 0; s < pre; ++s) load_stage(rA, rB, s, w.lds + s * kStageBuf, w.tid, w.wave);
}

// Wait for stage 0 of the ring and read its fragments into (fa, fb).
__device__ inline void prologue_wait(const Wave &w, int KB, v4i (&fa)[8], v4i (&fb)[8]) {
    const int pre = KB < kStages ? KB : kStages;
    switch (pre) {
    case 1: wait_vm<0>(); break;
    case 2: wait_vm<kLoadsPerStage>(); break;
    case 3: wait_vm<2 * kLoadsPerStage>(); break;
    default: wait_vm<3 * kLoadsPerStage>(); break;
    }
    stage_barrier();
#pragma unroll
    for (int f = 0; f < 8; ++f) {
        fa[f] = read_frag(w.lds, w.aoff, w.boff, w.lane, f);
        fb[f] = read_frag(w.lds, w.aoff, w.boff, w.lane, 8 + f);
    }
    wait_lds();
}

// Stage kb, its fragments in (ca, cb): wait until stage kb+1 has landed
// (`younger` later stages may stay in flight), barrier (every wave is done
// reading stage kb, so its buffer is free), then the 64 MFMAs of stage kb with
// the fragment reads of stage kb+1 into (na, nb) and, if `refill`, the copy of
// stage kb+4 of (rA, rB) into the freed buffer, both issued first.  Used for
// the last stages of a tile, where waits shrink.
__device__ inline void edge_stage(v4i (&acc)[8][8], const Wave &w, int kb, const v4i (&ca)[8], const v4i (&cb)[8],
                                  v4i (&na)[8], v4i (&nb)[8], int younger, bool next, bool refill,
                                  __amdgpu_buffer_rsrc_t rA, __amdgpu_buffer_rsrc_t rB) {
    if (younger >= 2) wait_vm<2 * kLoadsPerStage>();
    else if (younger == 1) wait_vm<kLoadsPerStage>();
    else wait_vm<0>();
    stage_barrier();
    const int8_t *nbuf = w.lds + ((kb + 1) % kStages) * kStageBuf;
    if (next) {
#pragma unroll
        for (int f = 0; f < 8; ++f) {
            na[f] = read_frag(nbuf, w.aoff, w.boff, w.lane, f);
            nb[f] = read_frag(nbuf, w.aoff, w.boff, w.lane, 8 + f);
        }
    }
    if (refill) load_stage(rA, rB, kb + kStages, w.lds + (kb % kStages) * kStageBuf, w.tid, w.wave);
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) mfma(acc[i][j], ca[i], cb[j]);
    wait_lds();  // the next stage's fragments are in registers
}

// Steady-state stage kb: as edge_stage with two younger stages in flight, but
// the fragment reads of stage kb+1 follow every other one of the first 32
// MFMAs and the 8 copies of stage `sstage` (= kb+4) of (sA, sB) into the
// freed buffer every fourth one of the last 32.
__device__ inline void steady_stage(v4i (&acc)[8][8], const Wave &w, int kb, const v4i (&ca)[8], const v4i (&cb)[8],
                                    v4i (&na)[8], v4i (&nb)[8], __amdgpu_buffer_rsrc_t sA,
                                    __amdgpu_buffer_rsrc_t sB, int sstage) {
    wait_vm<2 * kLoadsPerStage>();
    stage_barrier();
    const int8_t *nbuf = w.lds + ((kb + 1) % kStages) * kStageBuf;
    int8_t *rbuf = w.lds + (kb % kStages) * kStageBuf;
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            mfma(acc[i][j], ca[i], cb[j]);
            const int t = 8 * i + j;
            if (t < 32 && (t & 1) == 0) {
                const int f = t >> 1;
                if (f < 8) na[f] = read_frag(nbuf, w.aoff, w.boff, w.lane, f);
                else nb[f - 8] = read_frag(nbuf, w.aoff, w.boff, w.lane, f);
            }
            if (t >= 32 && (t & 3) == 0) load_part(sA, sB, sstage, rbuf, w.tid, w.wave, (t - 32) >> 2);
        }
    wait_lds();
}

// The tile's output block for this wave: C mod m as int8.
__device__ inline void epilogue(v4i (&acc)[8][8], const Wave &w, const GemmArgs &g, const TileCoord &tc) {
    acc_after_mfma(acc);
    const int wr = w.wave >> 1, wc = w.wave & 1;
    int8_t *C = g.c + (size_t)tc.p * g.c_pstride + (size_t)(tc.tj * 256 + wc * 128 + (w.lane & 15)) * g.ldc +
                tc.ti * 256 + wr * 128 + 16 * (w.lane >> 4);
    store_tile(acc, C, g.ldc, g.mod[tc.p], g.inv[tc.p]);
}

__device__ inline __amdgpu_buffer_rsrc_t rsrc_a(const GemmArgs &g, const TileCoord &tc) {
    return tile_rsrc(g.a + (size_t)tc.p * g.a_pstride + (size_t)tc.ti * g.kblocks * kStageBytes, g.kblocks);
}
__device__ inline __amdgpu_buffer_rsrc_t rsrc_b(const GemmArgs &g, const TileCoord &tc) {
    return tile_rsrc(g.b + (size_t)tc.p * g.b_pstride + (size_t)tc.tj * g.kblocks * kStageBytes, g.kblocks);
}

// One output tile per workgroup.
__global__ __launch_bounds__(kThreads, 1) void gemm_i8_kernel(GemmArgs g) {
    // One LDS object: the stage ring and, past its end, the claimed slot.  A
    // second __shared__ variable would give the compiler alias scopes for LDS,
    // with which it waits for every stage copy in flight (vmcnt(0)) before
    // each fragment read of the k-loop.
    __shared__ __attribute__((aligned(1024))) int8_t lds[kPipeBytes + 16];
    int *claimed = reinterpret_cast<int *>(lds + kPipeBytes);

    const Wave w = wave_of(lds);
    const int slots = g.chunk * g.batch;  // per XCD
    // all arguments of the tile arithmetic and the first stage copies are
    // loaded here in one round, rather than in rounds behind each other
    asm volatile("" ::"s"(g.a), "s"(g.b), "s"(g.a_pstride), "s"(g.b_pstride), "s"(g.kblocks), "s"(g.mt),
                 "s"(g.nt), "s"(g.deal), "s"(g.fixed));
    v4i acc[8][8];
    TileCoord tc;
    __amdgpu_buffer_rsrc_t rA, rB;
    if ((int)(blockIdx.x >> 3) < g.fixed) {
        tc = tile_of(blockIdx.x & 7, blockIdx.x >> 3, g.mt, g.nt, g.chunk, g.deal);
        if (!tc.valid) return;  // whole workgroup: no barrier is pending
    } else {
        if (w.wave == 0) {
            const int r = claim_slot(g.queue, (unsigned)g.fixed, (unsigned)slots, w.lane);
            if (w.lane == 0) *claimed = r;
        }
        __syncthreads();
        const int c = *claimed;
        if (c < 0) return;  // whole workgroup: no barrier is pending
        tc = tile_of(c >> kSlotBits, c & ((1 << kSlotBits) - 1), g.mt, g.nt, g.chunk, g.deal);
        if (!tc.valid) return;
    }
    rA = rsrc_a(g, tc);
    rB = rsrc_b(g, tc);
    const int KB = g.kblocks;
    // the first stage copies go out before the accumulator fill, which then
    // runs while they are in flight
    prologue_copies(w, rA, rB, KB);
    sched_fence();
    zero_acc(acc);
    // Fragments of the current stage (fa0, fb0) and of the next one.
    v4i fa0[8], fb0[8], fa1[8], fb1[8];
    prologue_wait(w, KB, fa0, fb0);

    // Steady state, two stages per trip so that the fragment sets alternate
    // statically; then at most five stages with shrinking waits, the sets
    // still alternating statically.
    int kb = 0;
    for (; kb + kStages + 1 < KB; kb += 2) {
        steady_stage(acc, w, kb, fa0, fb0, fa1, fb1, rA, rB, kb + kStages);
        steady_stage(acc, w, kb + 1, fa1, fb1, fa0, fb0, rA, rB, kb + 1 + kStages);
    }
    auto tail = [&](v4i (&ca)[8], v4i (&cb)[8], v4i (&na)[8], v4i (&nb)[8]) {
        if (kb < KB) {
            edge_stage(acc, w, kb, ca, cb, na, nb, min(KB - 1, kb + kStages - 1) - (kb + 1), kb + 1 < KB,
                       kb + kStages < KB, rA, rB);
            ++kb;
        }
    };
    tail(fa0, fb0, fa1, fb1);
    tail(fa1, fb1, fa0, fb0);
    tail(fa0, fb0, fa1, fb1);
    tail(fa1, fb1, fa0, fb0);
    tail(fa0, fb0, fa1, fb1);

    epilogue(acc, w, g, tc);
}

}  // namespace

hipError_t launch_gemm(const GemmArgs &ga_in, hipStream_t st) {
    static_assert(kThreads * 16 * kLoadsPerStage == 2 * kStageBytes, "stage copy covers A and B");
    GemmArgs ga = ga_in;
    const GemmSchedule sc = gemm_schedule(ga.mt, ga.nt, ga.kblocks, ga.batch, kStageBytes);
    if (sc.grid == 0) return hipSuccess;
    if (sc.grid > 0x7FFFFFFF || sc.slots >= (1L << kSlotBits)) return hipErrorInvalidValue;
    ga.deal = sc.deal;
    ga.chunk = sc.chunk;
    ga.fixed = (int)sc.fixed;
    const long grid = sc.grid;
    gemm_i8_kernel<<<(unsigned)grid, kThreads, 0, st>>>(ga);
    return hipGetLastError();
}

}  // namespace o2m
