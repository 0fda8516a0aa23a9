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
// Tiling for gfx950: a 256 x 256 output tile per workgroup of 8 waves (2 per
// SIMD, 2 x 4), each wave owning 128 x 64 = 8 x 4 accumulators of
// v_mfma_i32_16x16x64_i8.  On random int8 data this instruction sustains a
// markedly higher clock than v_mfma_i32_32x32x32_i8 at the same MAC rate, and
// the second wave per SIMD hides LDS and barrier latency.  A k-stage of 64 is
// 16 KB per operand, one contiguous chunk of the plane, copied by direct
// global->LDS loads (global_load_lds_dwordx4, no register staging) into a ring
// of 4 stages (128 KB of the 160 KB LDS), so loads run 3 stages ahead of the
// MFMAs.  Each wave reads an operand fragment with one ds_read_b128 (64 lanes
// x 16 contiguous bytes: no bank conflicts).  The two waves of a SIMD meet at
// a barrier every stage, so whatever they issue between MFMA batches leaves
// the MFMA pipe idle: the steady-state loop is kept free of branches and
// conditional waits, and the residues leave straight from the accumulators.

// Bound: int8 MFMA.  Algorithmic work per launch = 2 m n k int8 ops per
// product (counting the padded-free m, n, k of the problem).
#include "o2m_internal.h"

namespace o2m {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

constexpr int kThreads = 512;                    // 8 waves: 2 per SIMD
constexpr int kStages = 4;                       // LDS ring of k-stages (32 KB each)
constexpr int kStageBuf = 2 * kStageBytes;       // A and B of one stage
constexpr int kLoadsPerStage = 4;                // 16-byte direct loads per thread per stage
constexpr int kPipeBytes = kStages * kStageBuf;
constexpr double kMagic = 6755399441055744.0;  // 1.5 * 2^52
constexpr int kGroupRows = 8;

typedef __attribute__((address_space(3))) void lds_void;

__device__ inline uint32_t lo32(double d) { return (uint32_t)__double2loint(d); }

// a * b + c on the low 24 bits of a and b (v_mad_u32_u24)
__device__ inline uint32_t mad24(uint32_t a, uint32_t b, uint32_t c) { return __umul24(a, b) + c; }

__device__ inline uint32_t pack4(uint32_t b0, uint32_t b1, uint32_t b2, uint32_t b3) {
    const uint32_t lo = __builtin_amdgcn_perm(b1, b0, 0x0c0c0400u);
    const uint32_t hi = __builtin_amdgcn_perm(b3, b2, 0x0c0c0400u);
    return __builtin_amdgcn_perm(hi, lo, 0x05040100u);
}

// Tile schedule.  The hardware deals workgroups to the 8 XCDs round-robin
// (workgroup b -> XCD b % 8, in dispatch order b / 8 within it).  Each batch
// item (one int8 GEMM) is split into 8 contiguous chunks of its grouped tile
// order, one per XCD, and all XCDs sweep the batch items in the same order:
// at any time the whole chip works on one product, whose operand planes
// (2 x 64 MB at 8192^2) stay resident in the 256 MB Infinity Cache, while the
// tiles resident on one XCD (8 tile-rows x 4 tile-columns) share their A and
// B stages in that XCD's L2.  Slots beyond a product's tile count idle.
struct TileCoord {
    int p, ti, tj;
    bool valid;
};
__device__ inline TileCoord tile_of(int b, int mt, int nt, int chunk) {
    TileCoord c;
    const int x = b & 7, slot = b >> 3;
    c.p = slot / chunk;
    const int t = x * chunk + (slot - c.p * chunk);  // index in the product's grouped order
    c.valid = t < mt * nt;
    const int group = t / (kGroupRows * nt);
    const int first = group * kGroupRows;
    const int gsize = min(mt - first, kGroupRows);
    const int within = t - group * kGroupRows * nt;
    c.ti = first + within % gsize;
    c.tj = within / gsize;
    return c;
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
// global->LDS loads that each thread has already waited for (vmcnt), and the
// LDS reads of the stage being recycled have completed (lgkmcnt(0)).
__device__ inline void stage_barrier() {
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Issue the direct loads of one k-stage (A then B, 16 KB each) into LDS
// buffer `buf`: each wave copies 1 KB contiguous per instruction.
__device__ inline void load_stage(const int8_t *A, const int8_t *B, int8_t *buf, int tid, int wave) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        __builtin_amdgcn_global_load_lds(A + q * 8192 + tid * 16, (lds_void *)(buf + q * 8192 + wave * 1024), 16, 0, 0);
        __builtin_amdgcn_global_load_lds(B + q * 8192 + tid * 16,
                                         (lds_void *)(buf + kStageBytes + q * 8192 + wave * 1024), 16, 0, 0);
    }
}

// Operand fragments of a wave (128 rows of A, 64 rows of B) for one stage.
__device__ inline void read_a(const int8_t *buf, int wr, int lane, int i0, v4i (&a)[8]) {
#pragma unroll
    for (int i = i0; i < i0 + 4; ++i) a[i] = *reinterpret_cast<const v4i *>(buf + (wr * 8 + i) * kFragBytes + lane * 16);
}
__device__ inline void read_b(const int8_t *buf, int wc, int lane, v4i (&b)[4]) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
        b[j] = *reinterpret_cast<const v4i *>(buf + kStageBytes + (wc * 4 + j) * kFragBytes + lane * 16);
}

// 16 MFMAs: accumulator rows i0..i0+3 against all 4 B fragments.
__device__ inline void mfma_half(v4i (&acc)[8][4], const v4i (&a)[8], const v4i (&b)[4], int i0) {
#pragma unroll
    for (int i = i0; i < i0 + 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[i], b[j], acc[i][j], 0, 0, 0);
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
__device__ inline void store_tile(const v4i (&acc)[8][4], int8_t *C, int ldc, int m, double inv) {
    const uint32_t negm = (uint32_t)(-m) & 0xFFFFFFu;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
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

__global__ __launch_bounds__(kThreads, 1) void gemm_i8_kernel(GemmArgs g) {
    __shared__ __attribute__((aligned(1024))) int8_t lds[kPipeBytes];

    const TileCoord tc = tile_of((int)blockIdx.x, g.mt, g.nt, g.chunk);
    if (!tc.valid) return;  // whole workgroup: no barrier is pending
    const int p = tc.p, ti = tc.ti, tj = tc.tj;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (SGPR)
    const int wr = wave >> 2, wc = wave & 3;                     // 2 x 4 waves of 128 x 64
    const int KB = g.kblocks;

    const int8_t *A = g.a + (size_t)p * g.a_pstride + (size_t)ti * KB * kStageBytes;
    const int8_t *B = g.b + (size_t)p * g.b_pstride + (size_t)tj * KB * kStageBytes;

    v4i acc[8][4];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = v4i{};

    // prologue: fill the ring, then wait for stage 0
    const int pre = KB < kStages ? KB : kStages;
    for (int s = 0; s < pre; ++s)
        load_stage(A + (size_t)s * kStageBytes, B + (size_t)s * kStageBytes, lds + s * kStageBuf, tid, wave);
    switch (pre) {
    case 1: wait_vm<0>(); break;
    case 2: wait_vm<kLoadsPerStage>(); break;
    case 3: wait_vm<2 * kLoadsPerStage>(); break;
    default: wait_vm<3 * kLoadsPerStage>(); break;
    }
    stage_barrier();

    v4i fa[8], fb[4], nb[4];
    read_a(lds, wr, lane, 0, fa);
    read_b(lds, wc, lane, fb);

    // One k-stage: rows 4..7 of A are read while the MFMAs of rows 0..3 run;
    // the barrier that frees this stage's buffer sits between the two MFMA
    // halves; the next stage's rows 0..3 of A and its B are read while the
    // MFMAs of rows 4..7 run, and the freed buffer is refilled after them.
    // `younger` is the number of stages after the next one whose loads may
    // stay in flight at the barrier; `refill` whether stage kb + 4 exists.
    auto stage = [&](int kb, int younger, bool refill) {
        const int8_t *buf = lds + (kb % kStages) * kStageBuf;
        wait_lds();
        read_a(buf, wr, lane, 4, fa);
        sched_fence();
        mfma_half(acc, fa, fb, 0);
        sched_fence();
        if (younger >= 2) wait_vm<2 * kLoadsPerStage>();
        else if (younger == 1) wait_vm<kLoadsPerStage>();
        else wait_vm<0>();
        stage_barrier();  // every wave is done reading stage kb: its buffer is free
        const int8_t *nbuf = lds + ((kb + 1) % kStages) * kStageBuf;
        read_a(nbuf, wr, lane, 0, fa);
        read_b(nbuf, wc, lane, nb);
        sched_fence();
        mfma_half(acc, fa, fb, 4);
        sched_fence();
        // refill the freed buffer after the MFMAs, so that the fragment reads
        // above are not queued behind the stage copy
        if (refill)
            load_stage(A + (size_t)(kb + kStages) * kStageBytes, B + (size_t)(kb + kStages) * kStageBytes,
                       lds + (kb % kStages) * kStageBuf, tid, wave);
#pragma unroll
        for (int j = 0; j < 4; ++j) fb[j] = nb[j];
    };
    // Steady state (constant wait, always a refill), then the last stages
    // with shrinking waits.  The final stage is peeled off so that every
    // iteration has the same LDS-counter state (no conservative waits).
    int kb = 0;
    for (; kb + kStages < KB; ++kb) stage(kb, 2, true);
    for (; kb + 1 < KB; ++kb) stage(kb, min(KB - 1, kb + kStages - 1) - (kb + 1), false);
    wait_lds();
    read_a(lds + ((KB - 1) % kStages) * kStageBuf, wr, lane, 4, fa);
    mfma_half(acc, fa, fb, 0);
    mfma_half(acc, fa, fb, 4);

    int8_t *C = g.c + (size_t)p * g.c_pstride + (size_t)(tj * 256 + wc * 64 + (lane & 15)) * g.ldc + ti * 256 +
                wr * 128 + 16 * (lane >> 4);
    store_tile(acc, C, g.ldc, g.mod[p], g.inv[p]);
}

}  // namespace

hipError_t launch_gemm(const GemmArgs &ga_in, hipStream_t st) {
    static_assert(kThreads * 16 * kLoadsPerStage == 2 * kStageBytes, "stage copy covers A and B");
    GemmArgs ga = ga_in;
    const long tiles = (long)ga.mt * ga.nt;
    if (tiles <= 0 || ga.batch <= 0 || ga.kblocks <= 0) return hipSuccess;
    ga.chunk = (int)((tiles + 7) / 8);
    const long total = 8L * ga.chunk * ga.batch;
    if (total > 0x7FFFFFFF) return hipErrorInvalidValue;
    gemm_i8_kernel<<<(unsigned)total, kThreads, 0, st>>>(ga);
    return hipGetLastError();
}

}  // namespace o2m
