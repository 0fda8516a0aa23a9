// Measurement probe (not part of the 2M path): the int8 MFMA rate the chip
// sustains with operands held in registers, no memory traffic at all.  On
// random operands the part lowers its clock to stay in its power budget, so
// this rate, not the nominal 5.0 POP/s, is the practical ceiling of the int8
// GEMM.  Each workgroup (4 waves) runs `iters` rounds of 64 independent
// MFMAs per wave and writes one int per thread.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "o2m_probe.h"

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

__device__ inline int operand(unsigned &h, bool zero) {
    h ^= h << 13; h ^= h >> 17; h ^= h << 5;
    // four int8 values in [-60, 67] per dword (random bit patterns)
    return zero ? 0 : (int)(h & 0x7F7F7F7Fu) - 0x3C3C3C3C;
}

template <bool ZERO>
__global__ __launch_bounds__(256, 1) void mfma16(int iters, int *out) {
    v4i acc[8][8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[i][j] = v4i{};
    v4i a[8], b[8];
    unsigned h = threadIdx.x * 2654435761u + blockIdx.x * 40503u + 12345u;
    for (int i = 0; i < 8; ++i)
        for (int e = 0; e < 4; ++e) { a[i][e] = operand(h, ZERO); b[i][e] = operand(h, ZERO); }
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
            for (int j = 0; j < 8; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    int s = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) s += acc[i][j][0] ^ acc[i][j][1] ^ acc[i][j][2] ^ acc[i][j][3];
    out[blockIdx.x * 256 + threadIdx.x] = s;
}

__global__ __launch_bounds__(256, 1) void mfma32(int iters, int *out) {
    v16i acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = v16i{};
    v4i a[4], b[4];
    unsigned h = threadIdx.x * 2654435761u + blockIdx.x * 40503u + 777u;
    for (int i = 0; i < 4; ++i)
        for (int e = 0; e < 4; ++e) { a[i][e] = operand(h, false); b[i][e] = operand(h, false); }
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    int s = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) s ^= acc[i][j][e];
    out[blockIdx.x * 256 + threadIdx.x] = s;
}

}  // namespace

extern "C" double o2m_probe_int8_mfma(int variant, int blocks, int iters, int *out, void *stream) {
    if (blocks <= 0 || iters <= 0 || !out || variant < 0 || variant > 2) return -1.0;
    hipStream_t st = (hipStream_t)stream;
    hipEvent_t e0, e1;
    if (hipEventCreate(&e0) != hipSuccess) return -1.0;
    if (hipEventCreate(&e1) != hipSuccess) { (void)hipEventDestroy(e0); return -1.0; }
    double best = -1.0;
    for (int rep = 0; rep < 4; ++rep) {   // the first launch warms the clock up
        (void)hipEventRecord(e0, st);
        if (variant == 0) mfma16<false><<<blocks, 256, 0, st>>>(iters, out);
        else if (variant == 1) mfma16<true><<<blocks, 256, 0, st>>>(iters, out);
        else mfma32<<<blocks, 256, 0, st>>>(iters, out);
        (void)hipEventRecord(e1, st);
        if (hipEventSynchronize(e1) != hipSuccess) { best = -1.0; break; }
        float ms = 0.0f;
        (void)hipEventElapsedTime(&ms, e0, e1);
        // 4 waves x 64 (16x16x64: 32768 ops; 32x32x32 with 16 per wave: 65536 ops)
        const double ops = variant == 2 ? (double)blocks * 4 * 16 * 65536.0 * iters
                                        : (double)blocks * 4 * 64 * 32768.0 * iters;
        const double tops = ops / (ms * 1e-3) / 1e12;
        if (rep > 0 && tops > best) best = tops;
    }
    (void)hipEventDestroy(e0);
    (void)hipEventDestroy(e1);
    return best;
}
