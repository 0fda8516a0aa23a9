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

__device__ inline unsigned next(unsigned &h) {
    h ^= h << 13; h ^= h >> 17; h ^= h << 5;
    return h;
}

// Four int8 operand values per dword: modulus 0: random bit patterns in
// [-60, 67]; modulus -1: zeros; modulus m > 1: symmetric residues drawn
// uniformly from [-(m-1)/2, (m-1)/2], the values the int8 GEMM multiplies
// for the modulus m.
__device__ inline int operand(unsigned &h, int modulus) {
    if (modulus < 0) return 0;
    if (modulus == 0) return (int)(next(h) & 0x7F7F7F7Fu) - 0x3C3C3C3C;
    unsigned w = 0;
    for (int e = 0; e < 4; ++e) {
        const int r = (int)(next(h) % (unsigned)modulus) - (modulus - 1) / 2;
        w |= (unsigned)(r & 0xFF) << (8 * e);
    }
    return (int)w;
}

// clk (may be NULL): per workgroup, the shader clock cycles and the 100 MHz
// real-time ticks between its start and its end, read by thread 0
__global__ __launch_bounds__(256, 1) void mfma16(int iters, int modulus, int *out, long long *clk) {
    long long t0 = 0, r0 = 0;
    if (clk && threadIdx.x == 0) {
        t0 = (long long)__builtin_amdgcn_s_memtime();
        r0 = (long long)__builtin_amdgcn_s_memrealtime();
    }
    v4i acc[8][8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[i][j] = v4i{};
    v4i a[8], b[8];
    unsigned h = threadIdx.x * 2654435761u + blockIdx.x * 40503u + 12345u;
    for (int i = 0; i < 8; ++i)
        for (int e = 0; e < 4; ++e) { a[i][e] = operand(h, modulus); b[i][e] = operand(h, modulus); }
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
    if (clk && threadIdx.x == 0) {
        const long long t1 = (long long)__builtin_amdgcn_s_memtime();
        const long long r1 = (long long)__builtin_amdgcn_s_memrealtime();
        clk[2 * blockIdx.x] = t1 - t0;
        clk[2 * blockIdx.x + 1] = r1 - r0;
    }
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
        for (int e = 0; e < 4; ++e) { a[i][e] = operand(h, 0); b[i][e] = operand(h, 0); }
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
        if (variant == 0) mfma16<<<blocks, 256, 0, st>>>(iters, 0, out, nullptr);
        else if (variant == 1) mfma16<<<blocks, 256, 0, st>>>(iters, -1, out, nullptr);
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

extern "C" double o2m_probe_int8_mfma_residues(int modulus, int blocks, int iters, int *out, double *clock_ghz,
                                               void *stream) {
    if (modulus < 3 || modulus > 256 || blocks <= 0 || iters <= 0 || !out) return -1.0;
    hipStream_t st = (hipStream_t)stream;
    long long *clk = nullptr;
    if (hipMalloc((void **)&clk, sizeof(long long) * 2 * (size_t)blocks) != hipSuccess) return -1.0;
    hipEvent_t e0, e1;
    if (hipEventCreate(&e0) != hipSuccess) { (void)hipFree(clk); return -1.0; }
    if (hipEventCreate(&e1) != hipSuccess) { (void)hipEventDestroy(e0); (void)hipFree(clk); return -1.0; }
    double best = -1.0, best_clock = 0.0;
    long long *host = new long long[2 * (size_t)blocks];
    for (int rep = 0; rep < 4; ++rep) {   // the first launch warms the clock up
        (void)hipEventRecord(e0, st);
        mfma16<<<blocks, 256, 0, st>>>(iters, modulus, out, clk);
        (void)hipEventRecord(e1, st);
        if (hipGetLastError() != hipSuccess || hipEventSynchronize(e1) != hipSuccess) { best = -1.0; break; }
        float ms = 0.0f;
        (void)hipEventElapsedTime(&ms, e0, e1);
        const double tops = (double)blocks * 4 * 64 * 32768.0 * iters / (ms * 1e-3) / 1e12;
        if (rep > 0 && tops > best) {
            if (hipMemcpy(host, clk, sizeof(long long) * 2 * (size_t)blocks, hipMemcpyDeviceToHost) != hipSuccess) {
                best = -1.0;
                break;
            }
            double cyc = 0.0, ticks = 0.0;
            for (int b = 0; b < blocks; ++b) { cyc += (double)host[2 * b]; ticks += (double)host[2 * b + 1]; }
            best = tops;
            best_clock = ticks > 0.0 ? cyc / ticks * 0.1 : 0.0;   // real-time ticks are 100 MHz
        }
    }
    delete[] host;
    (void)hipEventDestroy(e0);
    (void)hipEventDestroy(e1);
    (void)hipFree(clk);
    if (clock_ghz) *clock_ghz = best_clock;
    return best;
}
