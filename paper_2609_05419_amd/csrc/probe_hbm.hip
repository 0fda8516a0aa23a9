// Measurement probe (not part of the 2M path): the HBM bandwidth the chip
// sustains for plain streaming kernels with 16-byte accesses, for the
// read:write mixes of the pre and post steps of the path (the paper puts them
// at Theta(mn + mk + nk) work, i.e. bandwidth-bound):
//   kind 0  read only            (the scaling maxima: 16 B read per element)
//   kind 1  write only
//   kind 2  copy, 1 read : 1 write
//   kind 3  1 read : 2 writes    (residues at N = 16: 16 B read, 32 B written)
//   kind 4  2 reads : 1 write    (CRT at N = 16: 32 B read, 16 B written)
// Workgroup b owns `chunks` consecutive 4 KB pieces of every buffer (thread t
// the 16-byte chunks t, t + 256, ...), all loads issued before the stores.
// Measured on MI355X, one chunk per thread and one workgroup per 4 KB is the
// fastest form (read 6.8, write 6.9, 1:2 and 2:1 mixes 6.0 TB/s); a
// grid-stride loop over a few thousand workgroups reaches 4.4-5.8 TB/s.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "o2m_probe.h"

namespace {

constexpr int kThreads = 256;

__device__ inline uint4 mix(uint4 x, uint4 y) { return make_uint4(x.x ^ y.x, x.y ^ y.y, x.z ^ y.z, x.w ^ y.w); }

template <int KIND, int CH>
__global__ __launch_bounds__(kThreads) void stream_kernel(const uint4 *__restrict__ a, const uint4 *__restrict__ b,
                                                          uint4 *__restrict__ c, uint4 *__restrict__ d, size_t n,
                                                          uint4 *__restrict__ sink) {
    const size_t base = (size_t)blockIdx.x * kThreads * CH + threadIdx.x;
    const uint4 pat = make_uint4(0x01020304u, 0x05060708u, (unsigned)base, 0x0A0B0C0Du);
    uint4 x[CH], y[CH];
    uint4 acc = make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int u = 0; u < CH; ++u) {
        const size_t j = base + (size_t)u * kThreads;
        if (j < n && (KIND == 0 || KIND >= 2)) x[u] = a[j];
        if (j < n && KIND == 4) y[u] = b[j];
    }
#pragma unroll
    for (int u = 0; u < CH; ++u) {
        const size_t j = base + (size_t)u * kThreads;
        if (j >= n) break;
        if (KIND == 0) acc = mix(acc, x[u]);
        if (KIND == 1) c[j] = pat;
        if (KIND == 2) c[j] = x[u];
        if (KIND == 3) { c[j] = x[u]; d[j] = mix(x[u], pat); }
        if (KIND == 4) c[j] = mix(x[u], y[u]);
    }
    // the read-only kind keeps its loads alive through a store that real data
    // takes only by accident (into the 4 KB sink)
    if (KIND == 0 && acc.x == pat.x && acc.y == pat.y && acc.z == pat.z && acc.w == pat.w) sink[threadIdx.x] = acc;
}

template <int KIND>
void launch(int chunks, unsigned blocks, const uint4 *A, const uint4 *B, uint4 *C, uint4 *D, size_t n, uint4 *S,
            hipStream_t st) {
    switch (chunks) {
    case 1: stream_kernel<KIND, 1><<<blocks, kThreads, 0, st>>>(A, B, C, D, n, S); break;
    case 2: stream_kernel<KIND, 2><<<blocks, kThreads, 0, st>>>(A, B, C, D, n, S); break;
    case 4: stream_kernel<KIND, 4><<<blocks, kThreads, 0, st>>>(A, B, C, D, n, S); break;
    default: stream_kernel<KIND, 8><<<blocks, kThreads, 0, st>>>(A, B, C, D, n, S); break;
    }
}

}  // namespace

extern "C" double o2m_probe_hbm(int kind, const void *a, const void *b, void *c, void *d, size_t bytes, int chunks,
                                void *sink, void *stream) {
    if (kind < 0 || kind > 4 || bytes < 16) return -1.0;
    if (chunks != 1 && chunks != 2 && chunks != 4 && chunks != 8) return -1.0;
    const bool need_a = kind == 0 || kind >= 2, need_b = kind == 4, need_c = kind >= 1, need_d = kind == 3;
    if ((need_a && !a) || (need_b && !b) || (need_c && !c) || (need_d && !d) || (kind == 0 && !sink)) return -1.0;
    const size_t n = bytes / 16;
    const size_t per_block = (size_t)kThreads * chunks;
    const size_t nblocks = (n + per_block - 1) / per_block;
    if (nblocks > 0x7FFFFFFFu) return -1.0;
    hipStream_t st = (hipStream_t)stream;
    const uint4 *A = (const uint4 *)a, *B = (const uint4 *)b;
    uint4 *C = (uint4 *)c, *D = (uint4 *)d, *S = (uint4 *)sink;
    hipEvent_t e0, e1;
    if (hipEventCreate(&e0) != hipSuccess) return -1.0;
    if (hipEventCreate(&e1) != hipSuccess) { (void)hipEventDestroy(e0); return -1.0; }
    const double moved = (double)(n * 16) * (kind == 0 || kind == 1 ? 1 : kind == 2 ? 2 : 3);
    double best = -1.0;
    for (int rep = 0; rep < 6; ++rep) {   // the first launch warms up
        (void)hipEventRecord(e0, st);
        switch (kind) {
        case 0: launch<0>(chunks, (unsigned)nblocks, A, B, C, D, n, S, st); break;
        case 1: launch<1>(chunks, (unsigned)nblocks, A, B, C, D, n, S, st); break;
        case 2: launch<2>(chunks, (unsigned)nblocks, A, B, C, D, n, S, st); break;
        case 3: launch<3>(chunks, (unsigned)nblocks, A, B, C, D, n, S, st); break;
        default: launch<4>(chunks, (unsigned)nblocks, A, B, C, D, n, S, st); break;
        }
        (void)hipEventRecord(e1, st);
        if (hipGetLastError() != hipSuccess || hipEventSynchronize(e1) != hipSuccess) { best = -1.0; break; }
        float ms = 0.0f;
        (void)hipEventElapsedTime(&ms, e0, e1);
        const double gbs = moved / (ms * 1e-3) / 1e9;
        if (rep > 0 && gbs > best) best = gbs;
    }
    (void)hipEventDestroy(e0);
    (void)hipEventDestroy(e1);
    return best;
}
