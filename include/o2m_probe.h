/*
 * o2m_probe.h -- measurement probe shipped beside the 2M library (separate
 * library libo2m_probe.so; not part of the 2M path).
 *
 * The int8 GEMM of the 2M path (K3) is bounded by the int8 MFMA rate the
 * MI355X sustains, which on random operands sits below the nominal 5.0 POP/s
 * because the part lowers its clock to stay in its power budget.  This probe
 * measures that practical ceiling: MFMAs on operands held in registers, with
 * no memory traffic.  The pre and post steps are bounded by HBM bandwidth;
 * o2m_probe_hbm measures what plain streaming kernels sustain for their
 * read:write mixes.
 */
#ifndef O2M_PROBE_H
#define O2M_PROBE_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Launch `blocks` workgroups of 4 waves, each wave running `iters` rounds of
   64 independent v_mfma_i32_16x16x64_i8 (variant 0: random operands;
   variant 1: zero operands) or 16 v_mfma_i32_32x32x32_i8 (variant 2: random
   operands), on `stream`, four times; return the best int8 rate of the last
   three launches in TOP/s, or a negative value on a bad argument or HIP
   error.  out: caller-owned device int array of blocks * 256 elements that
   receives one checksum per thread.  Synchronizes the stream. */
double o2m_probe_int8_mfma(int variant, int blocks, int iters, int *out, void *stream);

/* As variant 0 of o2m_probe_int8_mfma, with operands drawn uniformly from
   the symmetric residues [-(m-1)/2, (m-1)/2] of modulus m (3 <= m <= 256):
   the values the 2M path's int8 GEMM multiplies for that modulus.  Writes
   the average shader clock of the best launch (GHz, from the shader clock
   counter against the 100 MHz real-time counter, per workgroup) to
   *clock_ghz if it is not NULL.  Allocates and frees a small device buffer. */
double o2m_probe_int8_mfma_residues(int modulus, int blocks, int iters, int *out, double *clock_ghz,
                                    void *stream);

/* HBM bandwidth of a streaming kernel with 16-byte accesses over buffers of
   `bytes` each (caller-owned device memory): each workgroup of 256 threads
   owns `chunks` (1, 2, 4 or 8) consecutive 4 KB pieces of every buffer.
   Launched on `stream` six times; returns the best GB/s of the last five
   launches counting every byte read and written, or a negative value on a
   bad argument or HIP error.  kind 0: read a (sink: a 4 KB device buffer,
   rarely written); 1: write c; 2: copy a -> c; 3: read a, write c and d
   (1 read : 2 writes); 4: read a and b, write c (2 reads : 1 write).
   Unused pointers may be NULL.  Synchronizes the stream. */
double o2m_probe_hbm(int kind, const void *a, const void *b, void *c, void *d, size_t bytes, int chunks,
                     void *sink, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* O2M_PROBE_H */
