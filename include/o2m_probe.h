/*
 * o2m_probe.h -- measurement probe shipped beside the 2M library (separate
 * library libo2m_probe.so; not part of the 2M path).
 *
 * The int8 GEMM of the 2M path (K3) is bounded by the int8 MFMA rate the
 * MI355X sustains, which on random operands sits below the nominal 5.0 POP/s
 * because the part lowers its clock to stay in its power budget.  This probe
 * measures that practical ceiling: MFMAs on operands held in registers, with
 * no memory traffic.
 */
#ifndef O2M_PROBE_H
#define O2M_PROBE_H

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

#ifdef __cplusplus
}
#endif

#endif /* O2M_PROBE_H */
