/*
 * scpeak.h -- C ABI of libscpeak, the measurement companion of libscgemm (not part of
 * the SC GEMM path).
 *
 * The benchmark reports the SC GEMM's stream-bit-op rate against the rate at which the
 * vector ALUs of the device can do the same work as packed words: for 32 bit pairs one
 * bitwise product (AND; XNOR costs the same) and one population count accumulated into
 * a running total (v_bcnt_u32_b32 with the total as second source), i.e. two VALU
 * instructions per 32 stream-bit-ops (Sec. 4.2: the count is tiled AND-and-popcount
 * over the D x L binary comparisons).  Rather than derive that rate from a data sheet,
 * sc_peak_valu_bitop measures it: every wave runs 16 independent AND -> popcount chains
 * on registers (no memory traffic in the loop), and the shader clock under that load is
 * read inside the kernel (cycle counter against the constant-rate wall clock).
 *
 * The call allocates two small device buffers, synchronises the device and frees them.
 */
#ifndef SCPEAK_H
#define SCPEAK_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct sc_peak_result {
    double seconds;          /* kernel time (HIP events) */
    double lane_ops_per_s;   /* VALU lane-instructions per second (AND and popcount each count) */
    double bitops_per_s;     /* stream-bit-ops per second: 32 bit pairs per 2 lane-instructions */
    double clock_hz;         /* mean shader clock over the waves, measured in the kernel */
    int32_t cus;             /* compute units of the device */
    int32_t waves_per_simd;  /* waves resident per SIMD in the measurement */
} sc_peak_result;

/* Measures on the current device with `waves_per_simd` (1..8) waves per SIMD and `iters`
 * (>= 1) loop trips of 32 VALU instructions per lane.  Returns 0, -1 for bad arguments or
 * a NULL result, -7 when a HIP call fails. */
int sc_peak_valu_bitop(int32_t waves_per_simd, int32_t iters, sc_peak_result *result);

#ifdef __cplusplus
}
#endif

#endif /* SCPEAK_H */
