/*
 * scgemm.h -- C ABI of the MI355X (gfx950) stochastic-computing GEMM library.
 *
 * Operation (paper "Precision As You Need: Stochastic Computing Is a Dense
 * Adaptive Quantizer", Sec. 3.1 "SC matrix multiplication", Eq. (1), and Sec. 4.2
 * "Datapath"): for each batch entry b,
 *
 *     out[b] (M x N) = SC estimate of  (sA . A[b]) (sB . B[b])^T
 *
 * where A[b] is M x K int8 and B[b] is N x K int8 (both already quantised to
 * [-127, 127] with per-row symmetric scales sA, sB, as the paper assumes).  Every
 * int8 value is encoded into a stream of L_i bits by a comparator against a seeded
 * comparator sequence (Sec. 3.1 "Bitstream generation"), one sequence per operand
 * shared by all of its elements (Sec. 4.2: the table is indexed by boundary and
 * cycle only).  Row i of A runs L_i cycles (Sec. 3.1 "early termination", Sec. 4.2
 * row-length vector).  Bit products are XNOR (bipolar) or AND (unipolar,
 * sign-magnitude), counted over cycles and the inner dimension, and decoded:
 *
 *   bipolar   X_ij = sum_{d<K} sum_{l<L_i} XNOR(zA_idl, zB_jdl)
 *             out_ij = sA_i sB_j 127^2 (2 X_ij / L_i - K)                 (Eq. (1))
 *   unipolar  S_ij = c_pp + c_nn - c_pn - c_np  (signed AND counts)
 *             out_ij = sA_i sB_j 127^2 S_ij / L_i
 *   L_i = 0  gives out_ij = 0 and a zero count.
 *
 * Comparator encoding (the paper leaves the exact maps open; these are fixed here):
 *   sequence  r_l in [0,255]: 32-bit Galois LFSR (right shift, feedback mask
 *             0x80200003, polynomial x^32+x^22+x^2+x+1), 8 steps per draw, first
 *             output bit most significant; initial state = upper 32 bits of
 *             SplitMix64(2*seed + op), op 0 for A and 1 for B, 0 replaced by 1.
 *   bipolar   z = [r_l < beta(q)],  beta(q)   = floor((256 (q+127) + 127) / 254)
 *   unipolar  z = [r_l < beta_u(q)], beta_u(q) = floor((256 |q| + 63) / 127),
 *             sign = (q < 0)
 *   -128, outside the quantiser's range, gives the same streams as -127 (every
 *   boundary it would have lies at 0 or at 256 and above).
 *
 * Second comparator source, rng = SC_RNG_SOBOL8_CBSG (Sec. 4.2 "cumulative-indicator
 * C-BSG" and Sec. A.1 Eq. (4)-(6), readings fixed here): A draws from Sobol dimension 1
 * (the base-2 radical inverse), B from Sobol dimension 2 (polynomial x + 1, direction
 * numbers m = 1, 3, 5, 15, 17, 51, 85, 255), both 8-bit, natural order, each XORed with
 * the digital shift (SplitMix64(2*seed + op) >> 56).  A's stream is its comparator
 * stream; B's generator is gated by it: B walks r^B with one counter on the cycles
 * where A emits 1 and another on the cycles where A emits 0, so with
 * c = #{l < L_i : rA_l < beta_A}, the XNOR count of one element pair is
 *   #{k < c : rB_k < beta_B} + #{k < L_i - c : rB_k >= beta_B}
 * and the unipolar AND count is #{k < c : rB_k < beta_uB}.  Needs L_max <= 256.
 *
 * Memory: every array pointer is a HIP DEVICE pointer; the caller owns all memory.
 * A pointer may be NULL only when its array has no elements (e.g. A when K = 0).
 * The library allocates nothing in sc_gemm and keeps no state between calls; all
 * temporaries live in the caller's workspace.  Calls are asynchronous on `stream`
 * (a hipStream_t passed as void*; NULL = the default stream).  Two calls that share
 * one workspace must be ordered on the same stream.
 *
 * Errors: arguments are checked on the host before anything is enqueued and a
 * negative SC_ERR_* code is returned; nothing is launched then.  Launch failures
 * return SC_ERR_HIP.  Stream lengths live on the device, so their range is checked
 * by a kernel into a status word in the workspace; rows whose L_i is outside
 * [0, L_max] are computed as L_i = 0 and sc_gemm_status() reports
 * SC_ERR_DEVICE_STATUS.
 */
#ifndef SCGEMM_H
#define SCGEMM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    SC_OK = 0,
    SC_ERR_NULL = -1,          /* a required pointer is NULL */
    SC_ERR_SHAPE = -2,         /* batch, M, N or K negative, K > SC_K_LIMIT,
                                  K * L_max > SC_KL_LIMIT, or a problem whose workspace
                                  layout exceeds its limits (size_t overflow, more than
                                  2^20 work ranges); checked before the pointers */
    SC_ERR_LEN = -3,           /* L_max outside [1, SC_L_MAX_LIMIT] ([1, 256] for C-BSG),
                                  or L_hint outside [0, L_max] */
    SC_ERR_POLARITY = -4,      /* polarity not one of SC_BIPOLAR_XNOR / SC_UNIPOLAR_AND_SM */
    SC_ERR_RNG = -5,           /* rng not one of SC_RNG_* (or op not 0/1) */
    SC_ERR_WORKSPACE = -6,     /* workspace NULL or smaller than sc_gemm_workspace_size() */
    SC_ERR_HIP = -7,           /* a HIP runtime call or kernel launch failed */
    SC_ERR_DEVICE_STATUS = -8, /* (sc_gemm_status) some L_i was outside [0, L_max] */
    SC_ERR_STRIDE = -9,        /* a row stride is smaller than the row length */
    SC_ERR_RESERVED = -10      /* the descriptor's reserved field is not 0 */
};

enum { SC_BIPOLAR_XNOR = 0, SC_UNIPOLAR_AND_SM = 1 };
enum { SC_RNG_LFSR32 = 0, SC_RNG_SOBOL8_CBSG = 1 };

/* Counting: every stream bit becomes an fp4 (e2m1) value in {-1, 0, +1} and the matrix
 * cores sum their products in fp32.  A work unit sums at most 2^24 products per output,
 * so every partial sum is an exact integer; longer inner ranges are split into up to 8
 * such units whose int32 partial counts are added exactly.  Hence K * L_max <= 2^27. */

#define SC_L_MAX_LIMIT 4096             /* largest supported stream length */
#define SC_K_LIMIT (1 << 20)            /* largest inner dimension */
#define SC_KL_LIMIT (1ll << 27)         /* largest K * L_max */

typedef struct sc_gemm_desc {
    int32_t batch;              /* >= 0 independent problems */
    int32_t M, N, K;            /* A[b] is M x K, B[b] is N x K, out[b] is M x N */
    int64_t lda, ldb, ldo;      /* row strides in elements (>= K, >= K, >= N) */
    int64_t strideA, strideB, strideO;   /* batch strides in elements; 0 = broadcast */
    int64_t strideSA, strideSB;          /* batch strides of sA (M) and sB (N) */
    int64_t strideL;                     /* batch stride of L_per_row (M) */
    int32_t L_max;              /* 1..SC_L_MAX_LIMIT; every L_i must lie in [0, L_max] */
    int32_t polarity;           /* SC_BIPOLAR_XNOR or SC_UNIPOLAR_AND_SM */
    int32_t rng;                /* SC_RNG_LFSR32 or SC_RNG_SOBOL8_CBSG */
    int32_t L_hint;             /* optional expected mean of the L_i (0 = unknown, taken as
                                   L_max); only tunes how GEMM tiles are split over the
                                   compute units, never changes a result; 0..L_max */
    int32_t reserved;           /* must be 0 */
    uint64_t seed;              /* comparator seed; same seed => bit-identical results */
    void *prof_event_begin;     /* optional hipEvent_t recorded when the counting GEMM's */
    void *prof_event_end;       /*   first kernel starts and when its last kernel ends (the
                                     events ride on the kernels' dispatches); NULL = off */
} sc_gemm_desc;

/* Bytes of device workspace sc_gemm needs for `desc` on the current HIP device (the size
 * depends on the device's compute-unit count, which is queried once per device; with no
 * device visible an MI355X's 256 is assumed).  Enqueues nothing.  Returns SC_OK and writes
 * *bytes, or a negative SC_ERR_* code for a bad desc. */
int sc_gemm_workspace_size(const sc_gemm_desc *desc, size_t *bytes);

/*
 * The SC GEMM (Eq. (1) with per-row stream lengths).
 *   A          int8,  A[b*strideA + i*lda + d]
 *   sA         fp32,  sA[b*strideSA + i]       per-row scales of A
 *   B          int8,  B[b*strideB + j*ldb + d]
 *   sB         fp32,  sB[b*strideSB + j]       per-row scales of B
 *   L_per_row  int32, L[b*strideL + i]         stream length of row i of A
 *   out        fp32,  out[b*strideO + i*ldo + j]   decoded estimate (written)
 *   counts     int32, same layout as out, NULLABLE: raw X_ij (bipolar) or S_ij
 *              (unipolar) for bit-exact checks
 *   workspace  device memory of at least sc_gemm_workspace_size() bytes, 256-byte
 *              aligned; contents on entry are ignored, contents on exit are
 *              internal (only sc_gemm_status reads them)
 *   stream     hipStream_t or NULL
 * Returns SC_OK once everything is enqueued (results are ready when the stream
 * reaches that point), or a negative SC_ERR_* code.
 */
int sc_gemm(const sc_gemm_desc *desc,
            const int8_t *A, const float *sA,
            const int8_t *B, const float *sB,
            const int32_t *L_per_row,
            float *out, int32_t *counts,
            void *workspace, size_t workspace_bytes,
            void *stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): sc_gemm with the same arguments except
 * the workspace, which the library provides instead -- a static device array of
 * SC_NOALLOC_WORKSPACE_BYTES on each device the library runs on, held until the process
 * ends.  It calls no hipMalloc, hipFree or other allocating routine.
 *   Returns SC_ERR_WORKSPACE when sc_gemm_workspace_size(desc) exceeds
 *   SC_NOALLOC_WORKSPACE_BYTES (e.g. 6304 x 768 x 3072 at L = 128 needs 35 MiB), and the
 *   other codes as sc_gemm.
 *   status_out  NULLABLE device int32: after the call it holds the call's device status
 *               word, 0 when every L_i was in [0, L_max], nonzero (bit 0) otherwise.
 * Every call on a device uses that device's one array, which keeps the last call's
 * contents (each call rewrites all it reads): calls that overlap in time on one device
 * race, so order them, e.g. on one stream.
 */
#define SC_NOALLOC_WORKSPACE_BYTES ((size_t)64 << 20)
int sc_gemm_noalloc(const sc_gemm_desc *desc,
                    const int8_t *A, const float *sA,
                    const int8_t *B, const float *sB,
                    const int32_t *L_per_row,
                    float *out, int32_t *counts, int32_t *status_out,
                    void *stream);

/* Synchronises `stream` and reads the device status word that the last sc_gemm on
 * `workspace` wrote: SC_OK, or SC_ERR_DEVICE_STATUS if some L_i was out of range. */
int sc_gemm_status(const void *workspace, void *stream);

/*
 * The comparator sequence r_0 .. r_{n-1} of operand `op` (0 = A, 1 = B) for `seed`
 * and source `rng`, computed on the device exactly as sc_gemm computes it (Sec. 3.1
 * "Bitstream generation"; LFSR or scrambled Sobol-8 of Sec. A.1 under the readings
 * above).  `out` is a device buffer of n bytes.  1 <= n <= SC_L_MAX_LIMIT (<= 256 for
 * SC_RNG_SOBOL8_CBSG).  Asynchronous on `stream`.
 */
int sc_comparator_sequence(uint64_t seed, int32_t op, int32_t rng, int32_t n, uint8_t *out,
                           void *stream);

/*
 * Symmetric int8 quantisation of fp32 rows, the input preparation the SC GEMM takes
 * as given (Sec. 3.1: s_i = max_d |X_id| / q_max, integers in [-q_max, q_max]) and
 * that the paper's kernel fuses with emitting the row scale (Sec. 4.2 "fused
 * quantization").  For each batch entry b and row i of X (rows x K fp32):
 *   per_tensor = 0:  s_i = m_i / 127 with m_i = max_d |X_id|
 *   per_tensor = 1:  s_i = m / 127 for every row, m = max over the batch entry
 *   Q_id = clamp(rint(X_id / s_i), -127, 127), round half to even; s = 0 gives Q = 0.
 * All arithmetic is IEEE fp32 (the division correctly rounded), so the result is
 * bit-identical to the same formula evaluated in fp32 on the host.
 *   X       fp32 X[b*strideX + i*ldx + d]                (device, read)
 *   Q       int8 Q[b*strideQ + i*ldq + d]                (device, written)
 *   scale   fp32 scale[b*strideS + i]                    (device, written)
 *   rowmax  fp32 rowmax[b*strideS + i] = m_i, NULLABLE   (device, written): the row
 *           metric ||X_i||_inf of the mixed-precision policy (Sec. 4.4)
 * Needs ldx >= K, ldq >= K.  No workspace.  Asynchronous on `stream`.
 */
int sc_quantize(int32_t batch, int32_t rows, int32_t K, const float *X, int64_t ldx,
                int64_t strideX, int32_t per_tensor, int8_t *Q, int64_t ldq, int64_t strideQ,
                float *scale, float *rowmax, int64_t strideS, void *stream);

#define SC_MP_MAX_LEVELS 32

/*
 * Per-row stream lengths from a row metric (Sec. 4.4 "Row metrics" and "Threshold
 * fitting"): within each batch entry (one operator call) the metric is min-max
 * normalised, t_i = (g_i - min_j g_j) / (max_j g_j - min_j g_j) in fp32 (t_i = 0 when
 * all g_j are equal), and row i gets L_i = ladder[k*] with k* the first level whose
 * threshold it reaches, t_i >= tau[k] (k = 0 .. n_levels-2), else the shortest,
 * ladder[n_levels-1].
 *   metric  fp32 metric[b*strideM + i]   (device), e.g. the rowmax of sc_quantize
 *   tau     n_levels-1 fp32 thresholds in [0,1], non-increasing   (HOST array)
 *   ladder  n_levels int32 lengths, strictly decreasing, >= 0     (HOST array)
 *   L_out   int32 L_out[b*strideL + i]   (device, written): feeds sc_gemm directly
 * 1 <= n_levels <= SC_MP_MAX_LEVELS.  The thresholds come from an offline calibration
 * that is not part of this library.  Asynchronous on `stream`.
 */
int sc_mp_lengths(int32_t batch, int32_t M, const float *metric, int64_t strideM,
                  const float *tau, const int32_t *ladder, int32_t n_levels, int32_t *L_out,
                  int64_t strideL, void *stream);

/* Human-readable name of a status code (static string). */
const char *sc_strerror(int code);

/* Library ABI version (major*10000 + minor*100 + patch). */
int sc_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SCGEMM_H */
