/*
 * sc_oracle.c -- plain CPU oracle for emulated stochastic-computing (SC) matrix
 * multiplication.  TEST INFRASTRUCTURE ONLY: it is called by the tests, by the
 * smoke check and by the benchmark's CPU-baseline leg, never by the product path.
 * It shares no code, header, table or constant generator with the HIP library.
 *
 * Everything here is deliberately slow and literal: every comparator bit of every
 * stream is materialised as one byte, products are formed bit by bit with the
 * XNOR (bipolar) or AND (unipolar) gate, counts are plain sums, and the decode is
 * done in float64.
 *
 * What it follows (paper: "Precision As You Need: Stochastic Computing Is a Dense
 * Adaptive Quantizer"):
 *   - Sec. 3.1 "Encoding": unipolar value v in [0,1] -> Pr[z=1] = v; bipolar value
 *     v in [-1,1] -> Pr[z=1] = (v+1)/2.
 *   - Sec. 3.1 "Bitstream generation": comparator SNG, z_l = 1[r_l < input], with a
 *     signed int8 offset onto the unsigned RNG range; decode (2c - L)/L.
 *   - Sec. 3.1 "SC matrix multiplication", Eq. (1): per-row symmetric int8 inputs,
 *     XNOR products summed over cycles and the inner dimension, rescaled by
 *     s^A_i s^B_j q_max^2.
 *   - Sec. 3.1 "Precision and early termination": any non-negative integer length;
 *     row i stops at its own L_i (Sec. 4.2, row-length vector).
 *   - Sec. 4.2 "Datapath": V = 257 comparison boundaries per int8 value; the same
 *     comparator sequence is shared by every element of an operand (the table is
 *     indexed by boundary and cycle only).
 *   - Sec. A.1: LFSRs are the plain PRNG option for the comparator sequence.
 *
 * Readings taken where the paper is silent:
 *   R-LFSR   32-bit Galois LFSR, right shift, feedback mask 0x80200003, i.e. the
 *            polynomial x^32+x^22+x^2+x+1 (primitive, so the period is 2^32-1).  One draw is 8
 *            steps; the 8 output bits form a byte, first output bit most significant.
 *   R-SEED   initial state = upper 32 bits of SplitMix64(2*seed + op), op = 0 for
 *            the left operand A and 1 for the right operand B; a zero state is
 *            replaced by 1.  SplitMix64: Steele, Lea and Flood, OOPSLA 2014.
 *   R-BETA   bipolar boundary beta(q) = floor((256*(q+127) + 127) / 254) in [0,256]
 *            (round half up of 256*(q+127)/254); unipolar sign-magnitude boundary
 *            beta_u(q) = floor((256*|q| + 63) / 127), sign = (q < 0).
 *   R-SHARE  one sequence per operand per call, shared by all of its elements.
 *   R-L0     L_i = 0 is allowed: counts and outputs are 0.
 *   R-UNI    unipolar variant: magnitude streams split by sign into X+ and X-, the
 *            four partial products counted literally, S = c_pp + c_nn - c_pn - c_np.
 *
 * Second comparator source, the paper's own (Sec. 4.2 "Datapath: cumulative-indicator
 * C-BSG"; Sec. A.1 scrambled Sobol sequences and conditional bitstream generation,
 * Eq. (4)-(6)).  Readings taken:
 *   R-SOBOL  Sobol-8: r_k = shift XOR (XOR over the set bits j of k of V_j), k < 256,
 *            8-bit direction numbers V_j = m_j << (8 - j) from the published
 *            primitive-polynomial recurrence (Bratley and Fox; Joe and Kuo):
 *            dimension 1 m_j = 1 (van der Corput), dimension 2 polynomial x + 1 with
 *            m_1 = 1, m_j = 2 m_{j-1} xor m_{j-1}.  The digital shift of operand op is
 *            the top 8 bits of SplitMix64(2*seed + op).  A uses dimension 1, B dimension 2.
 *   R-CBSG   A's stream is its comparator stream on its own Sobol sequence.  B's
 *            generator is gated by A's stream (Fig. 1(c)): B keeps two counters that walk
 *            the same sequence r^B, one advanced on the cycles where A emits 1 and one on
 *            the cycles where A emits 0; at each cycle B compares the draw its active
 *            counter points at against its boundary.  This matches both conditional
 *            distributions of Eq. (6) to the marginal of r^B.
 *   R-CBSG-L L_max <= 256 (one Sobol-8 period); a shorter row takes the prefix.
 *
 * Build: gcc -O2 -fopenmp -shared -fPIC sc_oracle.c -o libsc_oracle.so
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <omp.h>

#define QMAX 127

/* SplitMix64 as published by Steele, Lea and Flood (2014): one increment of the
 * Weyl state by the golden-ratio constant, then the variant-13 finaliser. */
uint64_t oracle_splitmix64(uint64_t x)
{
    uint64_t z = x + 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

/* R-SEED: initial LFSR state of operand `op` (0 = A, 1 = B). */
uint32_t oracle_seed_state(uint64_t seed, uint32_t op)
{
    uint32_t s = (uint32_t)(oracle_splitmix64(2ull * seed + (uint64_t)op) >> 32);
    return s ? s : 1u;
}

/* R-LFSR: one step of the Galois right-shift register; returns the output bit. */
static int lfsr_step(uint32_t *s)
{
    int out = (int)(*s & 1u);
    *s >>= 1;
    if (out) *s ^= 0x80200003u;
    return out;
}

/* R-LFSR: n comparator draws r_0 .. r_{n-1} in [0,255] from initial state `state`;
 * each draw takes 8 steps, first output bit becomes the most significant bit. */
void oracle_lfsr_draws(uint32_t state, int32_t n, uint8_t *out)
{
    uint32_t s = state;
    for (int32_t l = 0; l < n; ++l) {
        int v = 0;
        for (int k = 0; k < 8; ++k) v = (v << 1) | lfsr_step(&s);
        out[l] = (uint8_t)v;
    }
}

/* Raw register states after each of n steps (used to pin the register to the
 * polynomial algebra in the tests). */
void oracle_lfsr_states(uint32_t state, int32_t n, uint32_t *out)
{
    uint32_t s = state;
    for (int32_t k = 0; k < n; ++k) { lfsr_step(&s); out[k] = s; }
}

/* R-BETA, bipolar: int8 q in [-127,127] -> boundary in [0,256]. */
int32_t oracle_beta_bipolar(int32_t q)
{
    return (256 * (q + QMAX) + 127) / 254;
}

/* R-BETA, unipolar sign-magnitude: |q| in [0,127] -> boundary in [0,256]. */
int32_t oracle_beta_unipolar(int32_t q)
{
    int32_t a = q < 0 ? -q : q;
    return (256 * a + 63) / 127;
}

/* Comparator SNG (Sec. 3.1): z_l = 1[r_l < beta] for l < len; bytes. */
static void sng(const uint8_t *r, int32_t beta, int32_t len, uint8_t *z)
{
    for (int32_t l = 0; l < len; ++l) z[l] = (uint8_t)((int32_t)r[l] < beta ? 1 : 0);
}

/* Materialised streams of one operand, for inspection by the tests:
 * z[(row*K + d)*len + l] for rows x K elements, `len` cycles each.
 * polarity 0: bipolar streams of beta(q); polarity 1: unipolar magnitude streams
 * of beta_u(q) (the sign is not folded in). */
void oracle_streams(int32_t rows, int32_t K, const int8_t *X, int32_t polarity,
                    uint64_t seed, uint32_t op, int32_t len, uint8_t *z)
{
    uint8_t *r = (uint8_t *)malloc((size_t)(len > 0 ? len : 1));
    oracle_lfsr_draws(oracle_seed_state(seed, op), len, r);
    for (int32_t i = 0; i < rows; ++i)
        for (int32_t d = 0; d < K; ++d) {
            int32_t q = X[(size_t)i * K + d];
            int32_t beta = polarity == 0 ? oracle_beta_bipolar(q) : oracle_beta_unipolar(q);
            sng(r, beta, len, z + ((size_t)i * K + d) * (size_t)len);
        }
    free(r);
}

/*
 * The SC GEMM itself.  A is M x K int8 row-major, B is N x K int8 row-major
 * (out = A . B^T, Eq. (1) with the paper's N, D, M renamed M, K, N).  L[i] is
 * row i's stream length, 0 <= L[i] <= L_max.  sA[M], sB[N] are the symmetric
 * per-row scales.  polarity 0 = bipolar XNOR, 1 = unipolar AND, sign-magnitude.
 *
 * counts (M x N, int32, may be NULL):
 *   bipolar   X_ij = sum_d sum_{l < L_i} XNOR(zA_idl, zB_jdl)
 *   unipolar  S_ij = c_pp + c_nn - c_pn - c_np  (four literal partial products)
 * out (M x N, float64, may be NULL):
 *   bipolar   sA_i sB_j q_max^2 (2 X_ij / L_i - K)         (Eq. (1))
 *   unipolar  sA_i sB_j q_max^2 S_ij / L_i
 *   L_i = 0 gives 0.
 * Returns 0, or -1 for bad arguments.  nthreads <= 0 leaves OpenMP's default.
 */
int oracle_sc_gemm(int32_t M, int32_t N, int32_t K,
                   const int8_t *A, const int8_t *B,
                   const float *sA, const float *sB,
                   const int32_t *L, int32_t L_max,
                   int32_t polarity, uint64_t seed,
                   int32_t *counts, double *out, int32_t nthreads)
{
    if (M < 0 || N < 0 || K < 0 || L_max < 0 || (polarity != 0 && polarity != 1)) return -1;
    for (int32_t i = 0; i < M; ++i)
        if (L[i] < 0 || L[i] > L_max) return -1;
    if (M == 0 || N == 0) return 0;

    const size_t Lm = (size_t)(L_max > 0 ? L_max : 1);
    uint8_t *rA = (uint8_t *)malloc(Lm), *rB = (uint8_t *)malloc(Lm);
    oracle_lfsr_draws(oracle_seed_state(seed, 0), L_max, rA);
    oracle_lfsr_draws(oracle_seed_state(seed, 1), L_max, rB);

    /* B streams for every (j, d), L_max cycles.  Unipolar keeps the two signed
     * halves B+ and B- as separate streams, exactly as the four-partial split. */
    const size_t bsz = (size_t)N * K * Lm;
    uint8_t *zBp = (uint8_t *)malloc(bsz);
    uint8_t *zBn = polarity == 1 ? (uint8_t *)malloc(bsz) : NULL;
    if (!rA || !rB || !zBp || (polarity == 1 && !zBn)) {
        free(rA); free(rB); free(zBp); free(zBn);
        return -2;
    }
    for (int32_t j = 0; j < N; ++j)
        for (int32_t d = 0; d < K; ++d) {
            int32_t q = B[(size_t)j * K + d];
            uint8_t *zp = zBp + ((size_t)j * K + d) * Lm;
            if (polarity == 0) {
                sng(rB, oracle_beta_bipolar(q), L_max, zp);
            } else {
                uint8_t *zn = zBn + ((size_t)j * K + d) * Lm;
                uint8_t *mag = q < 0 ? zn : zp, *zero = q < 0 ? zp : zn;
                sng(rB, oracle_beta_unipolar(q), L_max, mag);
                memset(zero, 0, Lm);
            }
        }

    if (nthreads > 0) omp_set_num_threads(nthreads);
    int err = 0;
#pragma omp parallel
    {
        uint8_t *zAp = (uint8_t *)malloc((size_t)K * Lm);
        uint8_t *zAn = (uint8_t *)malloc((size_t)K * Lm);
        if (!zAp || !zAn) {
#pragma omp atomic write
            err = -2;
        }
#pragma omp for schedule(dynamic, 1)
        for (int32_t i = 0; i < M; ++i) {
            if (!zAp || !zAn) continue;
            const int32_t Li = L[i];
            /* Row i's streams, L_i cycles (early termination of the whole row). */
            for (int32_t d = 0; d < K; ++d) {
                int32_t q = A[(size_t)i * K + d];
                uint8_t *zp = zAp + (size_t)d * Lm;
                if (polarity == 0) {
                    sng(rA, oracle_beta_bipolar(q), Li, zp);
                } else {
                    uint8_t *zn = zAn + (size_t)d * Lm;
                    uint8_t *mag = q < 0 ? zn : zp, *zero = q < 0 ? zp : zn;
                    sng(rA, oracle_beta_unipolar(q), Li, mag);
                    memset(zero, 0, (size_t)Li);
                }
            }
            for (int32_t j = 0; j < N; ++j) {
                int64_t c = 0;
                if (polarity == 0) {
                    /* XNOR(a, b) = 1 - (a xor b), summed over d and l < L_i. */
                    for (int32_t d = 0; d < K; ++d) {
                        const uint8_t *za = zAp + (size_t)d * Lm;
                        const uint8_t *zb = zBp + ((size_t)j * K + d) * Lm;
                        int32_t s = 0;
                        for (int32_t l = 0; l < Li; ++l) s += 1 - (za[l] ^ zb[l]);
                        c += s;
                    }
                } else {
                    int64_t cpp = 0, cnn = 0, cpn = 0, cnp = 0;
                    for (int32_t d = 0; d < K; ++d) {
                        const uint8_t *ap = zAp + (size_t)d * Lm, *an = zAn + (size_t)d * Lm;
                        const uint8_t *bp = zBp + ((size_t)j * K + d) * Lm;
                        const uint8_t *bn = zBn + ((size_t)j * K + d) * Lm;
                        int32_t spp = 0, snn = 0, spn = 0, snp = 0;
                        for (int32_t l = 0; l < Li; ++l) {
                            spp += ap[l] & bp[l];
                            snn += an[l] & bn[l];
                            spn += ap[l] & bn[l];
                            snp += an[l] & bp[l];
                        }
                        cpp += spp; cnn += snn; cpn += spn; cnp += snp;
                    }
                    c = cpp + cnn - cpn - cnp;
                }
                const size_t o = (size_t)i * N + j;
                if (counts) counts[o] = (int32_t)c;
                if (out) {
                    if (Li == 0) {
                        out[o] = 0.0;
                    } else {
                        const double scale = (double)sA[i] * (double)sB[j] * (double)(QMAX * QMAX);
                        if (polarity == 0)
                            out[o] = scale * (2.0 * (double)c / (double)Li - (double)K);
                        else
                            out[o] = scale * (double)c / (double)Li;
                    }
                }
            }
        }
        free(zAp); free(zAn);
    }
    free(rA); free(rB); free(zBp); free(zBn);
    return err;
}

/* Number of OpenMP threads a parallel region would use now. */
int32_t oracle_max_threads(void) { return (int32_t)omp_get_max_threads(); }

/* ------------------------------------------------------------------------- */
/* Sobol-8 and conditional bitstream generation (C-BSG)                       */
/* ------------------------------------------------------------------------- */

/* 8-bit direction numbers of Sobol dimension `dim` (1 or 2), V[j-1] for j = 1..8. */
static int sobol8_directions(int dim, uint32_t V[8])
{
    uint32_t m[9];
    if (dim == 1) {
        for (int j = 1; j <= 8; ++j) m[j] = 1;
    } else if (dim == 2) {
        /* primitive polynomial x + 1 (degree 1): m_j = 2 m_{j-1} xor m_{j-1} */
        m[1] = 1;
        for (int j = 2; j <= 8; ++j) m[j] = (2 * m[j - 1]) ^ m[j - 1];
    } else {
        return -1;
    }
    for (int j = 1; j <= 8; ++j) V[j - 1] = m[j] << (8 - j);
    return 0;
}

/* The digital shift of operand `op` for `seed`. */
uint32_t oracle_sobol_shift(uint64_t seed, uint32_t op)
{
    return (uint32_t)(oracle_splitmix64(2ull * seed + (uint64_t)op) >> 56);
}

/* r_k = shift xor (xor of V_j over the set bits of k), k = 0..n-1, n <= 256. */
int oracle_sobol8(int dim, uint32_t shift, int32_t n, uint8_t *out)
{
    uint32_t V[8];
    if (sobol8_directions(dim, V) != 0 || n < 0 || n > 256) return -1;
    for (int32_t k = 0; k < n; ++k) {
        uint32_t x = 0;
        for (int j = 0; j < 8; ++j)
            if ((k >> j) & 1) x ^= V[j];
        out[k] = (uint8_t)((x ^ shift) & 255u);
    }
    return 0;
}

/*
 * SC GEMM with C-BSG streams (same shapes, scales and decode as oracle_sc_gemm).
 * For every pair (i, j) and element d the three streams are materialised cycle by
 * cycle: zA_l = [rA_l < betaA] for l < L_i; B's draw at cycle l is r^B at counter k1
 * if zA_l = 1 (then k1 advances) or at counter k0 if zA_l = 0 (then k0 advances);
 * zB_l = [that draw < betaB].  Bipolar counts XNOR(zA, zB); unipolar counts the
 * AND of the magnitude streams with the pair's sign.  L_max <= 256.
 */
int oracle_sc_gemm_cbsg(int32_t M, int32_t N, int32_t K,
                        const int8_t *A, const int8_t *B,
                        const float *sA, const float *sB,
                        const int32_t *L, int32_t L_max,
                        int32_t polarity, uint64_t seed,
                        int32_t *counts, double *out, int32_t nthreads)
{
    if (M < 0 || N < 0 || K < 0 || L_max < 0 || L_max > 256 || (polarity != 0 && polarity != 1))
        return -1;
    for (int32_t i = 0; i < M; ++i)
        if (L[i] < 0 || L[i] > L_max) return -1;
    if (M == 0 || N == 0) return 0;
    uint8_t rA[256], rB[256];
    oracle_sobol8(1, oracle_sobol_shift(seed, 0), 256, rA);
    oracle_sobol8(2, oracle_sobol_shift(seed, 1), 256, rB);
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 1)
    for (int32_t i = 0; i < M; ++i) {
        const int32_t Li = L[i];
        uint8_t za[256], zb[256];
        for (int32_t j = 0; j < N; ++j) {
            int64_t c = 0;
            for (int32_t d = 0; d < K; ++d) {
                const int32_t qa = A[(size_t)i * K + d], qb = B[(size_t)j * K + d];
                const int32_t ba = polarity == 0 ? oracle_beta_bipolar(qa) : oracle_beta_unipolar(qa);
                const int32_t bb = polarity == 0 ? oracle_beta_bipolar(qb) : oracle_beta_unipolar(qb);
                sng(rA, ba, Li, za);
                int32_t k1 = 0, k0 = 0;
                for (int32_t l = 0; l < Li; ++l) {
                    const int32_t draw = za[l] ? rB[k1++] : rB[k0++];
                    zb[l] = (uint8_t)(draw < bb ? 1 : 0);
                }
                int32_t s = 0;
                if (polarity == 0) {
                    for (int32_t l = 0; l < Li; ++l) s += 1 - (za[l] ^ zb[l]);
                } else {
                    for (int32_t l = 0; l < Li; ++l) s += za[l] & zb[l];
                    if ((qa < 0) != (qb < 0)) s = -s;
                }
                c += s;
            }
            const size_t o = (size_t)i * N + j;
            if (counts) counts[o] = (int32_t)c;
            if (out) {
                if (Li == 0) {
                    out[o] = 0.0;
                } else {
                    const double scale = (double)sA[i] * (double)sB[j] * (double)(QMAX * QMAX);
                    out[o] = polarity == 0 ? scale * (2.0 * (double)c / (double)Li - (double)K)
                                           : scale * (double)c / (double)Li;
                }
            }
        }
    }
    return 0;
}
