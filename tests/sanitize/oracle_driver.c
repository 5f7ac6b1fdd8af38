/* Drives every function of the CPU oracle (oracle/sc_oracle.c) on small random problems,
 * including the edge cases (zero lengths, K = 0, M = 0, L_max = 0, saturated operands,
 * bad arguments), so that a build with AddressSanitizer and UndefinedBehaviorSanitizer
 * checks its memory accesses and arithmetic.  Test infrastructure only. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

uint64_t oracle_splitmix64(uint64_t x);
uint32_t oracle_seed_state(uint64_t seed, uint32_t op);
void oracle_lfsr_draws(uint32_t state, int32_t n, uint8_t *out);
void oracle_lfsr_states(uint32_t state, int32_t n, uint32_t *out);
int32_t oracle_beta_bipolar(int32_t q);
int32_t oracle_beta_unipolar(int32_t q);
void oracle_streams(int32_t rows, int32_t K, const int8_t *X, int32_t polarity, uint64_t seed, uint32_t op,
                    int32_t len, uint8_t *z);
int oracle_sc_gemm(int32_t M, int32_t N, int32_t K, const int8_t *A, const int8_t *B, const float *sA,
                   const float *sB, const int32_t *L, int32_t L_max, int32_t polarity, uint64_t seed,
                   int32_t *counts, double *out, int32_t nthreads);
uint32_t oracle_sobol_shift(uint64_t seed, uint32_t op);
int oracle_sobol8(int dim, uint32_t shift, int32_t n, uint8_t *out);
int oracle_sc_gemm_cbsg(int32_t M, int32_t N, int32_t K, const int8_t *A, const int8_t *B, const float *sA,
                        const float *sB, const int32_t *L, int32_t L_max, int32_t polarity, uint64_t seed,
                        int32_t *counts, double *out, int32_t nthreads);
int32_t oracle_max_threads(void);

static uint64_t st = 12345;
static uint32_t rnd(void) { st = st * 6364136223846793005ull + 1442695040888963407ull; return (uint32_t)(st >> 33); }

#define CHECK(c) do { if (!(c)) { printf("check failed: %s (line %d)\n", #c, __LINE__); return 1; } } while (0)

static int one_case(int M, int N, int K, int L_max, int polarity, int cbsg, uint64_t seed, int nthreads) {
    int8_t *A = malloc((size_t)(M * K + 1)), *B = malloc((size_t)(N * K + 1));
    float *sA = malloc(sizeof(float) * (size_t)(M + 1)), *sB = malloc(sizeof(float) * (size_t)(N + 1));
    int32_t *L = malloc(sizeof(int32_t) * (size_t)(M + 1)), *c = malloc(sizeof(int32_t) * (size_t)(M * N + 1));
    double *o = malloc(sizeof(double) * (size_t)(M * N + 1));
    for (int i = 0; i < M * K; ++i) A[i] = (int8_t)((int)(rnd() % 255) - 127);
    for (int i = 0; i < N * K; ++i) B[i] = (int8_t)((int)(rnd() % 255) - 127);
    if (M * K > 0) A[0] = 127;
    if (N * K > 0) B[0] = -127;
    for (int i = 0; i < M; ++i) { sA[i] = 0.01f * (float)(1 + rnd() % 50); L[i] = L_max > 0 ? (int32_t)(rnd() % (uint32_t)(L_max + 1)) : 0; }
    for (int j = 0; j < N; ++j) sB[j] = 0.01f * (float)(1 + rnd() % 50);
    if (M > 1) { L[0] = L_max; L[1] = 0; }
    int rc = cbsg ? oracle_sc_gemm_cbsg(M, N, K, A, B, sA, sB, L, L_max, polarity, seed, c, o, nthreads)
                  : oracle_sc_gemm(M, N, K, A, B, sA, sB, L, L_max, polarity, seed, c, o, nthreads);
    int bad = rc != 0;
    for (int i = 0; i < M && !bad; ++i)
        for (int j = 0; j < N; ++j) {
            const int32_t x = c[i * N + j];
            const int64_t KL = (int64_t)K * L[i];
            if (polarity == 0 ? (x < 0 || x > KL) : (x < -KL || x > KL)) bad = 1;
            if (L[i] == 0 && (x != 0 || o[i * N + j] != 0.0)) bad = 1;
        }
    free(A); free(B); free(sA); free(sB); free(L); free(c); free(o);
    return bad;
}

int main(void) {
    uint8_t r[4096];
    uint32_t s[64];
    CHECK(oracle_splitmix64(0) != 0);
    for (uint64_t seed = 0; seed < 4; ++seed)
        for (uint32_t op = 0; op < 2; ++op) {
            oracle_lfsr_draws(oracle_seed_state(seed, op), 4096, r);
            oracle_lfsr_states(oracle_seed_state(seed, op), 64, s);
            CHECK(oracle_sobol8(1 + (int)op, oracle_sobol_shift(seed, op), 256, r) == 0);
        }
    CHECK(oracle_sobol8(3, 0, 10, r) != 0 && oracle_sobol8(1, 0, 257, r) != 0);
    for (int q = -128; q <= 127; ++q) {
        const int32_t b = oracle_beta_bipolar(q), u = oracle_beta_unipolar(q);
        CHECK(b >= 0 && b <= 256 && u >= 0 && u <= 258);
    }
    {
        int8_t X[3 * 5];
        uint8_t z[3 * 5 * 70];
        for (int i = 0; i < 15; ++i) X[i] = (int8_t)((int)(rnd() % 255) - 127);
        oracle_streams(3, 5, X, 0, 9, 0, 70, z);
        oracle_streams(3, 5, X, 1, 9, 1, 70, z);
    }
    /* shapes: tiny, ragged, zero-sized, long streams; both polarities and sources */
    const int shapes[][4] = {{1, 1, 1, 1}, {7, 5, 33, 70}, {3, 9, 0, 16}, {0, 4, 8, 8}, {4, 0, 8, 8},
                             {5, 6, 40, 300}, {2, 3, 17, 0}, {9, 4, 65, 256}};
    for (unsigned k = 0; k < sizeof(shapes) / sizeof(shapes[0]); ++k)
        for (int pol = 0; pol < 2; ++pol)
            for (int cbsg = 0; cbsg < 2; ++cbsg) {
                const int Lm = shapes[k][3];
                if (cbsg && Lm > 256) continue;
                CHECK(one_case(shapes[k][0], shapes[k][1], shapes[k][2], Lm, pol, cbsg, 3 + k, k % 3 + 1) == 0);
            }
    /* bad arguments are refused */
    {
        int8_t a = 1, b = 1;
        float sa = 1.0f, sb = 1.0f;
        int32_t L = 5, cnt = 0;
        double out = 0.0;
        CHECK(oracle_sc_gemm(1, 1, 1, &a, &b, &sa, &sb, &L, 4, 0, 0, &cnt, &out, 1) != 0);
        CHECK(oracle_sc_gemm(1, 1, 1, &a, &b, &sa, &sb, &L, 8, 2, 0, &cnt, &out, 1) != 0);
        CHECK(oracle_sc_gemm_cbsg(1, 1, 1, &a, &b, &sa, &sb, &L, 300, 0, 0, &cnt, &out, 1) != 0);
        CHECK(oracle_sc_gemm(-1, 1, 1, &a, &b, &sa, &sb, &L, 8, 0, 0, &cnt, &out, 1) != 0);
    }
    CHECK(oracle_max_threads() >= 1);
    printf("oracle driver ok\n");
    return 0;
}
