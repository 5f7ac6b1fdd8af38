// Drives the host side of libscgemm -- descriptor checks, workspace layout, split choice,
// argument errors of every entry point -- over many random descriptors, so that a build with
// the host code instrumented by AddressSanitizer and UndefinedBehaviorSanitizer checks it.
// Every call returns before anything is enqueued (no GPU is used).  Test infrastructure.
#include <stdint.h>
#include <stdio.h>

#include "scgemm.h"

static uint64_t st = 99;
static uint32_t rnd() { st = st * 6364136223846793005ull + 1442695040888963407ull; return (uint32_t)(st >> 33); }
static int32_t pick(const int32_t *v, int n) { return v[rnd() % (uint32_t)n]; }

#define CHECK(c) do { if (!(c)) { printf("check failed: %s (line %d)\n", #c, __LINE__); return 1; } } while (0)

int main() {
    const int32_t Ms[] = {0, 1, 3, 64, 127, 128, 129, 255, 256, 257, 300, 577, 4096, 6304, 8224, 18464, 100000};
    const int32_t Ns[] = {0, 1, 17, 64, 65, 128, 129, 256, 577, 3072, 4608};
    const int32_t Ks[] = {0, 1, 5, 31, 32, 33, 64, 577, 768, 1024, 4128, 65600, 1 << 20, (1 << 20) + 1};
    const int32_t Ls[] = {-1, 0, 1, 7, 8, 31, 32, 33, 64, 128, 256, 257, 512, 4096, 4097};
    const int32_t Bs[] = {0, 1, 2, 16, 128};
    void *fake = (void *)(uintptr_t)(1ull << 40);     // never dereferenced
    int ok = 0, refused = 0;
    for (int it = 0; it < 20000; ++it) {
        sc_gemm_desc d = {};
        d.batch = pick(Bs, 5);
        d.M = pick(Ms, 17);
        d.N = pick(Ns, 11);
        d.K = pick(Ks, 14);
        d.lda = d.K + (int64_t)(rnd() % 3) * 16 - (rnd() % 17 == 0);
        d.ldb = d.K + (int64_t)(rnd() % 3);
        d.ldo = d.N + (int64_t)(rnd() % 2) * 4;
        d.strideA = (int64_t)d.M * d.lda * (rnd() % 2);
        d.strideB = (int64_t)d.N * d.ldb * (rnd() % 2);
        d.strideO = (int64_t)d.M * d.ldo;
        d.strideSA = d.M;
        d.strideSB = d.N * (rnd() % 2);
        d.strideL = d.M;
        d.L_max = pick(Ls, 15);
        d.polarity = (int32_t)(rnd() % 3) - (rnd() % 50 == 0);
        d.rng = (int32_t)(rnd() % 2) + (rnd() % 40 == 0);
        d.L_hint = d.L_max > 0 ? (int32_t)(rnd() % (uint32_t)(d.L_max + 1)) : 0;
        d.reserved = rnd() % 100 == 0;
        d.seed = ((uint64_t)rnd() << 32) | rnd();
        size_t n = 0;
        const int rc = sc_gemm_workspace_size(&d, &n);
        if (rc == SC_OK) {
            ++ok;
            CHECK(n % 256 == 0 && n > 0);
            // too small a workspace, and missing operands, are refused before any launch
            CHECK(sc_gemm(&d, (const int8_t *)fake, (const float *)fake, (const int8_t *)fake, (const float *)fake,
                          (const int32_t *)fake, (float *)fake, nullptr, fake, n - 1, nullptr) == SC_ERR_WORKSPACE);
            if (d.batch > 0 && d.M > 0 && d.N > 0)
                CHECK(sc_gemm(&d, (const int8_t *)fake, (const float *)fake, (const int8_t *)fake,
                              (const float *)fake, (const int32_t *)fake, nullptr, nullptr, fake, n, nullptr) ==
                      SC_ERR_NULL);
            if (n > SC_NOALLOC_WORKSPACE_BYTES)
                CHECK(sc_gemm_noalloc(&d, (const int8_t *)fake, (const float *)fake, (const int8_t *)fake,
                                      (const float *)fake, (const int32_t *)fake, (float *)fake, nullptr, nullptr,
                                      nullptr) == SC_ERR_WORKSPACE);
        } else {
            ++refused;
            CHECK(rc < 0 && rc >= -10);
            CHECK(sc_gemm(&d, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, 0, nullptr) ==
                  rc);
            CHECK(sc_strerror(rc)[0] == 'S');
        }
    }
    CHECK(ok > 1000 && refused > 1000);
    // the other entry points' argument checks
    CHECK(sc_comparator_sequence(0, 2, 0, 16, (uint8_t *)fake, nullptr) == SC_ERR_RNG);
    CHECK(sc_comparator_sequence(0, 0, 0, 4097, (uint8_t *)fake, nullptr) == SC_ERR_LEN);
    CHECK(sc_quantize(1, 4, -1, nullptr, 0, 0, 0, nullptr, 0, 0, nullptr, nullptr, 0, nullptr) == SC_ERR_SHAPE);
    CHECK(sc_quantize(1, 4, 8, nullptr, 4, 0, 0, nullptr, 8, 0, nullptr, nullptr, 0, nullptr) == SC_ERR_STRIDE);
    CHECK(sc_quantize(1, 4, 8, nullptr, 8, 0, 0, nullptr, 8, 0, nullptr, nullptr, 0, nullptr) == SC_ERR_NULL);
    const float tau[3] = {0.9f, 0.5f, 0.1f}, bad_tau[3] = {0.1f, 0.5f, 0.9f};
    const int32_t lad[4] = {256, 128, 64, 32}, bad_lad[4] = {32, 64, 128, 256};
    CHECK(sc_mp_lengths(1, 10, nullptr, 10, tau, lad, 33, nullptr, 10, nullptr) == SC_ERR_LEN);
    CHECK(sc_mp_lengths(1, 10, nullptr, 10, bad_tau, lad, 4, nullptr, 10, nullptr) == SC_ERR_LEN);
    CHECK(sc_mp_lengths(1, 10, nullptr, 10, tau, bad_lad, 4, nullptr, 10, nullptr) == SC_ERR_LEN);
    CHECK(sc_mp_lengths(1, 10, nullptr, 10, tau, lad, 4, nullptr, 10, nullptr) == SC_ERR_NULL);
    CHECK(sc_gemm_status(nullptr, nullptr) == SC_ERR_NULL);
    CHECK(sc_version() > 0);
    printf("host driver ok: %d descriptors laid out, %d refused\n", ok, refused);
    return 0;
}
