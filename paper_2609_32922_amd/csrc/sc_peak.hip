// libscpeak: measured VALU rate of the packed bit-op + popcount stream (see include/scpeak.h).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/scpeak.h"

namespace {

constexpr int CHAINS = 16;      // independent AND -> popcount chains per lane
constexpr int THREADS = 256;    // four waves per block, one per SIMD

// Each lane: CHAINS words a[k], b[k] and running counts; per trip one AND and one
// accumulating popcount per chain.  The instructions are written out so that exactly
// these two VALU instructions per 32 bit pairs are issued (the compiler would otherwise
// hoist the loop-invariant AND).  Lane 0 of each wave records the cycle-counter and
// wall-clock spans of its loop.
__global__ __launch_bounds__(THREADS) void k_and_bcnt(uint32_t seed, int iters, uint32_t *sink,
                                                      uint64_t *spans) {
    const uint32_t t = blockIdx.x * THREADS + threadIdx.x;
    uint32_t a[CHAINS], b[CHAINS], acc[CHAINS];
#pragma unroll
    for (int k = 0; k < CHAINS; ++k) {
        a[k] = seed * (t + 1u) + 0x9E3779B9u * (uint32_t)k;
        b[k] = ~a[k] ^ (t << (k & 7));
        acc[k] = 0u;
        asm volatile("" : "+v"(a[k]), "+v"(b[k]));    // opaque: no recomputation inside the loop
    }
    const uint64_t c0 = clock64(), w0 = wall_clock64();
    for (int it = 0; it < iters; ++it) {
        // all ANDs of a trip, then all counts, so that no count waits on the AND before it
        uint32_t x[CHAINS];
#pragma unroll
        for (int k = 0; k < CHAINS; ++k) asm volatile("v_and_b32 %0, %1, %2" : "=v"(x[k]) : "v"(a[k]), "v"(b[k]));
#pragma unroll
        for (int k = 0; k < CHAINS; ++k) asm volatile("v_bcnt_u32_b32 %0, %1, %0" : "+v"(acc[k]) : "v"(x[k]));
    }
    const uint64_t c1 = clock64(), w1 = wall_clock64();
    uint32_t s = 0u;
#pragma unroll
    for (int k = 0; k < CHAINS; ++k) s += acc[k];
    sink[t] = s;
    if ((threadIdx.x & 63) == 0) {
        spans[2 * (t >> 6)] = c1 - c0;
        spans[2 * (t >> 6) + 1] = w1 - w0;
    }
}

}  // namespace

extern "C" int sc_peak_valu_bitop(int32_t waves_per_simd, int32_t iters, sc_peak_result *res) {
    if (res == nullptr || waves_per_simd < 1 || waves_per_simd > 8 || iters < 1) return -1;
    int dev = 0, cus = 0, wall_khz = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipDeviceGetAttribute(&wall_khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess || cus <= 0 ||
        wall_khz <= 0)
        return -7;
    const unsigned blocks = (unsigned)(cus * waves_per_simd);
    const size_t threads = (size_t)blocks * THREADS, waves = threads / 64;
    uint32_t *sink = nullptr;
    uint64_t *spans = nullptr;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    int rc = -7;
    float ms = 0.0f;
    uint64_t *h = nullptr;
    if (hipMalloc(&sink, threads * 4) != hipSuccess || hipMalloc(&spans, waves * 16) != hipSuccess ||
        hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess)
        goto done;
    // one untimed launch brings the clock up and the code in
    hipLaunchKernelGGL(k_and_bcnt, dim3(blocks), dim3(THREADS), 0, 0, 12345u, iters / 4 + 1, sink, spans);
    if (hipGetLastError() != hipSuccess) goto done;
    if (hipEventRecord(e0, 0) != hipSuccess) goto done;
    hipLaunchKernelGGL(k_and_bcnt, dim3(blocks), dim3(THREADS), 0, 0, 777u, iters, sink, spans);
    if (hipGetLastError() != hipSuccess || hipEventRecord(e1, 0) != hipSuccess ||
        hipEventSynchronize(e1) != hipSuccess || hipEventElapsedTime(&ms, e0, e1) != hipSuccess)
        goto done;
    h = new uint64_t[2 * waves];
    if (hipMemcpy(h, spans, waves * 16, hipMemcpyDeviceToHost) != hipSuccess) goto done;
    {
        double clk = 0.0;
        size_t n = 0;
        for (size_t w = 0; w < waves; ++w) {
            if (h[2 * w + 1] == 0) continue;
            clk += (double)h[2 * w] / ((double)h[2 * w + 1] / (wall_khz * 1e3));
            ++n;
        }
        const double lane_ops = (double)threads * iters * CHAINS * 2.0;
        res->seconds = ms * 1e-3;
        res->lane_ops_per_s = lane_ops / res->seconds;
        res->bitops_per_s = res->lane_ops_per_s * 32.0 / 2.0;
        res->clock_hz = n ? clk / n : 0.0;
        res->cus = cus;
        res->waves_per_simd = waves_per_simd;
        rc = 0;
    }
done:
    delete[] h;
    if (e0) (void)hipEventDestroy(e0);
    if (e1) (void)hipEventDestroy(e1);
    if (sink) (void)hipFree(sink);
    if (spans) (void)hipFree(spans);
    return rc;
}
