// Front end of the SC GEMM on the device: fp32 -> int8 symmetric quantisation with the
// row scale and row metric in one pass (Sec. 3.1 PTQ inputs, Sec. 4.2 fused
// quantisation), and the per-row length policy (Sec. 4.4: min-max normalised row
// metric, calibrated thresholds, a ladder of stream lengths).
#include <math.h>

#include "sc_internal.h"

namespace scg {

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}
__device__ __forceinline__ float wave_min(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fminf(v, __shfl_xor(v, o, 64));
    return v;
}

// max over a 256-thread block (every thread gets the result)
__device__ float block_max_256(float v) {
    __shared__ float part[4];
    v = wave_max(v);
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = v;
    __syncthreads();
    const float r = fmaxf(fmaxf(part[0], part[1]), fmaxf(part[2], part[3]));
    __syncthreads();
    return r;
}

// round half to even, clamp to [-127, 127]; s == 0 gives 0
__device__ __forceinline__ int8_t quant1(float x, float s) {
    if (!(s > 0.0f)) return 0;
    const float q = fminf(fmaxf(rintf(x / s), -127.0f), 127.0f);
    return (int8_t)(int)q;
}

// per row: m = max |x|, scale = m/127, quantise (one 256-thread block per row)
__global__ __launch_bounds__(256) void k_quant_rows(int rows, int K, const float *__restrict__ X,
                                                    int64_t ldx, int64_t strideX,
                                                    int8_t *__restrict__ Q, int64_t ldq,
                                                    int64_t strideQ, float *scale, float *rowmax,
                                                    int64_t strideS) {
    const int i = blockIdx.x, b = blockIdx.y;
    const float *x = X + (size_t)b * strideX + (size_t)i * ldx;
    int8_t *q = Q + (size_t)b * strideQ + (size_t)i * ldq;
    float m = 0.0f;
    for (int d = threadIdx.x; d < K; d += 256) m = fmaxf(m, fabsf(x[d]));
    m = block_max_256(m);
    const float s = m / 127.0f;
    if (threadIdx.x == 0) {
        scale[(size_t)b * strideS + i] = s;
        if (rowmax) rowmax[(size_t)b * strideS + i] = m;
    }
    for (int d = threadIdx.x; d < K; d += 256) q[d] = quant1(x[d], s);
}

// per tensor, pass 1: row maxima into `dst` (rowmax, or scale as scratch)
__global__ __launch_bounds__(256) void k_row_max(int K, const float *__restrict__ X, int64_t ldx,
                                                 int64_t strideX, float *dst, int64_t strideS) {
    const int i = blockIdx.x, b = blockIdx.y;
    const float *x = X + (size_t)b * strideX + (size_t)i * ldx;
    float m = 0.0f;
    for (int d = threadIdx.x; d < K; d += 256) m = fmaxf(m, fabsf(x[d]));
    m = block_max_256(m);
    if (threadIdx.x == 0) dst[(size_t)b * strideS + i] = m;
}

// per tensor, pass 2: tensor maximum over the row maxima, scale broadcast to every row
__global__ __launch_bounds__(256) void k_tensor_scale(int rows, const float *src, float *scale,
                                                      int64_t strideS) {
    const int b = blockIdx.x;
    float m = 0.0f;
    for (int i = threadIdx.x; i < rows; i += 256) m = fmaxf(m, src[(size_t)b * strideS + i]);
    m = block_max_256(m);
    const float s = m / 127.0f;
    for (int i = threadIdx.x; i < rows; i += 256) scale[(size_t)b * strideS + i] = s;
}

// per tensor, pass 3: quantise with the broadcast scale
__global__ __launch_bounds__(256) void k_quant_with_scale(int K, const float *__restrict__ X,
                                                          int64_t ldx, int64_t strideX,
                                                          int8_t *__restrict__ Q, int64_t ldq,
                                                          int64_t strideQ, const float *scale,
                                                          int64_t strideS) {
    const int i = blockIdx.x, b = blockIdx.y;
    const float *x = X + (size_t)b * strideX + (size_t)i * ldx;
    int8_t *q = Q + (size_t)b * strideQ + (size_t)i * ldq;
    const float s = scale[(size_t)b * strideS + i];
    for (int d = threadIdx.x; d < K; d += 256) q[d] = quant1(x[d], s);
}

hipError_t launch_quantize(int batch, int rows, int K, const float *X, int64_t ldx, int64_t strideX,
                           int per_tensor, int8_t *Q, int64_t ldq, int64_t strideQ, float *scale,
                           float *rowmax, int64_t strideS, hipStream_t st) {
    const dim3 grid((unsigned)rows, (unsigned)batch);
    if (!per_tensor) {
        hipLaunchKernelGGL(k_quant_rows, grid, dim3(256), 0, st, rows, K, X, ldx, strideX, Q, ldq,
                           strideQ, scale, rowmax, strideS);
        return hipGetLastError();
    }
    float *tmp = rowmax ? rowmax : scale;
    hipLaunchKernelGGL(k_row_max, grid, dim3(256), 0, st, K, X, ldx, strideX, tmp, strideS);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_tensor_scale, dim3((unsigned)batch), dim3(256), 0, st, rows, tmp, scale,
                       strideS);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_quant_with_scale, grid, dim3(256), 0, st, K, X, ldx, strideX, Q, ldq,
                       strideQ, scale, strideS);
    return hipGetLastError();
}

// ----------------------------------------------------------------------------
// per-row lengths (one 1024-thread block per operator call)
// ----------------------------------------------------------------------------
__global__ __launch_bounds__(1024) void k_mp_lengths(int M, const float *__restrict__ metric,
                                                     int64_t strideM, MpParams p, int32_t *L_out,
                                                     int64_t strideL) {
    __shared__ float pmin[16], pmax[16];
    const int b = blockIdx.x, tid = threadIdx.x;
    const float *g = metric + (size_t)b * strideM;
    float lo = INFINITY, hi = -INFINITY;
    for (int i = tid; i < M; i += 1024) {
        lo = fminf(lo, g[i]);
        hi = fmaxf(hi, g[i]);
    }
    lo = wave_min(lo);
    hi = wave_max(hi);
    if ((tid & 63) == 0) {
        pmin[tid >> 6] = lo;
        pmax[tid >> 6] = hi;
    }
    __syncthreads();
    lo = pmin[0];
    hi = pmax[0];
    for (int w = 1; w < 16; ++w) {
        lo = fminf(lo, pmin[w]);
        hi = fmaxf(hi, pmax[w]);
    }
    const float range = hi - lo;
    for (int i = tid; i < M; i += 1024) {
        const float t = range > 0.0f ? (g[i] - lo) / range : 0.0f;
        int k = p.n - 1;
        for (int j = 0; j < p.n - 1; ++j) {
            if (t >= p.tau[j]) {
                k = j;
                break;
            }
        }
        L_out[(size_t)b * strideL + i] = p.ladder[k];
    }
}

hipError_t launch_mp_lengths(int batch, int M, const float *metric, int64_t strideM,
                             const MpParams &p, int32_t *L_out, int64_t strideL, hipStream_t st) {
    hipLaunchKernelGGL(k_mp_lengths, dim3((unsigned)batch), dim3(1024), 0, st, M, metric, strideM, p,
                       L_out, strideL);
    return hipGetLastError();
}

}  // namespace scg
