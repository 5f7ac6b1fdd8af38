// MFMA engine of libscgemm for gfx950: the SC counts as a dense contraction on the
// matrix cores.
//
// The count of one output (Sec. 3.1, Eq. (1)) sums bit products over every pair (d, l)
// of element and cycle, so it is the product of two matrices whose columns are the
// (d, l) pairs.  Each stream bit becomes an fp4 (e2m1) value in {-1, 0, +1}:
//   bipolar   +1 / -1 for z = 1 / 0 at cycles l < L, 0 beyond: the sum P of the
//             products is 2 X - K L, so X = (K L + P) / 2 (no marginals needed)
//   unipolar  sign(q) * z: P is the signed count S = c_pp + c_nn - c_pn - c_np
//   C-BSG     A holds sgn * D_k (bipolar) or sign(q) * [k < c] (unipolar) over B's draw
//             counter k, B holds its comparator stream on r^B as above; bipolar then
//             gives X = (K L + P) / 2 and unipolar S = P (Sec. 4.2, Eq. (6))
// v_mfma_scale_f32_16x16x128_f8f6f4 with unit scales sums 128 such products into fp32;
// every partial sum is an integer of magnitude <= K L <= 2^24, so the count is exact
// and independent of the summation order.
//
//   k_mplanes     nibble planes of A (sorted rows, per-row lengths) or B, one block per
//                 128-row tile x 32 cycles x 64 elements; element parameters and an
//                 8-cycle lookup table in LDS, 1 KB coalesced stores
//   k_mgemm       128x128 output tile per 256-thread block, 64x64 per wave as 4x4
//                 16x16 MFMA blocks, 16 slots (4 MFMA k-steps) per LDS stage
//   k_mgemm_reduce sums the partial counts of split tiles and decodes
#include "sc_internal.h"

namespace scg {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));   // one slot row: 32 nibbles

constexpr uint32_t NIB_POS = 0x2u;   // e2m1 +1.0
constexpr uint32_t NIB_NEG = 0xAu;   // e2m1 -1.0
constexpr int PRM_STRIDE = 145;      // LDS row stride (in words) of the element parameters:
                                     // 145 = 17 mod 64 keeps both access patterns spread
                                     // over the banks

// +1 -> -1 for every nonzero nibble: 0x2 | (0x2 << 2) = 0xA
__device__ __forceinline__ uint32_t negate_nibbles(uint32_t v) { return v | ((v << 2) & 0x88888888u); }

// ----------------------------------------------------------------------------
// nibble planes
// ----------------------------------------------------------------------------
struct MPlaneArgs {
    const int8_t *X;
    int64_t ld, strideX;
    int rows, K, KQP;
    int nchunk;                 // octet chunks of OCH per tile in the grid
    int uniformL;               // B side: L_max for every row
    int LBS;                    // B side: cycles of the planes (multiple of 32)
    int per_row;                // 1: A side (sorted rows, per-row lengths)
    size_t stride_batch;
    size_t off_perm, off_Ls, off_tileL, off_tileOff;
    size_t off_planes, off_r, off_CA;
};

// Comparator mode (CBSG = false): nibble of element d at cycle l is +1 for r_l < beta_d,
// else -1 (bipolar) or 0 (unipolar, then times sign(q)); 0 at cycles >= L_row and for
// padding.  Interval mode (CBSG = true, A side): nibble at counter k is sgn for
// lo_d <= k < hi_d, else 0 (see the header comment).
template <int POL, bool CBSG>
__global__ __launch_bounds__(256) void k_mplanes(MPlaneArgs a, uint8_t *ws) {
    __shared__ uint32_t prm[64 * PRM_STRIDE];    // [element][row] packed parameters
    __shared__ uint32_t lut[OCH * CA_COLS];      // comparator: 8 nibbles per octet and beta
    __shared__ uint32_t spread[256];             // interval: 8-bit mask -> 8 nibbles of +1
    const int t = blockIdx.x / a.nchunk, ch = blockIdx.x % a.nchunk;
    const int qg = blockIdx.y, b = blockIdx.z;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    uint8_t *wsb = ws + (size_t)b * a.stride_batch;

    int Lloop;
    int64_t off;
    const int32_t *perm = nullptr, *Ls = nullptr;
    if (a.per_row) {
        Lloop = ws_ptr<int32_t>(wsb, a.off_tileL)[t];
        off = ws_ptr<int64_t>(wsb, a.off_tileOff)[t];
        perm = ws_ptr<int32_t>(wsb, a.off_perm);
        Ls = ws_ptr<int32_t>(wsb, a.off_Ls);
    } else {
        Lloop = a.LBS;
        off = (int64_t)t * a.LBS * a.KQP * 64;
    }
    const int o0 = ch * OCH;
    if (o0 * MSTEP >= Lloop) return;
    const int no = min(OCH, Lloop / MSTEP - o0);
    const int8_t *Xb = a.X + (size_t)b * a.strideX;
    const uint16_t *CA = CBSG ? ws_ptr<uint16_t>(ws, a.off_CA) : nullptr;

    // 1. element parameters: one wave reads the 64 bytes of one row at a time
    const int d = qg * 64 + lane;
    for (int m = w; m < BM; m += 4) {
        const int p = t * BM + m;
        int row, Lr;
        if (a.per_row) {
            row = perm[p];
            Lr = row >= 0 ? Ls[p] : 0;
        } else {
            row = p < a.rows ? p : -1;
            Lr = a.uniformL;
        }
        const bool valid = row >= 0 && d < a.K;
        const int q = valid ? (int)Xb[(size_t)row * a.ld + d] : 0;
        const int beta = POL == SC_BIPOLAR_XNOR ? beta_bipolar(q) : beta_unipolar(q);
        uint32_t pk;
        if (CBSG) {
            const int c = valid ? (int)CA[(size_t)Lr * CA_COLS + beta] : 0;
            int lo = 0, hi = c;
            bool neg = valid && q < 0;
            if (POL == SC_BIPOLAR_XNOR) {
                const int e = Lr - c;
                lo = min(c, e);
                hi = max(c, e);
                neg = c < e;
            }
            if (!valid) lo = hi = 0;
            pk = (uint32_t)lo | ((uint32_t)hi << 9) | (neg ? 0x80000000u : 0u);
        } else {
            const bool neg = POL == SC_UNIPOLAR_AND_SM && valid && q < 0;
            const int Le = valid ? Lr : 0;
            pk = (uint32_t)beta | ((uint32_t)Le << 9) | (neg ? 0x80000000u : 0u);
        }
        prm[lane * PRM_STRIDE + m] = pk;
    }
    // 2. lookup tables
    if (CBSG) {
        const uint32_t v = (uint32_t)tid;
        uint32_t x = 0;
#pragma unroll
        for (int c = 0; c < 8; ++c) x |= ((v >> c) & 1u) ? (NIB_POS << (4 * c)) : 0u;
        spread[tid] = x;
    } else {
        const uint32_t *r = ws_ptr<uint32_t>(ws, a.off_r) + (size_t)o0 * MSTEP;
        const uint32_t zero_nib = POL == SC_BIPOLAR_XNOR ? NIB_NEG : 0u;
        for (int e = tid; e < no * CA_COLS; e += 256) {
            const int o = e / CA_COLS, beta = e % CA_COLS;
            uint32_t x = 0;
#pragma unroll
            for (int c = 0; c < 8; ++c)
                x |= (r[o * MSTEP + c] < (uint32_t)beta ? NIB_POS : zero_nib) << (4 * c);
            lut[e] = x;
        }
    }
    __syncthreads();

    // 3. planes: per slot, thread tid writes row tid/4 dword tid%4, then rows 64..127
    uint32_t *planes = ws_ptr<uint32_t>(wsb, a.off_planes) + off;
    for (int o = 0; o < no; ++o) {
        const int oa = o0 + o, c0 = oa * MSTEP;
        for (int dq = 0; dq < 16; ++dq) {
            const int qd = qg * 16 + dq;
            if (qd >= a.KQP) break;
            uint32_t *dst = planes + ((size_t)oa * a.KQP + qd) * BM * 4;
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int idx = tid + 256 * h;
                const int m = idx >> 2, e = idx & 3;
                const uint32_t pk = prm[(4 * dq + e) * PRM_STRIDE + m];
                uint32_t v;
                if (CBSG) {
                    const int lo = (int)(pk & 511u), hi = (int)((pk >> 9) & 511u);
                    const int a0 = min(max(lo - c0, 0), 8), a1 = min(max(hi - c0, 0), 8);
                    const uint32_t bits = ((1u << a1) - 1u) & ~((1u << a0) - 1u);
                    v = spread[bits];
                } else {
                    const int beta = (int)(pk & 511u), Le = (int)((pk >> 9) & 8191u);
                    const int rem = Le - c0;
                    v = lut[o * CA_COLS + beta];
                    if (rem <= 0) v = 0u;
                    else if (rem < 8) v &= (1u << (4 * rem)) - 1u;
                }
                if (pk >> 31) v = negate_nibbles(v);
                dst[idx] = v;
            }
        }
    }
}

template <bool CBSG>
static void launch_mplanes_side(int polarity, dim3 grid, const MPlaneArgs &pa, uint8_t *ws,
                                hipStream_t st) {
    if (polarity == SC_BIPOLAR_XNOR)
        hipLaunchKernelGGL((k_mplanes<SC_BIPOLAR_XNOR, CBSG>), grid, dim3(256), 0, st, pa, ws);
    else
        hipLaunchKernelGGL((k_mplanes<SC_UNIPOLAR_AND_SM, CBSG>), grid, dim3(256), 0, st, pa, ws);
}

hipError_t launch_mplanes(const sc_gemm_desc &d, const Layout &lay, const int8_t *A,
                          const int8_t *B, uint8_t *ws, hipStream_t st) {
    if (lay.KQP == 0) return hipSuccess;
    const unsigned qgroups = (unsigned)((lay.KQP + 15) / 16);
    const bool cbsg = d.rng == SC_RNG_SOBOL8_CBSG;
    MPlaneArgs pa{};
    pa.X = A;
    pa.ld = d.lda;
    pa.strideX = d.strideA;
    pa.rows = d.M;
    pa.K = d.K;
    pa.KQP = lay.KQP;
    pa.nchunk = (int)((round_up(d.L_max, MSTEP) / MSTEP + OCH - 1) / OCH);
    pa.uniformL = 0;
    pa.LBS = lay.LBS;
    pa.per_row = 1;
    pa.stride_batch = lay.stride_batchA;
    pa.off_perm = lay.off_perm;
    pa.off_Ls = lay.off_Ls;
    pa.off_tileL = lay.off_tileL;
    pa.off_tileOff = lay.off_tileOff;
    pa.off_planes = lay.off_Ap;
    pa.off_r = lay.off_rA;
    pa.off_CA = lay.off_CA;
    const dim3 gA((unsigned)(lay.MT * pa.nchunk), qgroups, (unsigned)d.batch);
    if (cbsg)
        launch_mplanes_side<true>(d.polarity, gA, pa, ws, st);
    else
        launch_mplanes_side<false>(d.polarity, gA, pa, ws, st);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;

    MPlaneArgs pb = pa;
    pb.X = B;
    pb.ld = d.ldb;
    pb.strideX = d.strideB;
    pb.rows = d.N;
    pb.nchunk = lay.LBS / (OCH * MSTEP);
    pb.uniformL = d.L_max;
    pb.per_row = 0;
    pb.stride_batch = lay.stride_batchB;
    pb.off_perm = pb.off_Ls = pb.off_tileL = pb.off_tileOff = 0;
    pb.off_planes = lay.off_Bp;
    pb.off_r = lay.off_rB;
    pb.off_CA = 0;
    const dim3 gB((unsigned)(lay.NT * pb.nchunk), qgroups, (unsigned)lay.nbB);
    launch_mplanes_side<false>(d.polarity, gB, pb, ws, st);
    return hipGetLastError();
}

// ----------------------------------------------------------------------------
// MFMA GEMM
// ----------------------------------------------------------------------------
struct MGemmArgs {
    int M, N, K, KQP, LBS, nbB, batch, S;
    const float *sA, *sB;
    int64_t strideSA, strideSB, strideO, ldo;
    float *out;
    int32_t *counts;
};

// decode of four adjacent columns j0.. of sorted row position p from the fp4 product sums
template <bool BIP>
__device__ __forceinline__ void mdecode4(const int32_t (&P)[4], int p, int j0, int ncol, int b,
                                         const MGemmArgs &g, const Layout &lay, uint8_t *ws) {
    uint8_t *wsa = ws + (size_t)b * lay.stride_batchA;
    const int i = ws_ptr<int32_t>(wsa, lay.off_perm)[p];
    if (i < 0) return;
    const int Li = ws_ptr<int32_t>(wsa, lay.off_Ls)[p];
    const float scale = g.sA[(size_t)b * g.strideSA + i] * 16129.0f;
    const float *sBb = g.sB + (size_t)b * g.strideSB;
    const int KL = g.K * Li;
    float o[4];
    int32_t cnt[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const int j = c < ncol ? j0 + c : j0;
        // bipolar: P = 2X - K L; unipolar: P = S
        cnt[c] = BIP ? (KL + P[c]) / 2 : P[c];
        o[c] = Li > 0 ? (float)P[c] / (float)Li * (scale * sBb[j]) : 0.0f;
        if (Li == 0) cnt[c] = 0;
    }
    float *op = g.out + (size_t)b * g.strideO + (size_t)i * g.ldo + j0;
    if (ncol == 4 && (reinterpret_cast<uintptr_t>(op) & 15) == 0) {
        *reinterpret_cast<float4 *>(op) = make_float4(o[0], o[1], o[2], o[3]);
    } else {
        for (int c = 0; c < ncol; ++c) op[c] = o[c];
    }
    if (g.counts) {
        int32_t *cp = g.counts + (size_t)b * g.strideO + (size_t)i * g.ldo + j0;
        if (ncol == 4 && (reinterpret_cast<uintptr_t>(cp) & 15) == 0) {
            *reinterpret_cast<int4 *>(cp) = make_int4(cnt[0], cnt[1], cnt[2], cnt[3]);
        } else {
            for (int c = 0; c < ncol; ++c) cp[c] = cnt[c];
        }
    }
}

__device__ __forceinline__ v8i frag(u4 x) {
    v8i r = {(int)x.x, (int)x.y, (int)x.z, (int)x.w, 0, 0, 0, 0};
    return r;
}

constexpr int PER_T = MSTAGE * BM / 256;   // uint4 of A (and of B) per thread per stage

// Loads the stage of slots [ks, ks + MSTAGE) into registers.  A short last stage re-reads
// its last slot row instead of running past the unit (the compute loop never reads
// those LDS entries), so every load is in bounds.
__device__ __forceinline__ void load_stage(const u4 *gA, const u4 *gB, int64_t ks, int64_t k1,
                                           int tid, u4 (&ra)[PER_T], u4 (&rb)[PER_T]) {
    const int last = (int)min((int64_t)MSTAGE, k1 - ks) * BM - 1;
    const u4 *pa = gA + ks * BM, *pb = gB + ks * BN;
#pragma unroll
    for (int k = 0; k < PER_T; ++k) {
        const int e = min(tid + 256 * k, last);
        ra[k] = pa[e];
        rb[k] = pb[e];
    }
}

// One block: the 128x128 tile (tm, tn) of batch entry b over a contiguous range of MFMA
// k-steps (4 slots each).  Wave w owns rows 64*(w/2).., columns 64*(w%2)..; lane l reads
// slot 4j + l/16 of row (or column) l%16 of each 16-row block, which is the operand
// layout of the 16x16x128 instruction (32 consecutive k per lane).  The accumulator
// element e of lane l is row 4*(l/16)+e, column l%16 of its 16x16 block.
template <bool BIP, bool SPLIT>
__global__ __launch_bounds__(256, 2) void k_mgemm(MGemmArgs g, Layout lay, uint8_t *ws) {
    __shared__ u4 smem[MSTAGE * (BM + BN)];
    u4 *As = smem, *Bs = smem + MSTAGE * BM;
    const int u = blockIdx.x;
    const int s = u % g.S;
    const int tile = u / g.S;
    const int tn = tile % lay.NT;
    const int tb = tile / lay.NT;
    const int b = tb % g.batch, tm = tb / g.batch;
    const int bB = g.nbB == 1 ? 0 : b;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int grp = lane >> 4, i16 = lane & 15;
    const int wr = (w >> 1) * 64, wc = (w & 1) * 64;
    uint8_t *wsa = ws + (size_t)b * lay.stride_batchA;
    uint8_t *wsbB = ws + (size_t)bB * lay.stride_batchB;
    const int Lloop = ws_ptr<int32_t>(wsa, lay.off_tileL)[tm];
    const int64_t nsteps = (int64_t)(Lloop / MSTEP) * g.KQP / 4;
    const int64_t k0 = (int64_t)s * nsteps / g.S * 4, k1 = (int64_t)(s + 1) * nsteps / g.S * 4;
    const u4 *gA = reinterpret_cast<const u4 *>(ws_ptr<uint32_t>(wsa, lay.off_Ap) +
                                                ws_ptr<int64_t>(wsa, lay.off_tileOff)[tm]);
    const u4 *gB = reinterpret_cast<const u4 *>(ws_ptr<uint32_t>(wsbB, lay.off_Bp)) +
                   (size_t)tn * (g.LBS / MSTEP) * g.KQP * BN;

    v4f acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[i][c] = v4f{0.0f, 0.0f, 0.0f, 0.0f};

    // software pipeline: the next stage's 16 KB of A and B slots are loaded into
    // registers while the current stage is multiplied out of LDS
    u4 ra[PER_T], rb[PER_T];
    if (k0 < k1) load_stage(gA, gB, k0, k1, tid, ra, rb);
    for (int64_t ks = k0; ks < k1; ks += MSTAGE) {
        const int nsl = (int)min((int64_t)MSTAGE, k1 - ks);
        __syncthreads();
#pragma unroll
        for (int k = 0; k < PER_T; ++k) {
            As[tid + 256 * k] = ra[k];
            Bs[tid + 256 * k] = rb[k];
        }
        __syncthreads();
        if (ks + MSTAGE < k1) load_stage(gA, gB, ks + MSTAGE, k1, tid, ra, rb);
#pragma unroll
        for (int j = 0; j < MSTAGE / 4; ++j) {
            if (4 * j >= nsl) break;
            u4 av[4], bv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) av[i] = As[(4 * j + grp) * BM + wr + 16 * i + i16];
#pragma unroll
            for (int c = 0; c < 4; ++c) bv[c] = Bs[(4 * j + grp) * BN + wc + 16 * c + i16];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int c = 0; c < 4; ++c)
                    acc[i][c] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(
                        frag(av[i]), frag(bv[c]), acc[i][c], 4, 4, 0, 127, 0, 127);
        }
    }

    if (SPLIT) {
        // partial sums of this split as int32 [tile][split][128 rows][128 columns]
        int32_t *part = ws_ptr<int32_t>(ws, lay.off_part) + ((size_t)tile * g.S + s) * BM * BN;
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int c = 0; c < 4; ++c)
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    part[(wr + 16 * i + 4 * grp + e) * BN + wc + 16 * c + i16] = (int32_t)acc[i][c][e];
    } else {
        // transpose through LDS, 64 rows at a time, so that each thread decodes four
        // adjacent columns of one row
        int32_t *T = reinterpret_cast<int32_t *>(smem);    // 64 x 132 int32
        constexpr int TS = BN + 4;
        for (int h = 0; h < 2; ++h) {
            __syncthreads();
            if (wr == 64 * h) {
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int c = 0; c < 4; ++c)
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            T[(16 * i + 4 * grp + e) * TS + wc + 16 * c + i16] = (int32_t)acc[i][c][e];
            }
            __syncthreads();
            for (int k = 0; k < 8; ++k) {
                const int idx = tid + 256 * k;        // 64 rows x 32 column quads
                const int rl = idx >> 5, cq = idx & 31;
                const int j0 = tn * BN + 4 * cq;
                if (j0 >= g.N) continue;
                const int4 v = *reinterpret_cast<const int4 *>(&T[rl * TS + 4 * cq]);
                const int32_t P[4] = {v.x, v.y, v.z, v.w};
                mdecode4<BIP>(P, tm * BM + 64 * h + rl, j0, min(4, g.N - j0), b, g, lay, ws);
            }
        }
    }
}

// sums the partial counts of every split of a tile and decodes (four blocks per tile,
// 32 rows each; thread = row x four adjacent columns)
template <bool BIP>
__global__ __launch_bounds__(256) void k_mgemm_reduce(MGemmArgs g, Layout lay, uint8_t *ws) {
    const int tile = blockIdx.x >> 2, quarter = blockIdx.x & 3;
    const int tn = tile % lay.NT;
    const int tb = tile / lay.NT;
    const int b = tb % g.batch, tm = tb / g.batch;
    const int4 *base = reinterpret_cast<const int4 *>(ws_ptr<int32_t>(ws, lay.off_part) +
                                                      (size_t)tile * g.S * BM * BN);
    for (int k = 0; k < 4; ++k) {
        const int idx = threadIdx.x + 256 * k;        // 32 rows x 32 column quads
        const int rl = quarter * 32 + (idx >> 5), cq = idx & 31;
        const int j0 = tn * BN + 4 * cq;
        if (j0 >= g.N) continue;
        int32_t P[4] = {0, 0, 0, 0};
        for (int s = 0; s < g.S; ++s) {
            const int4 v = base[((size_t)s * BM + rl) * (BN / 4) + cq];
            P[0] += v.x;
            P[1] += v.y;
            P[2] += v.z;
            P[3] += v.w;
        }
        mdecode4<BIP>(P, tm * BM + rl, j0, min(4, g.N - j0), b, g, lay, ws);
    }
}

template <bool BIP>
static hipError_t launch_mgemm_pol(const MGemmArgs &g, const Layout &lay, uint8_t *ws,
                                   hipStream_t st) {
    const unsigned tiles = (unsigned)(g.batch * lay.MT * lay.NT);
    if (g.S == 1) {
        hipLaunchKernelGGL((k_mgemm<BIP, false>), dim3(tiles), dim3(256), 0, st, g, lay, ws);
        return hipGetLastError();
    }
    hipLaunchKernelGGL((k_mgemm<BIP, true>), dim3(tiles * (unsigned)g.S), dim3(256), 0, st, g, lay,
                       ws);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((k_mgemm_reduce<BIP>), dim3(tiles * 4u), dim3(256), 0, st, g, lay, ws);
    return hipGetLastError();
}

hipError_t launch_mgemm(const sc_gemm_desc &d, const Layout &lay, const float *sA, const float *sB,
                        float *out, int32_t *counts, uint8_t *ws, hipStream_t st) {
    MGemmArgs g{};
    g.M = d.M;
    g.N = d.N;
    g.K = d.K;
    g.KQP = lay.KQP;
    g.LBS = lay.LBS;
    g.nbB = lay.nbB;
    g.batch = d.batch;
    g.S = lay.S;
    g.sA = sA;
    g.sB = sB;
    g.strideSA = d.strideSA;
    g.strideSB = d.strideSB;
    g.strideO = d.strideO;
    g.ldo = d.ldo;
    g.out = out;
    g.counts = counts;
    if (d.polarity == SC_BIPOLAR_XNOR) return launch_mgemm_pol<true>(g, lay, ws, st);
    return launch_mgemm_pol<false>(g, lay, ws, st);
}

}  // namespace scg
