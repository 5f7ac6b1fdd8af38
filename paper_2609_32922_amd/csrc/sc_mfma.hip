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
// v_mfma_scale_f32_32x32x64_f8f6f4 with unit scales sums 64 such products into fp32;
// a work unit sums at most 2^24 products per output (longer inner ranges are split, see
// make_layout), so every partial sum is an exact integer, the int32 partial counts of a
// split tile add exactly, and the count is independent of the summation order.
//
//   k_mplanes     nibble planes of A (sorted rows, per-row lengths) or B, one block per
//                 128-row tile x 64 cycles x 64 elements; element parameters and an
//                 8-cycle lookup table in LDS, 16-byte stores, 1 KB per wave; with
//                 comparator streams (M <= 128) both operands in one launch (k_mplanes2)
//   k_fgemm       N <= 128 with comparator streams where k_rgemm does not apply (M <= 128,
//                 or 64 < N <= 128): 128x128 tile, the fp4 fragments of both operands built
//                 in LDS from the int8 rows (an 8-cycle table per octet indexed by the int8
//                 byte), so no planes are written or read
//   k_rchunks     int8 operands (A in the scheduler's row order) laid out in 32-element
//                 chunks per 256-row pair through LDS (rows read along, chunks written
//                 contiguous), the input of k_rgemm; its last grid slice builds the table
//                 entries of every 32-cycle group once per call
//   k_rgemm       M > 128 and N > 128 (or N <= 64) with comparator streams: the tiles and
//                 division of k_qgemm, but every fp4 fragment is one LDS table read (a table
//                 per 32-cycle group indexed by the int8 byte), so no planes exist and the
//                 loop has no stage buffers; rows ending inside a group read tables masked
//                 to their length (a second variant masks every fragment when a row pair
//                 holds too many such lengths); for N <= 64 blocks of 256 x 64, two per CU,
//                 two waves on each row half splitting every chunk's k-steps (two waves per
//                 SIMD).
//                 A block copies each group's table entries into LDS (prefetched during
//                 the previous group); a whole tile decodes from row and column data
//                 staged in LDS, a part stores int32 partial sums
//   k_qgemm       N > 128 and M > 128 with C-BSG streams: 256x256 output tile per
//                 256-thread block, one block per CU, 128x128 per wave as 4x4 32x32 MFMA
//                 blocks, three LDS buffers of 4 slots (96 KB), memory instructions
//                 interleaved one per MFMA.  Whole tiles in full rounds, the tiles of a last
//                 partial round (or every tile, when row lengths vary) split along k.
//   k_qgemm_reduce sums the partial counts of the split tiles of k_qgemm or k_rgemm and
//                 decodes (8-row blocks when few tiles are split, 32-row blocks otherwise)
//   k_mgemm       the rest (M <= 128, or N <= 128 with C-BSG streams): 128x256 output
//                 tile per 256-thread block (128x128 and 64x64 when N <= 128), 64x128 per
//                 wave as 2x4 32x32 MFMA blocks, 4 slots (2 MFMA k-steps of 64) per LDS
//                 stage, two LDS buffers (48 KB: two blocks per CU).  The 32x32x64 form
//                 keeps the matrix cores fed where the 16x16x128 form loses several cycles
//                 per instruction to issue.
//   k_mgemm_reduce sums the partial counts of split tiles and decodes
#include <hip/hip_ext.h>
#include <limits.h>

#include "sc_internal.h"

namespace scg {

namespace {
thread_local hipEvent_t t_ev_begin = nullptr, t_ev_end = nullptr;
thread_local bool t_ev_taken = false;
}  // namespace

void set_gemm_events(hipEvent_t begin, hipEvent_t end) {
    t_ev_begin = begin;
    t_ev_end = end;
    t_ev_taken = false;
}
bool gemm_events_taken() { return t_ev_taken; }

// Launch of a counting-GEMM kernel, `last` when no other kernel of the call follows it
// (set_gemm_events: the events ride on the dispatches themselves)
template <typename F, typename... Args>
static void gemm_launch(F kernel, dim3 grid, dim3 block, hipStream_t st, bool last, Args... args) {
    hipEvent_t e0 = t_ev_begin, e1 = last ? t_ev_end : nullptr;
    if (e0 == nullptr && e1 == nullptr) {
        hipLaunchKernelGGL(kernel, grid, block, 0, st, args...);
        return;
    }
    hipExtLaunchKernelGGL(kernel, grid, block, 0, st, e0, e1, 0, args...);
    t_ev_begin = nullptr;
    t_ev_taken = true;
}

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v2i __attribute__((ext_vector_type(2)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));   // one slot row: 32 nibbles
typedef uint32_t u2 __attribute__((ext_vector_type(2)));

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
struct MPlaneShared {
    uint32_t prm[64 * PRM_STRIDE];    // [element][row] packed parameters
    uint32_t lut[OCH * CA_COLS];      // comparator: 8 nibbles per octet and beta
    uint32_t spread[256];             // interval: 8-bit mask -> 8 nibbles of +1
    uint32_t rr[OCH * MSTEP];         // comparator: the block's draws
    int rowok[BM];                    // row of the tile holds data (not padding)
};

// block (x, y = element group, z = batch entry) of one side's grid
template <int POL, bool CBSG>
__device__ __forceinline__ void mplanes_block(const MPlaneArgs &a, uint8_t *ws, MPlaneShared &sh, int bx,
                                              int by, int bz) {
    uint32_t *prm = sh.prm, *lut = sh.lut, *spread = sh.spread, *rr = sh.rr;
    int *rowok = sh.rowok;
    const int t = bx / a.nchunk, ch = bx % a.nchunk;
    const int qg = by, b = bz;
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
        // B: every cycle up to L_max, or only up to the longest tile pair of the call when
        // the scheduler recorded it (256-row GEMM): no tile reads B's planes beyond it
        Lloop = a.LBS;
        const int longest = (int)ws_ptr<uint32_t>(ws, 0)[1];
        if (longest > 0 && longest < Lloop) Lloop = longest;
        off = (int64_t)t * a.LBS * a.KQP * 64;
    }
    const int o0 = ch * OCH;
    if (o0 * MSTEP >= Lloop) return;
    const int no = min(OCH, Lloop / MSTEP - o0);
    const int8_t *Xb = a.X + (size_t)b * a.strideX;
    const uint16_t *CA = CBSG ? ws_ptr<uint16_t>(ws, a.off_CA) : nullptr;

    // 1. element parameters.  Wave w takes rows m = w + 4k, k < 32: lane k first loads
    //    row k's index and length (one vector load), then the wave issues the 32 element
    //    loads (64 bytes of one row each) back to back before using any of them.
    const int d = qg * 64 + lane;
    int rowv = -1, Lv = 0;
    if (lane < 32) {
        const int p = t * BM + w + 4 * lane;
        if (a.per_row) {
            rowv = perm[p];
            Lv = rowv >= 0 ? Ls[p] : 0;
        } else {
            rowv = p < a.rows ? p : -1;
            Lv = a.uniformL;
        }
    }
    // padding rows and elements read row 0 / element 0 (present whenever this kernel
    // runs: rows >= 1, K >= 1) and are zeroed below, so no load sits behind a branch
    if (lane < 32) rowok[w + 4 * lane] = rowv >= 0;
    int qv[32];
    const int dd = d < a.K ? d : 0;
#pragma unroll
    for (int k = 0; k < 32; ++k) {
        const int row = max(__builtin_amdgcn_readlane(rowv, k), 0);
        qv[k] = (int)Xb[(size_t)row * a.ld + dd];
    }
#pragma unroll
    for (int k = 0; k < 32; ++k) {
        const int m = w + 4 * k;
        const int row = __builtin_amdgcn_readlane(rowv, k), Lr = __builtin_amdgcn_readlane(Lv, k);
        const bool valid = row >= 0 && d < a.K;
        const int q = valid ? qv[k] : 0;
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
        if (tid < no * MSTEP) rr[tid] = ws_ptr<uint32_t>(ws, a.off_r)[(size_t)o0 * MSTEP + tid];
        __syncthreads();
        const uint32_t zero_nib = POL == SC_BIPOLAR_XNOR ? NIB_NEG : 0u;
        for (int e = tid; e < no * CA_COLS; e += 256) {
            const int o = e / CA_COLS, beta = e % CA_COLS;
            uint32_t x = 0;
#pragma unroll
            for (int c = 0; c < 8; ++c)
                x |= (rr[o * MSTEP + c] < (uint32_t)beta ? NIB_POS : zero_nib) << (4 * c);
            lut[e] = x;
        }
    }
    __syncthreads();

    // 3. planes: thread (half h = tid / 128, row m = tid % 128) writes the 16 bytes of
    //    row m in slot (octet, quad 2 * pair + h); one wave stores 1 KB contiguously.
    //    Padding rows (beyond M or N) are not written: the GEMM reads them (in bounds,
    //    and every e2m1 code is finite) only into outputs that are never stored.
    u4 *planes = reinterpret_cast<u4 *>(ws_ptr<uint32_t>(wsb, a.off_planes) + off);
    const int m = tid & (BM - 1), h = tid >> 7;
    const bool store_row = rowok[m] != 0;
    // the thread's 8 quads x 4 elements of row m, the same for every octet
    uint32_t pks[8][4];
#pragma unroll
    for (int pr = 0; pr < 8; ++pr)
#pragma unroll
        for (int e = 0; e < 4; ++e) pks[pr][e] = prm[(4 * (2 * pr + h) + e) * PRM_STRIDE + m];
    const int npr = min(8, (a.KQP - qg * 16 - h + 1) / 2);     // quads 2 pr + h below KQP
    for (int o = 0; o < no; ++o) {
        const int oa = o0 + o, c0 = oa * MSTEP;
#pragma unroll
        for (int pr = 0; pr < 8; ++pr) {
            const int dq = 2 * pr + h, qd = qg * 16 + dq;
            if (pr >= npr) break;
            u4 v;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const uint32_t pk = pks[pr][e];
                uint32_t x;
                if (CBSG) {
                    const int lo = (int)(pk & 511u), hi = (int)((pk >> 9) & 511u);
                    const int a0 = min(max(lo - c0, 0), 8), a1 = min(max(hi - c0, 0), 8);
                    x = spread[((1u << a1) - 1u) & ~((1u << a0) - 1u)];
                } else {
                    const int beta = (int)(pk & 511u), Le = (int)((pk >> 9) & 8191u);
                    const int rem = Le - c0;
                    x = lut[o * CA_COLS + beta];
                    if (rem <= 0) x = 0u;
                    else if (rem < 8) x &= (1u << (4 * rem)) - 1u;
                }
                v[e] = (pk >> 31) ? negate_nibbles(x) : x;
            }
            if (store_row) planes[((size_t)oa * a.KQP + qd) * BM + m] = v;
        }
    }
}

template <int POL, bool CBSG>
__global__ __launch_bounds__(256) void k_mplanes(MPlaneArgs a, uint8_t *ws) {
    __shared__ MPlaneShared sh;
    mplanes_block<POL, CBSG>(a, ws, sh, blockIdx.x, blockIdx.y, blockIdx.z);
}

// both sides in one launch (comparator streams): blocks [0, nA) are A's grid
// (gxA x gy x batch), the rest B's (gxB x gy x nbB), so B's blocks fill A's last wave
template <int POL>
__global__ __launch_bounds__(256) void k_mplanes2(MPlaneArgs a, MPlaneArgs bb, int gxA, int gxB, int gy,
                                                  int nA, uint8_t *ws) {
    __shared__ MPlaneShared sh;
    const int bid = blockIdx.x;
    if (bid < nA) {
        mplanes_block<POL, false>(a, ws, sh, bid % gxA, (bid / gxA) % gy, bid / (gxA * gy));
    } else {
        const int v = bid - nA;
        mplanes_block<POL, false>(bb, ws, sh, v % gxB, (v / gxB) % gy, v / (gxB * gy));
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
    if (cbsg) {
        launch_mplanes_side<true>(d.polarity, gA, pa, ws, st);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }

    MPlaneArgs pb = pa;
    pb.X = B;
    pb.ld = d.ldb;
    pb.strideX = d.strideB;
    pb.rows = d.N;
    pb.nchunk = (lay.LBS / MSTEP + OCH - 1) / OCH;
    pb.uniformL = d.L_max;
    pb.per_row = 0;
    pb.stride_batch = lay.stride_batchB;
    pb.off_perm = pb.off_Ls = pb.off_tileL = pb.off_tileOff = 0;
    pb.off_planes = lay.off_Bp;
    pb.off_r = lay.off_rB;
    pb.off_CA = 0;
    const dim3 gB((unsigned)(lay.NT * pb.nchunk), qgroups, (unsigned)lay.nbB);
    if (cbsg) {
        launch_mplanes_side<false>(d.polarity, gB, pb, ws, st);
        return hipGetLastError();
    }
    const int nA = (int)(gA.x * gA.y * gA.z), nB = (int)(gB.x * gB.y * gB.z);
    if (d.polarity == SC_BIPOLAR_XNOR)
        hipLaunchKernelGGL((k_mplanes2<SC_BIPOLAR_XNOR>), dim3((unsigned)(nA + nB)), dim3(256), 0, st, pa, pb,
                           (int)gA.x, (int)gB.x, (int)qgroups, nA, ws);
    else
        hipLaunchKernelGGL((k_mplanes2<SC_UNIPOLAR_AND_SM>), dim3((unsigned)(nA + nB)), dim3(256), 0, st, pa, pb,
                           (int)gA.x, (int)gB.x, (int)qgroups, nA, ws);
    return hipGetLastError();
}

// ----------------------------------------------------------------------------
// MFMA GEMM
// ----------------------------------------------------------------------------
struct MGemmArgs {
    int M, N, K, KQP, LBS, nbB, batch, S, F, KC;
    const float *sA, *sB;
    int64_t strideSA, strideSB, strideO, ldo;
    float *out;
    int32_t *counts;
    int vec_out, vec_cnt;   // four adjacent columns of out (counts) at a multiple of 4 are 16-byte aligned
};

// Eq. (1) decode in fp32, one formula for every kernel: row i of scale sA_i and length L
// gets the factor f_i = (sA_i 127^2) / L (0 when L = 0), and the output is (P f_i) sB_j,
// P the row's product sum (bipolar: 2X - K L; unipolar: the signed AND count S), an exact
// integer held in fp32.
__device__ __forceinline__ float decode_factor(float sAi, int L) {
    return L > 0 ? (sAi * 16129.0f) / (float)L : 0.0f;
}

// Store four adjacent columns j0.. (ncol of them in range) of original row i of batch entry
// b from their product sums: P as fp32 for the output; for the counts (bipolar: X = (K L +
// P) / 2) the exact int32 sums Pi when PINT, else P itself (an exact integer below 2^24).
template <bool BIP, bool PINT>
__device__ __forceinline__ void decode4_store(const float (&P)[4], const int32_t (&Pi)[4], int i, int Li, float f,
                                              const float (&sBj)[4], int j0, int ncol, int b, const MGemmArgs &g) {
    float o[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) o[c] = (P[c] * f) * sBj[c];
    const size_t off = (size_t)b * g.strideO + (size_t)i * g.ldo + j0;
    // (non-temporal: the outputs are not read again here; ViT-B fc1 with mixed lengths -0.9 %,
    // the compensator -2 %)
    typedef float f4nt __attribute__((ext_vector_type(4)));
    typedef int i4nt __attribute__((ext_vector_type(4)));
    if (ncol == 4 && g.vec_out) {
        __builtin_nontemporal_store(f4nt{o[0], o[1], o[2], o[3]}, reinterpret_cast<f4nt *>(g.out + off));
    } else {
        for (int c = 0; c < ncol; ++c) g.out[off + c] = o[c];
    }
    if (g.counts) {
        const int KL = Li > 0 ? g.K * Li : 0;
        int32_t cnt[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int32_t p = PINT ? Pi[c] : (int32_t)P[c];
            cnt[c] = Li > 0 ? (BIP ? (KL + p) / 2 : p) : 0;
        }
        if (ncol == 4 && g.vec_cnt) {
            __builtin_nontemporal_store(i4nt{cnt[0], cnt[1], cnt[2], cnt[3]}, reinterpret_cast<i4nt *>(g.counts + off));
        } else {
            for (int c = 0; c < ncol; ++c) g.counts[off + c] = cnt[c];
        }
    }
}

// the same for sorted row position p, its row, length and scales read from global memory
template <bool BIP>
__device__ __forceinline__ void mdecode4(const int32_t (&P)[4], int p, int j0, int ncol, int b,
                                         const MGemmArgs &g, const Layout &lay, uint8_t *ws) {
    uint8_t *wsa = ws + (size_t)b * lay.stride_batchA;
    const int i = ws_ptr<int32_t>(wsa, lay.off_perm)[p];
    if (i < 0) return;
    const int Li = ws_ptr<int32_t>(wsa, lay.off_Ls)[p];
    const float f = decode_factor(g.sA[(size_t)b * g.strideSA + i], Li);
    const float *sBb = g.sB + (size_t)b * g.strideSB;
    float sBj[4];
    const float Pf[4] = {(float)P[0], (float)P[1], (float)P[2], (float)P[3]};
#pragma unroll
    for (int c = 0; c < 4; ++c) sBj[c] = sBb[c < ncol ? j0 + c : j0];
    decode4_store<BIP, true>(Pf, P, i, Li, f, sBj, j0, ncol, b, g);
}

// What the decode of a whole 256-row tile needs, staged in LDS once per tile: per row of
// the pair its original row (-1: padding), length and decode factor; per column its scale.
struct DecodeLds {
    int32_t row[256], len[256];
    float f[256], sB[256];
};

template <int NT>
__device__ __forceinline__ void d_stage(DecodeLds &d, const int32_t *perm, const int32_t *Ls, int b, int tw,
                                        const MGemmArgs &g, int tid) {
    for (int r = tid; r < 256; r += NT) {
        const int i = perm[r];
        const int L = i >= 0 ? Ls[r] : 0;
        d.row[r] = i;
        d.len[r] = L;
        d.f[r] = i >= 0 ? decode_factor(g.sA[(size_t)b * g.strideSA + i], L) : 0.0f;
        const int j = tw * 256 + r;
        d.sB[r] = j < g.N ? g.sB[(size_t)b * g.strideSB + j] : 0.0f;
    }
}

// The same data for one row per thread (256 threads), in two steps: the loads (every row's
// length is in the layout, padding rows' too, so only the decode factor's scale waits for the
// row's original index), then the LDS stores
struct DRow {
    int32_t i, L;
    float sa, sb;
};
__device__ __forceinline__ DRow d_fetch(const int32_t *perm, const int32_t *Ls, int b, int tw, const MGemmArgs &g,
                                        int r) {
    DRow x;
    x.i = perm[r];
    x.L = Ls[r];
    const int j = tw * 256 + r;
    x.sb = j < g.N ? g.sB[(size_t)b * g.strideSB + j] : 0.0f;
    x.sa = x.i >= 0 ? g.sA[(size_t)b * g.strideSA + x.i] : 0.0f;
    return x;
}
__device__ __forceinline__ void d_put(DecodeLds &d, const DRow &x, int r) {
    d.row[r] = x.i;
    d.len[r] = x.i >= 0 ? x.L : 0;
    d.f[r] = x.i >= 0 ? decode_factor(x.sa, x.L) : 0.0f;
    d.sB[r] = x.sb;
}

// Decode of TR rows of a whole tile from their sums T (fp32, row-major, row stride TS, the
// tile's columns from 0): thread tid takes column quad tid % NQ of rows tid / NQ + k NT / NQ.
// All of a thread's LDS reads are issued before its stores.
template <bool BIP, int NT, int NQ, int TR, int TS>
__device__ __forceinline__ void d_rows(const DecodeLds &d, const float *T, int row0, int tw, int b,
                                       const MGemmArgs &g, int tid) {
    constexpr int RPW = NT / NQ, KQ = TR / RPW, KB = KQ < 8 ? KQ : 8;   // rows per thread, per batch
    const int cq = tid % NQ, r0 = tid / NQ;
    const int j0 = tw * 256 + 4 * cq;
    const int ncol = min(4, g.N - j0);
    if (ncol <= 0) return;
    float sBj[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) sBj[c] = d.sB[4 * cq + (c < ncol ? c : 0)];
#pragma unroll
    for (int k0 = 0; k0 < KQ; k0 += KB) {
        float4 v[KB];
        int row[KB], len[KB];
        float f[KB];
#pragma unroll
        for (int k = 0; k < KB; ++k) {
            const int rl = r0 + RPW * (k0 + k);
            v[k] = *reinterpret_cast<const float4 *>(&T[rl * TS + 4 * cq]);
            row[k] = d.row[row0 + rl];
            len[k] = d.len[row0 + rl];
            f[k] = d.f[row0 + rl];
        }
#pragma unroll
        for (int k = 0; k < KB; ++k) {
            if (row[k] < 0) continue;
            const float P[4] = {v[k].x, v[k].y, v[k].z, v[k].w};
            const int32_t none[4] = {0, 0, 0, 0};
            decode4_store<BIP, false>(P, none, row[k], len[k], f[k], sBj, j0, ncol, b, g);
        }
    }
}

// Partial sums of a piece of a 256-row tile, in the MFMA's own layout: [row block rb of 32
// rows][column block cb of 32 columns][quad q][lane][4] int32, with (rb, cb) numbered
// rb * (PC / 32) + cb for a piece PC columns wide.  Lane (grp, i32) of quad q holds rows
// 32 rb + 8 q + 4 grp + j (j = 0..3) of column 32 cb + i32: the four accumulator elements
// 4q .. 4q + 3 of its 32 x 32 block, stored as one 16-byte store (a wave writes 1 KB at a time).
template <int PC>
__device__ __forceinline__ void store_block(const v16f &a, __amdgpu_buffer_rsrc_t pr, int lane, int rb, int cb) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const v4i v = {(int)a[4 * q], (int)a[4 * q + 1], (int)a[4 * q + 2], (int)a[4 * q + 3]};
        __builtin_amdgcn_raw_buffer_store_b128(v, pr, lane * 16, (((rb * (PC / 32) + cb) * 4 + q) * 64) * 16, 0);
    }
}

// The same layout with int16 counts (8 bytes per lane and quad; the counts fit, see P16_STEPS)
template <int PC>
__device__ __forceinline__ void store_block16(const v16f &a, __amdgpu_buffer_rsrc_t pr, int lane, int rb, int cb) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const v2i v = {(int)(((uint32_t)(int)a[4 * q] & 0xFFFFu) | ((uint32_t)(int)a[4 * q + 1] << 16)),
                       (int)(((uint32_t)(int)a[4 * q + 2] & 0xFFFFu) | ((uint32_t)(int)a[4 * q + 3] << 16))};
        __builtin_amdgcn_raw_buffer_store_b64(v, pr, lane * 8, (((rb * (PC / 32) + cb) * 4 + q) * 64) * 8, 0);
    }
}

// A wave's 4 x NB blocks of 32 x 32 at rows wr + 32 i, columns wc + 32 c (256-column pieces)
template <int NB>
__device__ __forceinline__ void store_part(const v16f (&acc)[4][NB], int32_t *part, int wr, int wc, int lane) {
    const __amdgpu_buffer_rsrc_t pr = __builtin_amdgcn_make_buffer_rsrc(part, 0, 256 * 256 * 4, 0x00020000);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int c = 0; c < NB; ++c) store_block<256>(acc[i][c], pr, lane, wr / 32 + i, wc / 32 + c);
}

// The same for the int8-chunk GEMM, whose wave of row half rh holds the pair's row blocks
// starting at r_row0<SKIP>(rh, i) (declared with that GEMM below); a piece is the block's
// columns wide (256, or 64 for the 256 x 64 blocks).
template <bool SKIP>
__device__ __forceinline__ int r_row0(int rh, int i);
template <bool SKIP, int NB>
__device__ __forceinline__ void store_part_r(const v16f (&acc)[4][NB], uint8_t *part, bool p16, int rh, int wc,
                                             int lane) {
    constexpr int PC = NB == 2 ? 64 : 256;
    const __amdgpu_buffer_rsrc_t pr =
        __builtin_amdgcn_make_buffer_rsrc(part, 0, 256 * PC * (p16 ? 2 : 4), 0x00020000);
    if (p16) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int c = 0; c < NB; ++c) store_block16<PC>(acc[i][c], pr, lane, r_row0<SKIP>(rh, i) / 32, wc / 32 + c);
    } else {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int c = 0; c < NB; ++c) store_block<PC>(acc[i][c], pr, lane, r_row0<SKIP>(rh, i) / 32, wc / 32 + c);
    }
}

// Block tile: BM = 128 rows of A x WB columns of B, WB = 256 (two 128-column B plane
// tiles) or 128 (one; taken when N <= 128, where a wider tile would mostly multiply
// padding).
constexpr int PER_TA = MSTAGE * BM / 256;   // u4 of A per thread per stage
constexpr int KSTEPS = MSTAGE / 2;          // MFMA k-steps (2 slots = 64 k each) per stage

template <int WB>
struct MTile {
    static constexpr int PER_TB = MSTAGE * WB / 256;   // u4 of B per thread per stage
    static constexpr int BUF = MSTAGE * (BM + WB);     // u4 per LDS buffer (A slots, then B)
    static constexpr int NCB = WB / 64;                // 32-column MFMA blocks per wave
};

template <int WB>
struct Stage {
    u4 a[PER_TA], b[MTile<WB>::PER_TB];
};

// Loads the stage of slots [ks, ks + MSTAGE) into registers.  A short last stage re-reads
// its last slot instead of running past the unit (the compute loop never reads those
// LDS entries), so every load is in bounds.  In pass k thread tid takes A row tid % 128
// of slot 2k + tid / 128, and B column tid % WB (of the block's WB) of slot
// k * 256 / WB + tid / WB; columns 128.. come from the second B plane tile.
template <int WB>
__device__ __forceinline__ void load_stage(const u4 *gA, const u4 *gB0, const u4 *gB1, int64_t ks,
                                           int64_t k1, int tid, Stage<WB> &r) {
    const int last = (int)min((int64_t)MSTAGE, k1 - ks) - 1;
    const u4 *pa = gA + ks * BM + (tid & (BM - 1));
    const int col = tid % WB;
    const u4 *pb = (col < BN ? gB0 : gB1) + ks * BN + (col & (BN - 1));
#pragma unroll
    for (int k = 0; k < PER_TA; ++k) r.a[k] = pa[min(2 * k + (tid >> 7), last) * BM];
#pragma unroll
    for (int k = 0; k < MTile<WB>::PER_TB; ++k)
        r.b[k] = pb[min(k * (256 / WB) + tid / WB, last) * BN];
}

// LDS buffer: A [MSTAGE][128], then B [MSTAGE][WB]
template <int WB>
__device__ __forceinline__ void store_stage(u4 *buf, int tid, const Stage<WB> &r) {
#pragma unroll
    for (int k = 0; k < PER_TA; ++k) buf[tid + 256 * k] = r.a[k];
#pragma unroll
    for (int k = 0; k < MTile<WB>::PER_TB; ++k) buf[MSTAGE * BM + 256 * k + tid] = r.b[k];
}

// operand fragments of k-step j of an LDS buffer for one wave (64 rows x WB/2 columns):
// A rows wr + 32i + l%32, B columns wc + 32c + l%32, slot 2j + l/32 (the 32x32x64 operand
// layout: 32 consecutive k per lane, lanes 32..63 holding the second half of k)
template <int WB>
struct Frags {
    u4 a[2], b[MTile<WB>::NCB];
};
template <int WB>
__device__ __forceinline__ void read_frags(const u4 *buf, int j, int grp, int wr, int wc, int i32,
                                           Frags<WB> &f) {
    const u4 *As = buf + (2 * j + grp) * BM, *Bs = buf + MSTAGE * BM + (2 * j + grp) * WB;
#pragma unroll
    for (int i = 0; i < 2; ++i) f.a[i] = As[wr + 32 * i + i32];
#pragma unroll
    for (int c = 0; c < MTile<WB>::NCB; ++c) f.b[c] = Bs[wc + 32 * c + i32];
}

__device__ __forceinline__ v8i frag(u4 x) {
    v8i r = {(int)x[0], (int)x[1], (int)x[2], (int)x[3], 0, 0, 0, 0};
    return r;
}

// the MFMAs of one k-step of a wave's tile
template <int WB>
__device__ __forceinline__ void mma(v16f (&acc)[2][MTile<WB>::NCB], const Frags<WB> &f) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int c = 0; c < MTile<WB>::NCB; ++c)
            acc[i][c] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(frag(f.a[i]), frag(f.b[c]),
                                                                        acc[i][c], 4, 4, 0, 127, 0, 127);
}

// One stage of the block's pipeline.  On entry the fragments of the stage's first
// k-step are in fragment set PF, LDS buffer st % 2 holds the stage, and register set
// 1 - PR holds stage st + 1 (loaded during stage st - 1).  The loads of stage st + 2
// go into register set PR, so global latency is covered by two stages of MFMAs; k-step
// j+1's fragments are read while the MFMAs of k-step j issue, and the next stage's
// first k-step right after the barrier, while the last MFMAs of this stage still run.
template <int WB, int PF, int PR>
__device__ __forceinline__ void mstage(int64_t st, int64_t nst, int64_t k0, int64_t k1, const u4 *gA,
                                       const u4 *gB0, const u4 *gB1, u4 *smem, int tid, int grp,
                                       int wr, int wc, int i32, v16f (&acc)[2][MTile<WB>::NCB],
                                       Frags<WB> (&f)[2], Stage<WB> (&r)[2]) {
    constexpr int BUF = MTile<WB>::BUF;
    // Loads and LDS reads are issued unconditionally (past the last stage they re-read
    // the last stage, in bounds, and their data is never used) so that the wait counts
    // before each use are fixed and only cover the older group.
    const int64_t ks = k0 + st * MSTAGE, klast = k0 + (nst - 1) * MSTAGE;
    const int nk = (int)min((int64_t)MSTAGE, k1 - ks) / 2;        // k-steps in this stage
    const bool more = st + 1 < nst;
    load_stage<WB>(gA, gB0, gB1, min(ks + 2 * MSTAGE, klast), k1, tid, r[PR]);
    // keep the loads at the top of the stage: the scheduler would otherwise sink them
    // next to their LDS stores and expose their latency
    __builtin_amdgcn_sched_barrier(0);
    const u4 *buf = smem + (st & 1) * BUF;
    __builtin_amdgcn_s_setprio(1);       // favour this wave's MFMA issue over its neighbour's
#pragma unroll
    for (int j = 0; j < KSTEPS; ++j) {
        if (j + 1 < KSTEPS) read_frags<WB>(buf, j + 1, grp, wr, wc, i32, f[(PF + j + 1) & 1]);
        if (j < nk) mma<WB>(acc, f[(PF + j) & 1]);
    }
    __builtin_amdgcn_s_setprio(0);
    __builtin_amdgcn_sched_barrier(0);
    u4 *nbuf = smem + ((st + 1) & 1) * BUF;
    if (more) store_stage<WB>(nbuf, tid, r[1 - PR]);
    __syncthreads();
    // a stage that has a successor is full: its successor starts in set PF + KSTEPS
    read_frags<WB>(nbuf, 0, grp, wr, wc, i32, f[(PF + KSTEPS) & 1]);
}

// One block: the 128 x WB tile (tm, tw) of batch entry b over a contiguous range of MFMA
// k-steps (2 slots each).  Wave w owns rows 64*(w/2).., columns (WB/2)*(w%2)..; lane l
// reads slot 2j + l/32 of row (or column) l%32 of each 32-row block.  The accumulator
// element e of lane l is row 8*(e/4) + 4*(l/32) + e%4, column l%32 of its 32x32 block.
template <bool BIP, bool SPLIT, int WB>
__global__ __launch_bounds__(256, 2) void k_mgemm(MGemmArgs g, Layout lay, uint8_t *ws) {
    constexpr int BUF = MTile<WB>::BUF, NCB = MTile<WB>::NCB;
    __shared__ u4 smem[2 * BUF];
    const int NTW = lay.NT / (WB / BN);
    const int u = blockIdx.x;
    const int s = u % g.S;
    const int tile = u / g.S;
    const int tw = tile % NTW;
    const int tb = tile / NTW;
    const int b = tb % g.batch, tm = tb / g.batch;
    const int bB = g.nbB == 1 ? 0 : b;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int grp = lane >> 5, i32 = lane & 31;
    const int wr = (w >> 1) * 64, wc = (w & 1) * (WB / 2);
    uint8_t *wsa = ws + (size_t)b * lay.stride_batchA;
    uint8_t *wsbB = ws + (size_t)bB * lay.stride_batchB;
    const int Lloop = ws_ptr<int32_t>(wsa, lay.off_tileL)[tm];
    const int64_t nsteps = (int64_t)(Lloop / MSTEP) * g.KQP / 2;       // k-steps of 2 slots
    const int64_t k0 = (int64_t)s * nsteps / g.S * 2, k1 = (int64_t)(s + 1) * nsteps / g.S * 2;
    const u4 *gA = reinterpret_cast<const u4 *>(ws_ptr<uint32_t>(wsa, lay.off_Ap) +
                                                ws_ptr<int64_t>(wsa, lay.off_tileOff)[tm]);
    const size_t btile = (size_t)(g.LBS / MSTEP) * g.KQP * BN;          // u4 per B plane tile
    const u4 *gB0 = reinterpret_cast<const u4 *>(ws_ptr<uint32_t>(wsbB, lay.off_Bp)) +
                    (size_t)tw * (WB / BN) * btile;
    const u4 *gB1 = WB > BN ? gB0 + btile : gB0;

    v16f acc[2][NCB];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int c = 0; c < NCB; ++c) acc[i][c] = v16f{};

    Stage<WB> r[2];
    Frags<WB> f[2];
    const int64_t nst = (k1 - k0 + MSTAGE - 1) / MSTAGE;
    if (nst > 0) {
        load_stage<WB>(gA, gB0, gB1, k0, k1, tid, r[0]);
        store_stage<WB>(smem, tid, r[0]);
        load_stage<WB>(gA, gB0, gB1, k0 + min((int64_t)1, nst - 1) * MSTAGE, k1, tid, r[1]);
    }
    __syncthreads();
    if (nst > 0) read_frags<WB>(smem, 0, grp, wr, wc, i32, f[0]);
    // stages in pairs, so that the register set of a stage (st % 2) and the fragment set
    // of its first k-step are fixed at compile time
    for (int64_t st = 0; st < nst; st += 2) {
        mstage<WB, 0, 0>(st, nst, k0, k1, gA, gB0, gB1, smem, tid, grp, wr, wc, i32, acc, f, r);
        if (st + 1 < nst)
            mstage<WB, KSTEPS & 1, 1>(st + 1, nst, k0, k1, gA, gB0, gB1, smem, tid, grp, wr, wc, i32,
                                      acc, f, r);
    }

    if (SPLIT) {
        // partial sums of this split as int32 [tile][split][128 rows][WB columns]
        int32_t *part = ws_ptr<int32_t>(ws, lay.off_part) + ((size_t)tile * g.S + s) * BM * WB;
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int c = 0; c < NCB; ++c)
#pragma unroll
                for (int e = 0; e < 16; ++e)
                    part[(wr + 32 * i + 8 * (e >> 2) + 4 * grp + (e & 3)) * WB + wc + 32 * c + i32] =
                        (int32_t)acc[i][c][e];
    } else {
        // transpose through LDS, 32 rows at a time, so that each thread decodes four
        // adjacent columns of one row
        constexpr int TS = WB + 4, TR = 32;
        static_assert(TR * TS * 4 <= 2 * BUF * 16, "the epilogue transpose must fit the LDS buffers");
        int32_t *T = reinterpret_cast<int32_t *>(smem);    // 32 x (WB + 4) int32
        for (int h = 0; h < BM / TR; ++h) {
            __syncthreads();
            // pass h holds rows 32h .. 32h + 31: MFMA block i = h % 2 of the waves at wr = 64 (h / 2)
            if (wr == 64 * (h >> 1)) {
#pragma unroll
                for (int i = 0; i < 2; ++i) {
                    if (i != (h & 1)) continue;
#pragma unroll
                    for (int c = 0; c < NCB; ++c)
#pragma unroll
                        for (int e = 0; e < 16; ++e)
                            T[(8 * (e >> 2) + 4 * grp + (e & 3)) * TS + wc + 32 * c + i32] =
                                (int32_t)acc[i][c][e];
                }
            }
            __syncthreads();
            for (int k = 0; k < TR * (WB / 4) / 256; ++k) {
                const int idx = tid + 256 * k;        // 32 rows x WB/4 column quads
                const int rl = idx / (WB / 4), cq = idx % (WB / 4);
                const int j0 = tw * WB + 4 * cq;
                if (j0 >= g.N) continue;
                const int4 v = *reinterpret_cast<const int4 *>(&T[rl * TS + 4 * cq]);
                const int32_t P[4] = {v.x, v.y, v.z, v.w};
                mdecode4<BIP>(P, tm * BM + TR * h + rl, j0, min(4, g.N - j0), b, g, lay, ws);
            }
        }
    }
}

// sums the partial counts of every split of a tile and decodes (four blocks per tile,
// 32 rows each; thread = row x four adjacent columns).  The partial tiles are full-size,
// so every load is in bounds and all of a split's loads are issued together; padding
// rows and columns are dropped only at the decode.
template <bool BIP, int WB>
__global__ __launch_bounds__(256) void k_mgemm_reduce(MGemmArgs g, Layout lay, uint8_t *ws) {
    constexpr int NK = 32 * (WB / 4) / 256;           // row x column-quad items per thread
    const int NTW = lay.NT / (WB / BN);
    const int tile = blockIdx.x >> 2, quarter = blockIdx.x & 3;
    const int tw = tile % NTW;
    const int tb = tile / NTW;
    const int b = tb % g.batch, tm = tb / g.batch;
    const int4 *base = reinterpret_cast<const int4 *>(ws_ptr<int32_t>(ws, lay.off_part) +
                                                      (size_t)tile * g.S * BM * WB) +
                       (size_t)quarter * 32 * (WB / 4) + threadIdx.x;
    int4 sum[NK];
#pragma unroll
    for (int k = 0; k < NK; ++k) sum[k] = make_int4(0, 0, 0, 0);
    for (int s = 0; s < g.S; ++s) {
        const int4 *src = base + (size_t)s * BM * (WB / 4);
        int4 v[NK];
#pragma unroll
        for (int k = 0; k < NK; ++k) v[k] = src[256 * k];
#pragma unroll
        for (int k = 0; k < NK; ++k) {
            sum[k].x += v[k].x;
            sum[k].y += v[k].y;
            sum[k].z += v[k].z;
            sum[k].w += v[k].w;
        }
    }
    const int32_t *perm = ws_ptr<int32_t>(ws + (size_t)b * lay.stride_batchA, lay.off_perm);
#pragma unroll
    for (int k = 0; k < NK; ++k) {
        const int idx = threadIdx.x + 256 * k;        // 32 rows x WB/4 column quads
        const int rl = quarter * 32 + idx / (WB / 4), cq = idx % (WB / 4);
        const int j0 = tw * WB + 4 * cq;
        if (j0 >= g.N || perm[tm * BM + rl] < 0) continue;
        const int32_t P[4] = {sum[k].x, sum[k].y, sum[k].z, sum[k].w};
        mdecode4<BIP>(P, tm * BM + rl, j0, min(4, g.N - j0), b, g, lay, ws);
    }
}

template <bool BIP, int WB>
static hipError_t launch_mgemm_tile(const MGemmArgs &g, const Layout &lay, uint8_t *ws,
                                    hipStream_t st) {
    const unsigned tiles = (unsigned)(g.batch * lay.MT * (lay.NT / (WB / BN)));
    if (g.S == 1) {
        gemm_launch((k_mgemm<BIP, false, WB>), dim3(tiles), dim3(256), st, true, g, lay, ws);
        return hipGetLastError();
    }
    gemm_launch((k_mgemm<BIP, true, WB>), dim3(tiles * (unsigned)g.S), dim3(256), st, false, g, lay, ws);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    gemm_launch((k_mgemm_reduce<BIP, WB>), dim3(tiles * 4u), dim3(256), st, true, g, lay, ws);
    return hipGetLastError();
}

// ----------------------------------------------------------------------------
// Fused generation for N <= 128 (one B tile) with comparator streams: every A plane
// would be written once and read once, so the block builds its fp4 fragments in LDS
// straight from the int8 operands instead.  Block = 128 rows of A x 128 columns of B,
// four waves of 64 x 64 (2 x 2 MFMA blocks); a stage is 4 slots = 4 element quads of one
// octet, so one 8-cycle lookup table per operand serves the whole stage.  Thread tid < 128
// builds row tid of A, thread 128 + j builds row j of B: one 16-byte window of its int8
// row per stage (two aligned buffer loads, so rows need no alignment), 16 table lookups,
// the row-length mask and the sign, four 16-byte LDS stores.
// ----------------------------------------------------------------------------
constexpr int FWB = 128;                         // columns of B per fused block
constexpr int FBUF = MSTAGE * (BM + FWB);        // u4 per LDS stage buffer

struct FArgs {
    const int8_t *A, *B;
    int64_t lda, ldb, strideA, strideB;
    uint32_t bytesA, bytesB;    // extent of one batch entry of A / B from its first byte,
                                // rounded up to a whole dword
    int nbB, L_max;
};

// Stages per unit and the octet / first quad of a stage: stage index st of the tile covers
// slots 4 st .. 4 st + 3, all in octet (4 st) / KQP (KQP is a multiple of 4).
__device__ __forceinline__ void f_stage_pos(int st, int KQP, int &o, int &dq0) {
    const int ks = 4 * st;
    o = ks / KQP;
    dq0 = ks - o * KQP;
}

// the 20-byte aligned window holding bytes [off, off + 16) of the operand
struct FWin {
    u4 lo;
    uint32_t hi;
};
__device__ __forceinline__ void f_load(__amdgpu_buffer_rsrc_t rs, int off, FWin &w) {
    const int a0 = off & ~3;
    w.lo = __builtin_amdgcn_raw_buffer_load_b128(rs, a0, 0, 0);
    w.hi = __builtin_amdgcn_raw_buffer_load_b32(rs, a0 + 16, 0, 0);
}

// Table of octet o for both operands, indexed by the int8 value itself (as a byte):
// lut[side * 256 + byte] = the 8 nibbles of cycles 8o .. 8o + 7 (cycle c at bits 4c..4c+3),
// sign included (unipolar), so generating a slot row needs no boundary arithmetic
constexpr int FLUT = 512;
template <int POL>
__device__ __forceinline__ void f_build_lut(uint32_t *lut, const uint32_t *rA, const uint32_t *rB, int o,
                                            int tid) {
    const uint32_t zero_nib = POL == SC_BIPOLAR_XNOR ? NIB_NEG : 0u;
    for (int e = tid; e < FLUT; e += 256) {
        const int side = e >> 8;
        const int q = (int)(int8_t)(uint8_t)(e & 255);
        const uint32_t *r = (side ? rB : rA) + 8 * o;
        const uint32_t beta = (uint32_t)(POL == SC_BIPOLAR_XNOR ? beta_bipolar(q) : beta_unipolar(q));
        uint32_t x = 0;
#pragma unroll
        for (int c = 0; c < 8; ++c) x |= (r[c] < beta ? NIB_POS : zero_nib) << (4 * c);
        lut[e] = (POL == SC_UNIPOLAR_AND_SM && q < 0) ? negate_nibbles(x) : x;
    }
}

// the four slot rows of one stage for this thread's row, written into LDS at dst
// (slot k at dst + k * dstride); lut points at this operand's 256 entries
__device__ __forceinline__ void f_gen(const FWin &win, int sh, int elem0, int K, int Lr, bool rowok,
                                      int o, const uint32_t *lut, u4 *dst, int dstride) {
    // bytes [sh, sh + 16) of the window, four per dword
    uint32_t wd[4];
    const uint32_t v[5] = {win.lo[0], win.lo[1], win.lo[2], win.lo[3], win.hi};
#pragma unroll
    for (int k = 0; k < 4; ++k) wd[k] = __builtin_amdgcn_alignbyte(v[k + 1], v[k], (uint32_t)sh);
    // cycles at or beyond the row's length and padding rows give zero nibbles
    const int rem = Lr - MSTEP * o;
    const uint32_t lmask =
        (!rowok || rem <= 0) ? 0u : (rem >= 8 ? 0xFFFFFFFFu : (1u << (4 * rem)) - 1u);
    u4 out[4];
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
        for (int e = 0; e < 4; ++e) out[k][e] = lut[(wd[k] >> (8 * e)) & 255u] & lmask;
    // elements at or beyond K (only in a row's last quads; the same for every thread)
    if (elem0 + 16 > K) {
#pragma unroll
        for (int k = 0; k < 4; ++k)
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (elem0 + 4 * k + e >= K) out[k][e] = 0u;
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) dst[k * dstride] = out[k];
}

__device__ __forceinline__ int f_octet(int st, int KQP) { return (4 * st) / KQP; }

// window load of (unit-relative) stage st, clamped to the unit's last stage
__device__ __forceinline__ void f_load_stage(__amdgpu_buffer_rsrc_t rs, int rowoff, int st0, int st, int nst,
                                             int KQP, FWin &wv) {
    int o, dq0;
    f_stage_pos(st0 + min(st, nst - 1), KQP, o, dq0);
    f_load(rs, rowoff + 4 * dq0, wv);
}

struct FRow {
    int rowoff, Lr, lside;
    bool rowok;
    __amdgpu_buffer_rsrc_t rs;
    u4 *gdst0;
};

template <int POL>
__device__ __forceinline__ void f_gen_stage(const FRow &fr, const FWin &wv, int st0, int st, int KQP, int K,
                                            const uint32_t (*lut)[FLUT], u4 *dst) {
    if (!fr.rowok) {      // padding row (a whole wave of B rows when N <= 64): zero nibbles
#pragma unroll
        for (int k = 0; k < 4; ++k) dst[k * BM] = u4{0u, 0u, 0u, 0u};
        return;
    }
    int o, dq0;
    f_stage_pos(st0 + st, KQP, o, dq0);
    f_gen(wv, (fr.rowoff + 4 * dq0) & 3, 4 * dq0, K, fr.Lr, fr.rowok, o, &lut[o & 1][fr.lside], dst, BM);
}

// Stage st (parity P): MFMAs of stage st from buffer P, generation of stage st + 1 into
// buffer 1 - P from window 1 - P, which then loads stage st + 3; the table of stage st + 2
// is built first when that stage opens an octet (its parity differs from the table stage
// st + 1 uses, and the stages that last used it are finished).
template <int POL, int P>
__device__ __forceinline__ void f_stage(int st, int st0, int nst, const MGemmArgs &g, const FRow &fr,
                                        const uint32_t *rA, const uint32_t *rB, uint32_t (*lut)[FLUT],
                                        u4 *smem, int tid, int grp, int wr, int wc, int i32,
                                        v16f (&acc)[2][2], Frags<FWB> (&fg)[2], FWin (&win)[2]) {
    if (st + 2 < nst) {
        const int o2 = f_octet(st0 + st + 2, g.KQP);
        if (o2 != f_octet(st0 + st + 1, g.KQP)) f_build_lut<POL>(lut[o2 & 1], rA, rB, o2, tid);
    }
    const u4 *buf = smem + P * FBUF;
    read_frags<FWB>(buf, 1, grp, wr, wc, i32, fg[1]);
    mma<FWB>(acc, fg[0]);
    if (st + 1 < nst) {
        f_gen_stage<POL>(fr, win[1 - P], st0, st + 1, g.KQP, g.K, lut, fr.gdst0 + (1 - P) * FBUF);
        f_load_stage(fr.rs, fr.rowoff, st0, st + 3, nst, g.KQP, win[1 - P]);
    }
    mma<FWB>(acc, fg[1]);
    __syncthreads();
    if (st + 1 < nst) read_frags<FWB>(smem + (1 - P) * FBUF, 0, grp, wr, wc, i32, fg[0]);
}

template <int POL, bool SPLIT>
__global__ __launch_bounds__(256, 2) void k_fgemm(MGemmArgs g, FArgs f, Layout lay, uint8_t *ws) {
    constexpr bool BIP = POL == SC_BIPOLAR_XNOR;
    __shared__ u4 smem[2 * FBUF];
    __shared__ uint32_t lut[2][FLUT];            // [octet parity][side * 256 + byte]
    const int u = blockIdx.x;
    const int s = u % g.S;
    const int tile = u / g.S;                     // one B tile: tile = tm * batch + b
    const int b = tile % g.batch, tm = tile / g.batch;
    const int bB = f.nbB == 1 ? 0 : b;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int grp = lane >> 5, i32 = lane & 31;
    const int wr = (w >> 1) * 64, wc = (w & 1) * 64;
    uint8_t *wsa = ws + (size_t)b * lay.stride_batchA;
    const int Lloop = ws_ptr<int32_t>(wsa, lay.off_tileL)[tm];
    const int nstg = (Lloop / MSTEP) * (g.KQP / MSTAGE);
    const int st0 = (int)((int64_t)s * nstg / g.S), nst = (int)((int64_t)(s + 1) * nstg / g.S) - st0;
    const uint32_t *rA = ws_ptr<uint32_t>(ws, lay.off_rA), *rB = ws_ptr<uint32_t>(ws, lay.off_rB);

    // this thread's generation row: waves 0-1 rows of A (sorted order), waves 2-3 rows of B
    const bool isA = wave_uniform(tid >> 7) == 0;
    const int r = tid & (BM - 1);
    FRow fr;
    int row;
    if (isA) {
        const int p = tm * BM + r;
        row = ws_ptr<int32_t>(wsa, lay.off_perm)[p];
        fr.Lr = row >= 0 ? ws_ptr<int32_t>(wsa, lay.off_Ls)[p] : 0;
    } else {
        row = r < g.N ? r : -1;
        fr.Lr = f.L_max;
    }
    fr.rowok = row >= 0;
    const int8_t *base = isA ? f.A + (size_t)b * f.strideA : f.B + (size_t)bB * f.strideB;
    fr.rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<int8_t *>(base), 0, (int)(isA ? f.bytesA : f.bytesB),
                                              0x00020000);
    fr.rowoff = fr.rowok ? (int)((int64_t)row * (isA ? f.lda : f.ldb)) : 0;
    fr.lside = isA ? 0 : 256;
    fr.gdst0 = smem + (isA ? 0 : MSTAGE * BM) + r;

    v16f acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int c = 0; c < 2; ++c) acc[i][c] = v16f{};

    FWin win[2];
    Frags<FWB> fg[2];
    if (nst > 0) {
        f_load_stage(fr.rs, fr.rowoff, st0, 0, nst, g.KQP, win[0]);
        f_load_stage(fr.rs, fr.rowoff, st0, 1, nst, g.KQP, win[1]);
        const int o0 = f_octet(st0, g.KQP), o1 = f_octet(st0 + min(1, nst - 1), g.KQP);
        f_build_lut<POL>(lut[o0 & 1], rA, rB, o0, tid);
        if (o1 != o0) f_build_lut<POL>(lut[o1 & 1], rA, rB, o1, tid);
        __syncthreads();
        f_gen_stage<POL>(fr, win[0], st0, 0, g.KQP, g.K, lut, fr.gdst0);
        f_load_stage(fr.rs, fr.rowoff, st0, 2, nst, g.KQP, win[0]);
    }
    __syncthreads();
    if (nst > 0) read_frags<FWB>(smem, 0, grp, wr, wc, i32, fg[0]);
    for (int st = 0; st < nst; st += 2) {
        f_stage<POL, 0>(st, st0, nst, g, fr, rA, rB, lut, smem, tid, grp, wr, wc, i32, acc, fg, win);
        if (st + 1 < nst)
            f_stage<POL, 1>(st + 1, st0, nst, g, fr, rA, rB, lut, smem, tid, grp, wr, wc, i32, acc, fg, win);
    }

    if (SPLIT) {
        // partial sums of this split as int32 [tile][split][128][128], as the 128-row GEMM
        int32_t *part = ws_ptr<int32_t>(ws, lay.off_part) + ((size_t)tile * g.S + s) * BM * FWB;
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int c = 0; c < 2; ++c)
#pragma unroll
                for (int e = 0; e < 16; ++e)
                    part[(wr + 32 * i + 8 * (e >> 2) + 4 * grp + (e & 3)) * FWB + wc + 32 * c + i32] =
                        (int32_t)acc[i][c][e];
    } else {
        constexpr int TS = FWB + 4, TR = 32;
        static_assert(TR * TS * 4 <= 2 * FBUF * 16, "the epilogue transpose must fit the LDS buffers");
        int32_t *T = reinterpret_cast<int32_t *>(smem);
        for (int h = 0; h < BM / TR; ++h) {
            __syncthreads();
            if (wr == 64 * (h >> 1)) {
#pragma unroll
                for (int i = 0; i < 2; ++i) {
                    if (i != (h & 1)) continue;
#pragma unroll
                    for (int c = 0; c < 2; ++c)
#pragma unroll
                        for (int e = 0; e < 16; ++e)
                            T[(8 * (e >> 2) + 4 * grp + (e & 3)) * TS + wc + 32 * c + i32] = (int32_t)acc[i][c][e];
                }
            }
            __syncthreads();
            for (int k = 0; k < TR * (FWB / 4) / 256; ++k) {
                const int idx = tid + 256 * k;        // 32 rows x 32 column quads
                const int rl = idx / (FWB / 4), cq = idx % (FWB / 4);
                const int j0 = 4 * cq;
                if (j0 >= g.N) continue;
                const int4 v = *reinterpret_cast<const int4 *>(&T[rl * TS + 4 * cq]);
                const int32_t P[4] = {v.x, v.y, v.z, v.w};
                mdecode4<BIP>(P, tm * BM + TR * h + rl, j0, min(4, g.N - j0), b, g, lay, ws);
            }
        }
    }
}

template <int POL>
static hipError_t launch_fgemm_pol(const MGemmArgs &g, const FArgs &f, const Layout &lay, uint8_t *ws,
                                   hipStream_t st) {
    const unsigned tiles = (unsigned)(g.batch * lay.MT);
    if (g.S == 1) {
        gemm_launch((k_fgemm<POL, false>), dim3(tiles), dim3(256), st, true, g, f, lay, ws);
        return hipGetLastError();
    }
    gemm_launch((k_fgemm<POL, true>), dim3(tiles * (unsigned)g.S), dim3(256), st, false, g, f, lay, ws);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    gemm_launch((k_mgemm_reduce<POL == SC_BIPOLAR_XNOR, FWB>), dim3(tiles * 4u), dim3(256), st, true, g, lay,
                ws);
    return hipGetLastError();
}

// ----------------------------------------------------------------------------
// 256 x 256 GEMM tile: a pair of A row tiles (equal cycle counts) x a pair of B tiles,
// one 256-thread block per CU.  Wave w owns rows 128 (w / 2).., columns 128 (w % 2).. as
// 4 x 4 32x32 MFMA blocks (its 256 accumulator registers); per MFMA k-step it reads 8 KB
// of LDS for 16 MFMAs, two thirds of what the 128-row tile needs per product.  A stage
// is QSTAGE slots (two k-steps) in one of three LDS buffers: stage st computes from
// buffer st % 3 while stage st + 2 is written into the third buffer, so the first
// fragments of stage st + 1 can be read before the barrier that ends stage st; three
// register sets carry the global loads two stages ahead.
// ----------------------------------------------------------------------------
constexpr int QSTAGE = 4;                     // slots per stage
constexpr int QKS = QSTAGE / 2;               // MFMA k-steps per stage
constexpr int QBUF = QSTAGE * 512;            // u4 per LDS buffer: A [QSTAGE][256], B [QSTAGE][256]
constexpr int QNBUF = 3;

struct QRegs {
    u4 a[QSTAGE], b[QSTAGE];
};
struct QFrags {
    u4 a[4], b[4];
};

// Thread tid loads row tid % 128 of A tile tid / 128 of the pair (and the same of B) for
// each slot of the stage starting at slot ks, as buffer loads: one descriptor per wave
// spanning exactly its plane tile (a load past it would read zero), the slot as a scalar
// offset and the row as the one vector offset, so the loads need no 64-bit address
// arithmetic.  A short last stage re-reads its last slot (never used), so every load is in
// bounds.
struct QSrc {
    __amdgpu_buffer_rsrc_t a, b;   // this wave's A and B plane tiles
    int voff;                      // byte offset of the thread's row within a slot
};
__device__ __forceinline__ void q_load(const QSrc &q, int64_t ks, int64_t k1, QRegs &r) {
    const int last = (int)min((int64_t)QSTAGE, k1 - ks) - 1;
#pragma unroll
    for (int k = 0; k < QSTAGE; ++k)
        r.a[k] = __builtin_amdgcn_raw_buffer_load_b128(q.a, q.voff, (int)(ks + min(k, last)) * (BM * 16), 0);
#pragma unroll
    for (int k = 0; k < QSTAGE; ++k)
        r.b[k] = __builtin_amdgcn_raw_buffer_load_b128(q.b, q.voff, (int)(ks + min(k, last)) * (BN * 16), 0);
}

__device__ __forceinline__ void q_store(u4 *buf, int tid, const QRegs &r) {
#pragma unroll
    for (int k = 0; k < QSTAGE; ++k) buf[256 * k + tid] = r.a[k];
#pragma unroll
    for (int k = 0; k < QSTAGE; ++k) buf[QSTAGE * 256 + 256 * k + tid] = r.b[k];
}

// fragments of k-step j: A rows wr + 32i + l%32, B columns wc + 32c + l%32, slot 2j + l/32
__device__ __forceinline__ void q_frags(const u4 *buf, int j, int grp, int wr, int wc, int i32,
                                        QFrags &f) {
    const u4 *As = buf + (2 * j + grp) * 256, *Bs = buf + QSTAGE * 256 + (2 * j + grp) * 256;
#pragma unroll
    for (int i = 0; i < 4; ++i) f.a[i] = As[wr + 32 * i + i32];
#pragma unroll
    for (int c = 0; c < 4; ++c) f.b[c] = Bs[wc + 32 * c + i32];
}

__device__ __forceinline__ void q_mma(v16f (&acc)[4][4], const QFrags &f) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int c = 0; c < 4; ++c)
            acc[i][c] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(frag(f.a[i]), frag(f.b[c]),
                                                                        acc[i][c], 4, 4, 0, 127, 0, 127);
}

// Stage st, with CB = st % 3 the LDS buffer it computes from.  On entry the next buffer
// holds stage st + 1 (visible), fragment set 0 the first k-step of stage st, and the
// three register sets stages st + 2 (set (CB + 2) % 3, loaded two stages ago), st + 3
// (set CB, in flight) and nothing (set (CB + 1) % 3).  The stage loads stage st + 4 into
// the free set and writes stage st + 2 into the third buffer, so every load has two
// stages to arrive.  A FULL stage (both k-steps present: one branch-free region)
// interleaves its memory instructions one per MFMA: with one wave per SIMD the wave issues
// in order, and a burst of LDS or global instructions would hold back the next MFMA
// (measured on the 6304 x 768 x 3072 layer at L = 128: 1.20 ms unordered, 0.83 with one
// instruction per MFMA, 0.77 with the global loads spread over 16 MFMAs).
template <int CB, bool FULL>
__device__ __forceinline__ void q_stage(int st, int nst, int64_t k0, int64_t k1, const QSrc &q,
                                        u4 *smem, int tid, int grp, int wr, int wc,
                                        int i32, v16f (&acc)[4][4], QFrags (&f)[2], QRegs (&r)[3]) {
    constexpr int RL = (CB + 1) % 3, RW = (CB + 2) % 3, cb = CB;
    static_assert(QKS == 2, "the interleave below is written for two k-steps per stage");
    const int64_t klast = k0 + (int64_t)(nst - 1) * QSTAGE;
    const int64_t ks = k0 + (int64_t)st * QSTAGE;
    const int nb = cb == QNBUF - 1 ? 0 : cb + 1, wb = nb == QNBUF - 1 ? 0 : nb + 1;
    const u4 *buf = smem + cb * QBUF;
    u4 *wbuf = smem + wb * QBUF;
    const u4 *nbuf = smem + nb * QBUF;
    if (FULL) {
        q_frags(buf, 1, grp, wr, wc, i32, f[1]);
        q_load(q, min(ks + 4 * QSTAGE, klast), k1, r[RL]);
        q_mma(acc, f[0]);
        q_store(wbuf, tid, r[RW]);
        q_frags(nbuf, 0, grp, wr, wc, i32, f[0]);
        q_mma(acc, f[1]);
        // k-step 0: the reads of k-step 1's fragments, then global loads and LDS writes
        // alternating over the next 16 MFMAs; k-step 1 ends with the reads of the next
        // stage's first fragments
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // LDS read
        }
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);   // global load
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);   // LDS write
        }
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
    } else {
        const int nk = (int)min((int64_t)QSTAGE, k1 - ks) / 2;
        q_load(q, min(ks + 4 * QSTAGE, klast), k1, r[RL]);
        q_frags(buf, 1, grp, wr, wc, i32, f[1]);
        q_store(wbuf, tid, r[RW]);
        q_mma(acc, f[0]);
        q_frags(nbuf, 0, grp, wr, wc, i32, f[0]);
        if (nk > 1) q_mma(acc, f[1]);
    }
    __syncthreads();
}

// The division of the call's tiles into units: (F, S) from the host, or, when the host
// split every tile (F = 0), the split count chosen again with the longest tile pair the
// scheduler found (never above the host's, for which grid and partial sums are sized, nor
// below Smin, which keeps every part's sums exact).
__device__ __forceinline__ void q_division(const MGemmArgs &g, const Layout &lay, uint8_t *ws, int &F, int &S) {
    const int tiles = g.batch * (lay.MT / 2) * (lay.NT / 2);
    F = g.F;
    S = g.S;
    if (F == 0 && S > 1 && !lay.vsplit) {
        const double Lmax = (double)ws_ptr<uint32_t>(ws, lay.off_status)[1];
        double best = 0.0;
        for (int s = lay.Smin; s <= g.S; s *= 2) {
            const double est = quad_split_time(tiles, s, lay.q_perL, lay.q_Lmean, Lmax, lay.q_one != 0, lay.q_slots,
                                               lay.q_pbytes);
            if (s == lay.Smin || est < best * 0.97) {
                best = est;
                S = s;
            }
        }
        if (S == 1) F = tiles;
    }
}

// XCDs of the chip: the dispatcher hands workgroup u to XCD u % 8, and each XCD has its own L2
constexpr int NXCD = 8;
// pair rows per band in the order of the whole tiles
constexpr int QG = 4;

// The whole tile that unit u (< F) computes.  With one row length every tile is the same
// work, and units are regrouped so that the 8 C units that run at once on the 8 XCDs take
// 8 runs of C consecutive tiles, one run per XCD, and consecutive tiles go column by column
// through bands of QG pair rows: a run of 32 tiles covers 4 A pairs and 8 B pairs, which
// then hit in that XCD's L2.  Both steps are permutations of 0 .. F-1 (tiles past the last
// full run, or past the last full row of pair tiles, keep their place).  With varying
// lengths the tiles come longest first and unit u stays tile u: dealt round-robin over the
// XCDs, each XCD gets an even share of long and short tiles, where the runs above would
// give the first XCDs the longest pairs of every round (ViT-L/14 MLP fc1, lengths 8..512:
// 4.06 ms with the runs, 2.99 ms without).
__device__ __forceinline__ int q_whole_tile(int u, int F, int NTW, int one_length) {
    if (!one_length) return u;
    const int C = min(32, F / NXCD);
    if (C >= 2 && u < F / (NXCD * C) * (NXCD * C)) {
        const int j = u / NXCD, x = u % NXCD;
        u = ((j / C) * NXCD + x) * C + j % C;
    }
    const int R = F / NTW;
    if (u < R * NTW) {
        const int gb = u / (QG * NTW), idx = u % (QG * NTW);
        const int gs = min(QG, R - gb * QG);
        return (gb * QG + idx % gs) * NTW + idx / gs;
    }
    return u;
}

// Work unit u of the 256-row GEMM when every tile has one division (not vsplit): its tile,
// part s of S parts, and the partial index v of a split unit; false when u is past the call's
// units (the grid is sized for the most).  Units 0 .. F-1 are whole tiles (q_whole_tile),
// unit F + v part v % S of tile F + v / S.
__device__ __forceinline__ bool q_unit(const MGemmArgs &g, const Layout &lay, uint8_t *ws, int u, int &tile, int &s,
                                       int &S, int &v, bool &split) {
    const int NTW = lay.NT / 2;
    int F, SS;
    q_division(g, lay, ws, F, SS);
    if (u >= F + (g.batch * (lay.MT / 2) * NTW - F) * SS) return false;
    split = u >= F;
    v = u - F;
    s = split ? v % SS : 0;
    S = split ? SS : 1;
    tile = split ? F + v / SS : q_whole_tile(u, F, NTW, lay.q_one);
    return true;
}

// One work unit: tile `tile` (pair tp of batch entry b x B pair tw) over k-steps
// [s, s + 1) / S of the pair's k-steps.  Units 0 .. F-1 are the whole tiles 0 .. F-1,
// decoded here; unit F + v is part v % S of tile F + v / S, stored as a partial sum;
// units beyond those (a grid sized for a larger split) return at once.
template <bool BIP>
__global__ __launch_bounds__(256, 1) void k_qgemm(MGemmArgs g, Layout lay, uint8_t *ws) {
    static_assert(QKS % 2 == 0, "the fragment sets alternate within a stage");
    __shared__ u4 smem[QNBUF * QBUF];
    __shared__ DecodeLds dl;                          // filled after the k loop
    const int NTW = lay.NT / 2;
    int tile, s, S, v;
    bool split;
    if (!q_unit(g, lay, ws, blockIdx.x, tile, s, S, v, split)) return;
    const int tw = tile % NTW;
    const int tb = tile / NTW;
    const int b = tb % g.batch, tp = tb / g.batch;
    const int bB = g.nbB == 1 ? 0 : b;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int grp = lane >> 5, i32 = lane & 31;
    const int wr = (w >> 1) * 128, wc = (w & 1) * 128;
    uint8_t *wsa = ws + (size_t)b * lay.stride_batchA;
    uint8_t *wsbB = ws + (size_t)bB * lay.stride_batchB;
    const int Lloop = ws_ptr<int32_t>(wsa, lay.off_tileL)[2 * tp];
    const int64_t nsteps = (int64_t)(Lloop / MSTEP) * g.KQP / 2;
    const int64_t k0 = (int64_t)s * nsteps / S * 2, k1 = (int64_t)(s + 1) * nsteps / S * 2;
    const int half = wave_uniform(tid >> 7);
    const size_t btile = (size_t)(g.LBS / MSTEP) * g.KQP * BN;
    QSrc q;
    q.a = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint32_t *>(ws_ptr<uint32_t>(wsa, lay.off_Ap) + ws_ptr<int64_t>(wsa, lay.off_tileOff)[2 * tp + half]),
        0, (int)((Lloop / MSTEP) * g.KQP * BM * 16), 0x00020000);
    q.b = __builtin_amdgcn_make_buffer_rsrc(
        reinterpret_cast<u4 *>(ws_ptr<uint32_t>(wsbB, lay.off_Bp)) + (size_t)(2 * tw + half) * btile, 0,
        (int)(btile * 16), 0x00020000);
    q.voff = (tid & (BM - 1)) * 16;

    v16f acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[i][c] = v16f{};

    QRegs r[3];
    QFrags f[2];
    const int nst = (int)((k1 - k0 + QSTAGE - 1) / QSTAGE);
    if (nst > 0) {
        const int64_t klast = k0 + (int64_t)(nst - 1) * QSTAGE;
        q_load(q, k0, k1, r[0]);
        q_load(q, min(k0 + QSTAGE, klast), k1, r[1]);
        q_store(smem, tid, r[0]);
        q_store(smem + QBUF, tid, r[1]);
        q_load(q, min(k0 + 2 * QSTAGE, klast), k1, r[2]);
        q_load(q, min(k0 + 3 * QSTAGE, klast), k1, r[0]);
    }
    __syncthreads();
    if (nst > 0) q_frags(smem, 0, grp, wr, wc, i32, f[0]);
    // the first fragments complete before the loop, so that its first MFMAs need no wait
    __syncthreads();
    // triples of full stages (none is the last one), so that buffers and register sets are
    // fixed at compile time, then the last one to three stages: the loop body is
    // branch-free and its back edge always carries the same loads
    int st = 0;
    for (; st + 3 < nst; st += 3) {
        q_stage<0, true>(st, nst, k0, k1, q, smem, tid, grp, wr, wc, i32, acc, f, r);
        q_stage<1, true>(st + 1, nst, k0, k1, q, smem, tid, grp, wr, wc, i32, acc, f, r);
        q_stage<2, true>(st + 2, nst, k0, k1, q, smem, tid, grp, wr, wc, i32, acc, f, r);
    }
    if (st < nst) q_stage<0, false>(st, nst, k0, k1, q, smem, tid, grp, wr, wc, i32, acc, f, r);
    if (st + 1 < nst) q_stage<1, false>(st + 1, nst, k0, k1, q, smem, tid, grp, wr, wc, i32, acc, f, r);
    if (st + 2 < nst) q_stage<2, false>(st + 2, nst, k0, k1, q, smem, tid, grp, wr, wc, i32, acc, f, r);

    if (split) {
        // partial sums of this unit as int32 [256 rows][256 columns]
        store_part<4>(acc, ws_ptr<int32_t>(ws, lay.off_part) + (size_t)v * 256 * 256, wr, wc, lane);
    } else {
        // the rows' and columns' data staged in LDS, the sums transposed through LDS, 64 rows
        // at a time, so that each thread decodes four adjacent columns of one row
        d_stage<256>(dl, ws_ptr<int32_t>(wsa, lay.off_perm) + tp * 256, ws_ptr<int32_t>(wsa, lay.off_Ls) + tp * 256,
                     b, tw, g, tid);
        constexpr int TS = 256 + 4, TR = 64;
        static_assert(TR * TS * 4 <= QNBUF * QBUF * 16, "the epilogue transpose must fit the LDS buffers");
        float *T = reinterpret_cast<float *>(smem);
        for (int h = 0; h < 256 / TR; ++h) {
            __syncthreads();
            // rows 64h .. 64h + 63: MFMA blocks i = 2 (h % 2), 2 (h % 2) + 1 of the waves at wr = 128 (h / 2)
            if (wr == 128 * (h >> 1)) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    if ((i >> 1) != (h & 1)) continue;
#pragma unroll
                    for (int c = 0; c < 4; ++c)
#pragma unroll
                        for (int e = 0; e < 16; ++e)
                            T[(32 * (i & 1) + 8 * (e >> 2) + 4 * grp + (e & 3)) * TS + wc + 32 * c + i32] =
                                acc[i][c][e];
                }
            }
            __syncthreads();
            d_rows<BIP, 256, 64, TR, TS>(dl, T, TR * h, tw, b, g, tid);
        }
    }
}

// Sums the partial counts of every piece of the split tiles F.. and decodes.  Pieces are in
// the MFMA layout (store_block), PC columns wide; a thread takes NK quads of it, each four
// rows of one column, and a block of 256 threads 256 NK quads (BPT blocks per tile).  Few
// quads per thread when few tiles are split, so that enough waves keep loads in flight; more
// when many are (less per-block overhead).  With vsplit, tinfo gives each tile's pieces
// (tiles that ran whole have none).  P16: the pieces hold int16 counts (Layout::p16).
template <bool P16>
struct PQuad;
template <>
struct PQuad<false> {
    typedef int4 T;
    static __device__ __forceinline__ int4 get(const int4 &x) { return x; }
};
template <>
struct PQuad<true> {
    typedef int2 T;
    static __device__ __forceinline__ int4 get(const int2 &x) {
        return make_int4((int)(int16_t)(x.x & 0xFFFF), x.x >> 16, (int)(int16_t)(x.y & 0xFFFF), x.y >> 16);
    }
};
template <bool BIP, int NK, int PC, bool P16>
__global__ __launch_bounds__(256) void k_qgemm_reduce(MGemmArgs g, Layout lay, uint8_t *ws) {
    constexpr int QPT = 256 * PC / 4;         // quads per tile
    constexpr int BPT = QPT / (256 * NK);     // blocks per tile
    constexpr int CB = PC / 32;               // 32-column blocks of a piece
    constexpr int RPB = 32 * ((NK + CB - 1) / CB);   // rows a block's NK MFMA blocks span
    static_assert(RPB <= 256, "rows of a block");
    __shared__ int32_t srow[RPB], slen[RPB];
    __shared__ float sfac[RPB];
    const int NTW = lay.NT / 2;
    int F, SS;
    q_division(g, lay, ws, F, SS);
    const int tile = F + (int)(blockIdx.x / BPT), part = (int)(blockIdx.x % BPT);
    if (tile >= g.batch * (lay.MT / 2) * NTW) return;
    size_t pbase = (size_t)(tile - F) * SS;
    if (lay.vsplit) {
        const int2 ti = ws_ptr<int2>(ws, lay.off_tinfo)[tile];
        if (ti.x < 2) return;
        SS = ti.x;
        pbase = (size_t)ti.y;
    }
    const int tw = tile % NTW;
    const int tb = tile / NTW;
    const int b = tb % g.batch, tp = tb / g.batch;
    typedef typename PQuad<P16>::T Q;
    const Q *base = reinterpret_cast<const Q *>(ws_ptr<uint8_t>(ws, lay.off_part)) + pbase * QPT +
                    (size_t)part * 256 * NK + threadIdx.x;
    // the first pieces' loads go out before the block stages its rows' decode data
    constexpr int SB = NK <= 2 ? MAX_SPLIT : (NK <= 4 ? 2 : 1);
    Q q[SB][NK];
#pragma unroll
    for (int s = 0; s < SB; ++s)
#pragma unroll
        for (int k = 0; k < NK; ++k)
            q[s][k] = s < SS ? base[(size_t)s * QPT + 256 * k] : Q{};
    // the block's rows rbase .. rbase + RPB - 1 of the pair: original row (-1: padding),
    // length, decode factor
    const int rbase = (part * NK / CB) * 32;
    uint8_t *wsa = ws + (size_t)b * lay.stride_batchA;
    if ((int)threadIdx.x < RPB) {
        const int r = rbase + (int)threadIdx.x;
        const int i = ws_ptr<int32_t>(wsa, lay.off_perm)[tp * 256 + r];
        const int Li = i >= 0 ? ws_ptr<int32_t>(wsa, lay.off_Ls)[tp * 256 + r] : 0;
        srow[threadIdx.x] = i;
        slen[threadIdx.x] = Li;
        sfac[threadIdx.x] = i >= 0 ? decode_factor(g.sA[(size_t)b * g.strideSA + i], Li) : 0.0f;
    }
    int4 sum[NK];
#pragma unroll
    for (int k = 0; k < NK; ++k) sum[k] = make_int4(0, 0, 0, 0);
    for (int s0 = 0; s0 < SS; s0 += SB) {
        if (s0 > 0) {
#pragma unroll
            for (int s = 0; s < SB; ++s)
#pragma unroll
                for (int k = 0; k < NK; ++k)
                    q[s][k] = s0 + s < SS ? base[(size_t)(s0 + s) * QPT + 256 * k] : Q{};
        }
#pragma unroll
        for (int s = 0; s < SB; ++s)
#pragma unroll
            for (int k = 0; k < NK; ++k) {
                const int4 t = PQuad<P16>::get(q[s][k]);
                sum[k].x += t.x;
                sum[k].y += t.y;
                sum[k].z += t.z;
                sum[k].w += t.w;
            }
    }
    __syncthreads();
    const float *sBb = g.sB + (size_t)b * g.strideSB;
    const int lane = threadIdx.x & 63, grp = lane >> 5, i32 = lane & 31;
#pragma unroll
    for (int k = 0; k < NK; ++k) {
        const int qd = (part * 256 * NK + 256 * k + (int)threadIdx.x) >> 6;   // quad index of the wave
        const int blk = qd >> 2, qq = qd & 3;
        const int rl = (blk / CB) * 32 + 8 * qq + 4 * grp - rbase;   // first of its 4 rows, in the block
        const int j = tw * 256 + (blk % CB) * 32 + i32;
        if (j >= g.N) continue;
        const float sBj = sBb[j];
        const int32_t P[4] = {sum[k].x, sum[k].y, sum[k].z, sum[k].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int i = srow[rl + e];
            if (i < 0) continue;
            const int Li = slen[rl + e];
            const size_t off = (size_t)b * g.strideO + (size_t)i * g.ldo + j;
            g.out[off] = ((float)P[e] * sfac[rl + e]) * sBj;
            if (g.counts) g.counts[off] = Li > 0 ? (BIP ? (g.K * Li + P[e]) / 2 : P[e]) : 0;
        }
    }
}

template <bool BIP, bool P16>
static void launch_qreduce_p(const MGemmArgs &g, const Layout &lay, uint8_t *ws, unsigned tail, hipStream_t st) {
    if (lay.pcols == 64) {
        if (tail * 16u < 1024u)
            gemm_launch((k_qgemm_reduce<BIP, 1, 64, P16>), dim3(tail * 16u), dim3(256), st, true, g, lay, ws);
        else
            gemm_launch((k_qgemm_reduce<BIP, 4, 64, P16>), dim3(tail * 4u), dim3(256), st, true, g, lay, ws);
    } else {
        if (tail * 8u < 1024u)
            gemm_launch((k_qgemm_reduce<BIP, 2, 256, P16>), dim3(tail * 32u), dim3(256), st, true, g, lay, ws);
        else
            gemm_launch((k_qgemm_reduce<BIP, 8, 256, P16>), dim3(tail * 8u), dim3(256), st, true, g, lay, ws);
    }
}
template <bool BIP>
static hipError_t launch_qreduce(const MGemmArgs &g, const Layout &lay, uint8_t *ws, unsigned tail, hipStream_t st) {
    if (lay.p16) launch_qreduce_p<BIP, true>(g, lay, ws, tail, st);
    else launch_qreduce_p<BIP, false>(g, lay, ws, tail, st);
    return hipGetLastError();
}

template <bool BIP>
static hipError_t launch_qgemm(const MGemmArgs &g, const Layout &lay, uint8_t *ws, hipStream_t st) {
    const unsigned tiles = (unsigned)(g.batch * (lay.MT / 2) * (lay.NT / 2));
    const unsigned tail = tiles - (unsigned)g.F;
    gemm_launch((k_qgemm<BIP>), dim3((unsigned)g.F + tail * (unsigned)g.S), dim3(256), st, tail == 0, g, lay,
                ws);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || tail == 0) return e;
    return launch_qreduce<BIP>(g, lay, ws, tail, st);
}

// ----------------------------------------------------------------------------
// 256 x 256 GEMM with fragments built from int8 chunks (comparator streams)
// ----------------------------------------------------------------------------
// One comparator sequence per operand makes the 32 stream bits of an element over the
// cycles 32G .. 32G + 31 a function of its int8 value alone: one 16-byte fp4 slot row.  The
// GEMM keeps that table for its current cycle group G in LDS and builds every MFMA
// fragment with one table read indexed by the element's byte, so the operands stream in
// as bytes (k_rchunks lays them out) instead of as fp4 planes 8 L times their size.
// Slot rows: a k-step takes one element per lane half (lanes 0-31 the elements 0..15 of
// their row's chunk, lanes 32-63 the elements 16..31, one element per k-step) over the 32
// cycles of the group; both operands use the same order, so the k-step sums the products
// of matching elements and cycles.
constexpr int RCH = 32;          // elements per chunk, cycles per group
constexpr int RREP = 8;          // copies of each table entry (16-byte reads spread over the banks)
constexpr int RPAD = 0x80;       // chunk byte of a padding element or row: the table gives zero
constexpr int RREP1 = 4;         // copies of each masked table entry
constexpr int RGROUPS = SC_L_MAX_LIMIT / RCH;
static_assert(RSLOTS * RREP1 == 16, "the masked tables fill one 256-byte row per byte value");

// bytes equal to 0x80 (-128) become 0x81 (-127): same comparator boundaries, and 0x80 stays
// free to mark padding
__device__ __forceinline__ uint32_t r_clamp4(uint32_t x) {
    const uint32_t t = x ^ 0x80808080u;                                      // 0 where x was 0x80
    const uint32_t nz = (((t & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | t) & 0x80808080u;  // 0x80 where t != 0
    return x | ((~nz & 0x80808080u) >> 7);
}

// Entry (byte, operand) of the table of cycle group G: the 32 nibbles of cycles 32G .. 32G+31
// (cycle 32G + k at bits 4 (k % 8) of dword k / 8), sign folded in (unipolar), zero for the
// padding byte; r points at the operand's draw of cycle 32G.  The tables of every group are
// built once per call (k_rchunks) into the workspace, [G][operand][byte].
template <bool BIP>
__device__ __forceinline__ u4 r_entry(const uint32_t *r, int byte) {
    u4 x = u4{0u, 0u, 0u, 0u};
    if (byte == RPAD) return x;
    const uint32_t zero_nib = BIP ? NIB_NEG : 0u;
    const int q = (int)(int8_t)(uint8_t)byte;
    const uint32_t beta = (uint32_t)(BIP ? beta_bipolar(q) : beta_unipolar(q));
#pragma unroll
    for (int dw = 0; dw < 4; ++dw) {
        uint32_t w = 0;
#pragma unroll
        for (int c = 0; c < 8; ++c) w |= (r[8 * dw + c] < beta ? NIB_POS : zero_nib) << (4 * c);
        x[dw] = (!BIP && q < 0) ? negate_nibbles(w) : w;
    }
    return x;
}

struct RChunkArgs {
    const int8_t *X[2];
    int64_t ld[2], strideX[2];
    int rows[2], rows_pad[2], nb[2];
    size_t stride_batch[2], off_out[2];
    size_t off_perm;      // side 0 (A) takes its rows in the scheduler's order
    int K, KC;
    int vec[2];           // 16-byte loads are aligned (base and row stride multiples of 16)
    int groups, bip;      // tables: 32-cycle groups, polarity
    size_t off_r[2], off_rtab;
};

// One 16-byte half of a chunk: bytes d0 .. d0 + 15 of row xrow (K bytes; null: a padding
// row), clamped to [-127, 127], 0x80 past K.
__device__ __forceinline__ u4 r_half(const int8_t *xrow, int d0, int K, bool vec) {
    u4 v = u4{0x80808080u, 0x80808080u, 0x80808080u, 0x80808080u};
    if (xrow == nullptr || d0 >= K) return v;
    if (vec && d0 + 16 <= K) {
        v = *reinterpret_cast<const u4 *>(xrow + d0);
    } else {
        // any byte alignment: the two aligned 16-byte blocks that cover the 16 bytes, each
        // loaded only when it holds a byte of the row before K (an aligned block never crosses
        // a page, so it is readable when one of its bytes is; the first always holds byte d0),
        // then shifted into place; bytes at or past K are replaced below
        const uintptr_t p = reinterpret_cast<uintptr_t>(xrow + d0);
        const uintptr_t end = reinterpret_cast<uintptr_t>(xrow + K);
        const u4 *w = reinterpret_cast<const u4 *>(p & ~(uintptr_t)15);
        const u4 lo = w[0];
        const u4 hi = reinterpret_cast<uintptr_t>(w + 1) < end ? w[1] : v;   // (v: padding bytes)
        const uint32_t t[8] = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        const uint32_t q = (uint32_t)(p >> 2) & 3u, sh = (uint32_t)(p & 3);
        // dwords q .. q + 4 of t, picked with selects (q differs between the rows of a wave)
        uint32_t wv[5];
#pragma unroll
        for (int k = 0; k < 5; ++k)
            wv[k] = q == 0 ? t[k] : q == 1 ? t[k + 1] : q == 2 ? t[k + 2] : t[k + 3];
#pragma unroll
        for (int k = 0; k < 4; ++k) v[k] = __builtin_amdgcn_alignbyte(wv[k + 1], wv[k], sh);
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = r_clamp4(v[k]);
    if (d0 + 16 > K) {          // the elements past K keep the padding byte
#pragma unroll
        for (int k = 0; k < 4; ++k)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (d0 + 4 * k + j >= K) v[k] = (v[k] & ~(0xFFu << (8 * j))) | ((uint32_t)RPAD << (8 * j));
    }
    return v;
}

// Chunks of both operands, through LDS: a block takes 64 rows (of the tile order) x 8 chunks
// (256 bytes of each row).  It reads them row by row, 16 lanes per row (coalesced along the
// row), into LDS as [chunk][row][half], then writes each chunk's 64 rows x 32 bytes, which are
// contiguous in the chunk layout.  Side and batch entry from blockIdx.z.
constexpr int RC_ROWS = 64, RC_CH = 8;
constexpr int RC_CSTRIDE = RC_ROWS * 2 + 1;      // u4 per chunk in LDS (+1: banks shift by chunk)
__global__ __launch_bounds__(256) void k_rchunks(RChunkArgs a, uint8_t *ws) {
    if (blockIdx.z == (unsigned)(a.nb[0] + a.nb[1])) {
        // the last slice of the grid builds the tables of every cycle group
        u4 *tab = ws_ptr<u4>(ws, a.off_rtab);
        const int nblk = gridDim.x * gridDim.y;
        for (int e = (blockIdx.y * gridDim.x + blockIdx.x) * 256 + threadIdx.x; e < a.groups * 512; e += nblk * 256) {
            const int G = e >> 9, side = (e >> 8) & 1, byte = e & 255;
            const uint32_t *r = ws_ptr<uint32_t>(ws, a.off_r[side]) + RCH * G;
            tab[e] = a.bip ? r_entry<true>(r, byte) : r_entry<false>(r, byte);
        }
        return;
    }
    __shared__ u4 sm[RC_CH * RC_CSTRIDE];
    const int side = blockIdx.z >= (unsigned)a.nb[0];
    const int b = side ? blockIdx.z - a.nb[0] : blockIdx.z;
    const int r0 = blockIdx.x * RC_ROWS, c0 = blockIdx.y * RC_CH;
    if (r0 >= a.rows_pad[side]) return;                 // (uniform over the block)
    const int nc = min(RC_CH, a.KC - c0);
    uint8_t *wsb = ws + (size_t)b * a.stride_batch[side];
    const int tid = threadIdx.x, hl = tid & 15;         // hl = 2 * chunk + half
    const bool vec = a.vec[side] != 0;
    for (int pass = 0; pass < RC_ROWS / 16; ++pass) {
        const int rl = pass * 16 + (tid >> 4), r = r0 + rl;
        if ((hl >> 1) >= nc) continue;
        const int src = side == 0 ? ws_ptr<int32_t>(wsb, a.off_perm)[r] : (r < a.rows[side] ? r : -1);
        const int8_t *xrow = src >= 0 ? a.X[side] + (size_t)b * a.strideX[side] + (size_t)src * a.ld[side] : nullptr;
        sm[(hl >> 1) * RC_CSTRIDE + rl * 2 + (hl & 1)] = r_half(xrow, (c0 + (hl >> 1)) * RCH + 16 * (hl & 1), a.K, vec);
    }
    __syncthreads();
    u4 *out = reinterpret_cast<u4 *>(ws_ptr<uint8_t>(wsb, a.off_out[side])) + (size_t)(r0 >> 8) * a.KC * 512 +
              (r0 & 255) * 2;
    for (int k = tid; k < nc * RC_ROWS * 2; k += 256) {
        const int c = k / (RC_ROWS * 2), e = k % (RC_ROWS * 2);
        out[(size_t)(c0 + c) * 512 + e] = sm[c * RC_CSTRIDE + e];
    }
}

hipError_t launch_rchunks(const sc_gemm_desc &d, const Layout &lay, const int8_t *A, const int8_t *B,
                          uint8_t *ws, hipStream_t st) {
    if (lay.KC == 0) return hipSuccess;       // no chunk and no table is read
    RChunkArgs a{};
    a.X[0] = A;
    a.X[1] = B;
    a.ld[0] = d.lda;
    a.ld[1] = d.ldb;
    a.strideX[0] = d.strideA;
    a.strideX[1] = d.strideB;
    a.rows[0] = d.M;
    a.rows[1] = d.N;
    a.rows_pad[0] = lay.MT * BM;
    // the 256 x 64 blocks read the first 64 rows of B's pair only
    a.rows_pad[1] = lay.narrow ? 64 : lay.NT * BN;
    a.nb[0] = d.batch;
    a.nb[1] = lay.nbB;
    a.stride_batch[0] = lay.stride_batchA;
    a.stride_batch[1] = lay.stride_batchB;
    a.off_out[0] = lay.off_Ap;
    a.off_out[1] = lay.off_Bp;
    a.off_perm = lay.off_perm;
    a.K = d.K;
    a.KC = lay.KC;
    a.vec[0] = (reinterpret_cast<uintptr_t>(A) % 16 == 0) && d.lda % 16 == 0 && d.strideA % 16 == 0;
    a.vec[1] = (reinterpret_cast<uintptr_t>(B) % 16 == 0) && d.ldb % 16 == 0 && d.strideB % 16 == 0;
    a.groups = lay.LBS / RCH;
    a.bip = d.polarity == SC_BIPOLAR_XNOR;
    a.off_r[0] = lay.off_rA;
    a.off_r[1] = lay.off_rB;
    a.off_rtab = lay.off_rtab;
    const int rows = a.rows_pad[0] > a.rows_pad[1] ? a.rows_pad[0] : a.rows_pad[1];
    hipLaunchKernelGGL(k_rchunks, dim3((unsigned)((rows + RC_ROWS - 1) / RC_ROWS), (unsigned)((lay.KC + RC_CH - 1) / RC_CH),
                                       (unsigned)(d.batch + lay.nbB + 1)),
                       dim3(256), 0, st, a, ws);
    return hipGetLastError();
}

// the nibbles of cycles 32G .. 32G+31 that lie below a row length L (cycle order as in the table)
__device__ __forceinline__ u4 r_len_mask(int L, int G) {
    const int rem = L - RCH * G;
    u4 m;
#pragma unroll
    for (int dw = 0; dw < 4; ++dw) {
        const int n = rem - 8 * dw;
        m[dw] = n >= 8 ? 0xFFFFFFFFu : (n <= 0 ? 0u : (1u << (4 * n)) - 1u);
    }
    return m;
}

// Entries of one group's table held by a thread: of the group's 512 (A's 256 bytes, then B's),
// entry k NT + tid, i.e. bytes tid, tid + NT, .. of A, then the same bytes of B.
template <int NT>
__device__ __forceinline__ void r_load_ent(u4 (&ent)[512 / NT], const u4 *tab, int tid) {
#pragma unroll
    for (int k = 0; k < 512 / NT; ++k) ent[k] = tab[k * NT + tid];
}

// The LDS table of one group from the thread's entries (r_load_ent): copies laid out
// [byte][operand][copy], so a read's byte address is byte * 256 + operand * 128 + copy * 16.
// A second region (from byte 65536) holds, for the k-th length set in `rems` (bit r: a row of
// the pair ends r cycles into the group), A's entries masked to that length: [byte][k][copy],
// address 65536 + byte * 256 + (k * RREP1 + copy) * 16.  Each store instruction rotates the
// copy by the lane, so that a wave's 64 lanes spread over 8 (masked: 4) 16-byte columns of the
// 256-byte rows instead of all falling into one.
template <int NT>
__device__ __forceinline__ void r_fill_lut(u4 *lut, const u4 (&ent)[512 / NT], int tid, uint32_t rems) {
    constexpr int BPT = 256 / NT;     // bytes per thread
    const int lane = tid & 63;
#pragma unroll
    for (int i = 0; i < BPT; ++i) {
        u4 *row = lut + (i * NT + tid) * 16;
#pragma unroll
        for (int j = 0; j < RREP; ++j) {
            const int c = (j + lane) & (RREP - 1);
            row[c] = ent[i];
            row[RREP + c] = ent[BPT + i];
        }
        int k = 0;
        for (uint32_t m = rems; m != 0u; m &= m - 1u, ++k) {
            const u4 xm = ent[i] & r_len_mask(__builtin_ctz(m), 0);
#pragma unroll
            for (int j = 0; j < RREP1; ++j) row[256 * 16 + k * RREP1 + ((j + lane) & (RREP1 - 1))] = xm;
        }
    }
}

// NB: B blocks of 32 columns per wave.  NB = 4: a wave takes 128 x 128 and every k-step
// of a chunk (16 elements of each of its lane's rows).  NB = 2 (N <= 64): a wave takes
// 128 x 64 and half of each chunk's k-steps (8 elements of each row), two waves sharing the
// rows, so that a SIMD runs two waves and one wave's waits overlap the other's MFMAs.
template <int NB>
struct RShape;
template <>
struct RShape<4> {
    typedef u4 V;
    static constexpr int KS = 16;   // k-steps per chunk per wave
};
template <>
struct RShape<2> {
    typedef u2 V;
    static constexpr int KS = 8;
};
template <int NB>
struct RData {
    typename RShape<NB>::V a[4], b[NB];   // the chunk's elements of the lane's 4 A rows and NB B columns
};
template <int NB>
struct RFrags {
    u4 a[4], b[NB];
};
struct RSrc {
    __amdgpu_buffer_rsrc_t a, b;   // the pair's A chunks and the B pair's chunks
    int voffA, voffB;              // the lane's row and half within a chunk
    int boffA[4];                  // byte offsets of the wave's four A blocks within a chunk
    uint32_t loA[4], loB;          // table rows of the lane's A rows (copy, region) and of B
    const char *lut;
    int KC;
};

// The 32-row blocks of a 256-row pair that row-half rh of the block computes: {0, 1, 6, 7}
// and {2, 3, 4, 5}.  Rows are sorted by length, so each half holds long and short rows
// alike, and the second two blocks of a half end no later than its first two: once they
// have ended, the half runs the MFMAs of its first two blocks only (Sec. 4.2: row i stops
// after its l_i cycles; Sec. 4.1: the cost follows the sum of the l_i).
__device__ __forceinline__ int r_block(int rh, int i) { return rh == 0 ? (i < 2 ? i : i + 4) : i + 2; }

// First row (within the pair) of the wave's block i: interleaved as above when the wave skips
// ended blocks (SKIP), else row half rh's four consecutive blocks.  SKIP is taken by the
// 256 x 64 blocks (N <= 64): there the rows of a pair vary the most in length (attention
// rows, padded heads).  The 256 x 256 blocks keep consecutive blocks: on the MLP layers the
// skip saved under 3 % of the MFMAs and its second loop cost more (5 % on ViT-B fc1).
template <bool SKIP>
__device__ __forceinline__ int r_row0(int rh, int i) { return SKIP ? 32 * r_block(rh, i) : 128 * rh + 32 * i; }

template <int NB>
__device__ __forceinline__ void r_load(const RSrc &q, int c, RData<NB> &d) {
    if constexpr (NB == 2) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
            d.a[i] = __builtin_amdgcn_raw_buffer_load_b64(q.a, q.voffA, c * 256 * RCH + q.boffA[i], 0);
#pragma unroll
        for (int i = 0; i < NB; ++i)
            d.b[i] = __builtin_amdgcn_raw_buffer_load_b64(q.b, q.voffB, c * 256 * RCH + i * 32 * RCH, 0);
    } else {
#pragma unroll
        for (int i = 0; i < 4; ++i)
            d.a[i] = __builtin_amdgcn_raw_buffer_load_b128(q.a, q.voffA, c * 256 * RCH + q.boffA[i], 0);
#pragma unroll
        for (int i = 0; i < NB; ++i)
            d.b[i] = __builtin_amdgcn_raw_buffer_load_b128(q.b, q.voffB, c * 256 * RCH + i * 32 * RCH, 0);
    }
}

// rows that have ended before this cycle group read the padding byte, whose table row is zero
template <int NB>
__device__ __forceinline__ void r_finish(RData<NB> &d, const bool (&fin)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
        if (fin[i]) d.a[i] = 0x80808080u;
}

// the table row of element E of the lane's elements (0..15, or 0..7 with NB = 2): address
// byte 1 = the element's byte, bytes 0 and 2 = the copy and the region (from lo)
template <int E>
__device__ __forceinline__ u4 r_look(const RSrc &q, uint32_t word, uint32_t lo) {
    constexpr uint32_t sel = 0x0C020000u | ((4u + (E & 3)) << 8);
    return *reinterpret_cast<const u4 *>(q.lut + __builtin_amdgcn_perm(word, lo, sel));
}
template <int E, typename V>
__device__ __forceinline__ uint32_t r_word(const V &v) {
    return v[E >> 2];
}

// the MFMAs of A blocks 2h, 2h + 1 with every B block
template <int NB>
__device__ __forceinline__ void q_mma_half(v16f (&acc)[4][NB], const RFrags<NB> &f, int h) {
#pragma unroll
    for (int i = 2 * h; i < 2 * h + 2; ++i)
#pragma unroll
        for (int c = 0; c < NB; ++c)
            acc[i][c] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(frag(f.a[i]), frag(f.b[c]),
                                                                        acc[i][c], 4, 4, 0, 127, 0, 127);
}

// the MFMAs of the first A block only (its B blocks)
template <int NB>
__device__ __forceinline__ void q_mma_one(v16f (&acc)[4][NB], const RFrags<NB> &f) {
#pragma unroll
    for (int c = 0; c < NB; ++c)
        acc[0][c] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(frag(f.a[0]), frag(f.b[c]), acc[0][c], 4, 4, 0,
                                                                    127, 0, 127);
}

// fragments of k-step E (element E of the lane's 16) from chunk data d
template <int E, bool MASK, int NB>
__device__ __forceinline__ void r_frags(const RSrc &q, const RData<NB> &d, const u4 (&m)[4], RFrags<NB> &f) {
#pragma unroll
    for (int c = 0; c < NB; ++c) f.b[c] = r_look<E>(q, r_word<E>(d.b[c]), q.loB);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        f.a[i] = r_look<E>(q, r_word<E>(d.a[i]), q.loA[i]);
        if (MASK) f.a[i] &= m[i];
    }
}

// fragments of k-step E for the first two A blocks only (the other two have ended)
template <int E, bool MASK, int NB>
__device__ __forceinline__ void r_frags_h(const RSrc &q, const RData<NB> &d, const u4 (&m)[4], RFrags<NB> &f) {
#pragma unroll
    for (int c = 0; c < NB; ++c) f.b[c] = r_look<E>(q, r_word<E>(d.b[c]), q.loB);
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        f.a[i] = r_look<E>(q, r_word<E>(d.a[i]), q.loA[i]);
        if (MASK) f.a[i] &= m[i];
    }
}

// fragments of k-step E for the first A block only (the wave's other three have ended)
template <int E, bool MASK, int NB>
__device__ __forceinline__ void r_frags_q(const RSrc &q, const RData<NB> &d, const u4 (&m)[4], RFrags<NB> &f) {
#pragma unroll
    for (int c = 0; c < NB; ++c) f.b[c] = r_look<E>(q, r_word<E>(d.b[c]), q.loB);
    f.a[0] = r_look<E>(q, r_word<E>(d.a[0]), q.loA[0]);
    if (MASK) f.a[0] &= m[0];
}

// Stage S (k-steps 2S, 2S+1) of a chunk: fragment set 0 holds k-step 2S on entry and the
// next k-step (2S + 2, or the next chunk's first) on exit; stage 0 loads the next chunk.
// A chunk has KS / 2 stages (RShape).
// MASK: the A fragments are masked with the rows' lengths (some row of the pair ends
// inside a cycle group); else rows that have ended read the padding byte (r_finish).
template <int NB>
__device__ __forceinline__ void r_mask(const u4 (&m)[4], RFrags<NB> &f) {
#pragma unroll
    for (int i = 0; i < 4; ++i) f.a[i] &= m[i];
}

// a quarter holds 2 NB MFMAs (A blocks 2h, 2h + 1 with every B block)
template <bool LOADS, int NB>
__device__ __forceinline__ void r_quarter_reads() {
    // the 4 + NB table reads of the next fragments with their address bytes
#pragma unroll
    for (int k = 0; k < 2 * NB; ++k) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
        __builtin_amdgcn_sched_group_barrier(0x002, 1, 0);   // VALU (address)
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // LDS read
        if (LOADS) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);   // global load
    }
    __builtin_amdgcn_sched_barrier(0);
}
template <bool MASK, int NB>
__device__ __forceinline__ void r_quarter_masks() {
#pragma unroll
    for (int k = 0; k < 2 * NB; ++k) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        if (MASK) __builtin_amdgcn_sched_group_barrier(0x002, 16 / (2 * NB), 0);   // masks
    }
    __builtin_amdgcn_sched_barrier(0);
}

// Stage S in four quarters of 8 MFMAs: the table reads of the next fragments go with the
// first quarter of each k-step, their length masks (MASK) with the second, once the reads
// have landed, so no AND waits on a read in the in-order issue
template <int S, bool MASK, int NB>
__device__ __forceinline__ void r_stage(const RSrc &q, int cnext, RData<NB> &cur, RData<NB> &nxt,
                                        const u4 (&m)[4], const bool (&fin)[4], v16f (&acc)[4][NB],
                                        RFrags<NB> (&f)[2]) {
    if (S == 0) r_load(q, cnext, nxt);
    r_frags<2 * S + 1, false>(q, cur, m, f[1]);
    q_mma_half(acc, f[0], 0);
    r_quarter_reads<S == 0, NB>();
    if (MASK) r_mask(m, f[1]);
    q_mma_half(acc, f[0], 1);
    r_quarter_masks<MASK, NB>();
    if (S < RShape<NB>::KS / 2 - 1) {
        r_frags<2 * S + 2, false>(q, cur, m, f[0]);
    } else {
        if (!MASK) r_finish(nxt, fin);
        r_frags<0, false>(q, nxt, m, f[0]);
    }
    q_mma_half(acc, f[1], 0);
    r_quarter_reads<false, NB>();
    if (MASK) r_mask(m, f[0]);
    q_mma_half(acc, f[1], 1);
    r_quarter_masks<MASK, NB>();
}

// Stage S when only the first two A blocks of the wave run: half the MFMAs, two A table
// reads per k-step instead of four.  The reads of the next fragments go with the k-step's
// MFMAs and their length masks (MASK) after them, right before the MFMAs that use them.
template <int NB>
__device__ __forceinline__ void r_mask_h(const u4 (&m)[4], RFrags<NB> &f) {
#pragma unroll
    for (int i = 0; i < 2; ++i) f.a[i] &= m[i];
}
template <int S, bool MASK, int NB>
__device__ __forceinline__ void r_stage_h(const RSrc &q, int cnext, RData<NB> &cur, RData<NB> &nxt,
                                          const u4 (&m)[4], const bool (&fin)[4], v16f (&acc)[4][NB],
                                          RFrags<NB> (&f)[2]) {
    if (S == 0) r_load(q, cnext, nxt);
    r_frags_h<2 * S + 1, false>(q, cur, m, f[1]);
    q_mma_half(acc, f[0], 0);
    r_quarter_reads<S == 0, NB>();
    if (MASK) r_mask_h(m, f[1]);
    if (S < RShape<NB>::KS / 2 - 1) {
        r_frags_h<2 * S + 2, false>(q, cur, m, f[0]);
    } else {
        if (!MASK) r_finish(nxt, fin);
        r_frags_h<0, false>(q, nxt, m, f[0]);
    }
    q_mma_half(acc, f[1], 0);
    r_quarter_reads<false, NB>();
    if (MASK) r_mask_h(m, f[0]);
}

// Stage S when only the wave's first A block runs: NB MFMAs and 1 + NB table reads per k-step
template <int S, bool MASK, int NB>
__device__ __forceinline__ void r_stage_q(const RSrc &q, int cnext, RData<NB> &cur, RData<NB> &nxt,
                                          const u4 (&m)[4], const bool (&fin)[4], v16f (&acc)[4][NB],
                                          RFrags<NB> (&f)[2]) {
    if (S == 0) r_load(q, cnext, nxt);
    r_frags_q<2 * S + 1, MASK>(q, cur, m, f[1]);
    q_mma_one(acc, f[0]);
    if (S < RShape<NB>::KS / 2 - 1) {
        r_frags_q<2 * S + 2, MASK>(q, cur, m, f[0]);
    } else {
        if (!MASK) r_finish(nxt, fin);
        r_frags_q<0, MASK>(q, nxt, m, f[0]);
    }
    q_mma_one(acc, f[1]);
}
template <bool MASK, int NB>
__device__ __forceinline__ void r_chunks_q(const RSrc &q, int c, int ce, RData<NB> &cur, RData<NB> &nxt,
                                           const u4 (&m)[4], const bool (&fin)[4], v16f (&acc)[4][NB],
                                           RFrags<NB> (&f)[2]) {
    for (; c < ce; ++c) {
        const int x = c + 1 < q.KC ? c + 1 : 0;
        r_stage_q<0, MASK>(q, x, cur, nxt, m, fin, acc, f);
        r_stage_q<1, MASK>(q, x, cur, nxt, m, fin, acc, f);
        r_stage_q<2, MASK>(q, x, cur, nxt, m, fin, acc, f);
        r_stage_q<3, MASK>(q, x, cur, nxt, m, fin, acc, f);
        if constexpr (RShape<NB>::KS == 16) {
            r_stage_q<4, MASK>(q, x, cur, nxt, m, fin, acc, f);
            r_stage_q<5, MASK>(q, x, cur, nxt, m, fin, acc, f);
            r_stage_q<6, MASK>(q, x, cur, nxt, m, fin, acc, f);
            r_stage_q<7, MASK>(q, x, cur, nxt, m, fin, acc, f);
        }
        cur = nxt;
    }
}

template <bool MASK, int NB>
__device__ __forceinline__ void r_chunks_h(const RSrc &q, int c, int ce, RData<NB> &cur, RData<NB> &nxt,
                                           const u4 (&m)[4], const bool (&fin)[4], v16f (&acc)[4][NB],
                                           RFrags<NB> (&f)[2]) {
    for (; c < ce; ++c) {
        const int x = c + 1 < q.KC ? c + 1 : 0;
        r_stage_h<0, MASK>(q, x, cur, nxt, m, fin, acc, f);
        r_stage_h<1, MASK>(q, x, cur, nxt, m, fin, acc, f);
        r_stage_h<2, MASK>(q, x, cur, nxt, m, fin, acc, f);
        r_stage_h<3, MASK>(q, x, cur, nxt, m, fin, acc, f);
        if constexpr (RShape<NB>::KS == 16) {
            r_stage_h<4, MASK>(q, x, cur, nxt, m, fin, acc, f);
            r_stage_h<5, MASK>(q, x, cur, nxt, m, fin, acc, f);
            r_stage_h<6, MASK>(q, x, cur, nxt, m, fin, acc, f);
            r_stage_h<7, MASK>(q, x, cur, nxt, m, fin, acc, f);
        }
        cur = nxt;
    }
}

// chunks c .. ce-1 of one cycle group; on exit cur holds the chunk after them (chunk ce, or
// chunk 0 of the next group) and fragment set 0 its first k-step (from this group's table)
template <bool MASK, int NB>
__device__ __forceinline__ void r_chunks(const RSrc &q, int c, int ce, RData<NB> &cur, RData<NB> &nxt,
                                         const u4 (&m)[4], const bool (&fin)[4], v16f (&acc)[4][NB],
                                         RFrags<NB> (&f)[2]) {
    for (; c < ce; ++c) {
        const int x = c + 1 < q.KC ? c + 1 : 0;
        r_stage<0, MASK>(q, x, cur, nxt, m, fin, acc, f);
        r_stage<1, MASK>(q, x, cur, nxt, m, fin, acc, f);
        r_stage<2, MASK>(q, x, cur, nxt, m, fin, acc, f);
        r_stage<3, MASK>(q, x, cur, nxt, m, fin, acc, f);
        if constexpr (RShape<NB>::KS == 16) {
            r_stage<4, MASK>(q, x, cur, nxt, m, fin, acc, f);
            r_stage<5, MASK>(q, x, cur, nxt, m, fin, acc, f);
            r_stage<6, MASK>(q, x, cur, nxt, m, fin, acc, f);
            r_stage<7, MASK>(q, x, cur, nxt, m, fin, acc, f);
        }
        cur = nxt;
    }
}

// One work unit, as in k_qgemm: tile `tile` over chunk steps [s, s + 1) / S of the pair's
// (group, chunk) steps, whole tiles decoded here, parts stored as partial sums.  Rows that
// have ended read the padding byte, whose table row is zero; a row that ends inside a
// cycle group reads there the table masked to its length.  MASK runs when some row pair
// holds more lengths inside a group than there are masked tables (then every A fragment is
// masked with its row's length instead): one launch, each block takes the variant the
// scheduler's flag names.
// NARROW (N <= 64): a block takes the pair's 256 rows x the first 64 columns of the B pair,
// two blocks per CU: wave (rh, kh) the rows of half rh and k-steps kh of every chunk, so that
// each SIMD runs two waves; the two k-halves are summed through the LDS at the end.  It has no
// masked tables (every length inside a group makes the call take the MASK variant).
// The LDS of a GEMM block: the group's table (64 KB, or 128 KB with the masked tables; the
// epilogue's transpose reuses it), bit r of rems[G]: a row ends r cycles into group G, and
// what the decode needs (filled after the chunk loop)
template <bool TABLES>
struct RLds {
    u4 lut[(TABLES ? 2 : 1) * 256 * 16];
    uint32_t rems[TABLES ? RGROUPS : 1];
    DecodeLds dl;
};

template <bool BIP, bool MASK, bool NARROW, bool TABLES>
__device__ __forceinline__ void rgemm_body(const MGemmArgs &g, const Layout &lay, uint8_t *ws, RLds<TABLES> &sh) {
    constexpr int NT = 256;                           // threads
    constexpr int NB = NARROW ? 2 : 4;                // B blocks of 32 columns per wave
    constexpr bool SKIP = NARROW;                     // skip the MFMAs of blocks whose rows ended
    static_assert(TABLES == (!MASK && !NARROW), "masked tables: the 256 x 256 variant without MASK");
    u4 *lut = sh.lut;
    uint32_t *rems = sh.rems;
    DecodeLds &dl = sh.dl;
    const int NTW = lay.NT / 2;
    // the block's units: one, or with vsplit its range of the work (k_units)
    int ub = blockIdx.x, ue = blockIdx.x + 1;
    if (lay.vsplit) {
        // The 256 x 64 blocks run two per CU; the dispatcher gives every CU one block before
        // any a second, so blocks b and b + sk_slots / 2 usually share a CU.  They take ranges
        // 2b and 2b + 1, neighbours in the tile order, so that the two blocks of a CU run
        // alike tiles and end together (measured 2 % faster on attention-V than CUs that each
        // hold one range of long tiles and one of short)
        const uint32_t *sl = ws_ptr<uint32_t>(ws, lay.off_slot);
        const int half = lay.sk_slots / 2, bi = (int)blockIdx.x;
        const int r = NARROW && lay.sk_slots % 2 == 0 ? (bi < half ? 2 * bi : 2 * (bi - half) + 1) : bi;
        ub = (int)sl[r];
        ue = (int)sl[r + 1];
    }
    for (int u = ub; u < ue; ++u) {
    // (the previous unit's epilogue is done with the LDS)
    if (u != ub) __syncthreads();
    int tile, s = 0, S = 1, v = -1;
    int64_t ux0 = 0, ux1 = 0;
    bool split;
    if (lay.vsplit) {
        const int4 e = ws_ptr<int4>(ws, lay.off_units)[u];
        tile = e.x;
        ux0 = e.y;
        ux1 = e.z;
        v = e.w;
        split = v >= 0;
    } else if (!q_unit(g, lay, ws, u, tile, s, S, v, split)) {
        return;
    }
    const int tw = tile % NTW;
    const int tb = tile / NTW;
    const int b = tb % g.batch, tp = tb / g.batch;
    const int bB = g.nbB == 1 ? 0 : b;
    // the thread index passes through an empty asm statement on every unit, so that nothing
    // derived from it is hoisted out of the unit loop and held (spilled) across it
    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    const int lane = tid & 63, w = tid >> 6;
    const int grp = lane >> 5, i32 = lane & 31;
    // (NARROW: the second block of a CU, block index cus.., swaps its waves' row halves, so
    // that when only row half 0 runs the two blocks' busy waves sit on different SIMDs)
    const int rswap = NARROW ? ((int)blockIdx.x / max(lay.cus, 1)) & 1 : 0;
    const int rh = NARROW ? (w & 1) ^ rswap : (w >> 1), wc = NARROW ? 0 : (w & 1) * 128;   // row half, columns
    const int kh = NARROW ? (w >> 1) : 0;                                          // k-half (NARROW)
    uint8_t *wsa = ws + (size_t)b * lay.stride_batchA;
    uint8_t *wsbB = ws + (size_t)bB * lay.stride_batchB;
    const int32_t *perm = ws_ptr<int32_t>(wsa, lay.off_perm) + tp * 256;
    const int32_t *Ls = ws_ptr<int32_t>(wsa, lay.off_Ls) + tp * 256;
    // (NARROW) a whole tile's decode data: loaded here, so that their latency overlaps the
    // unit's first loads instead of following its last chunk step, and staged in LDS before
    // the steps (compensator 3 % faster; the 256 x 256 blocks stage them after the steps, as
    // loading them here made them slower on per-row lengths)
    static_assert(NT == 256, "one row of decode data per thread");
    DRow drow{};
    if (NARROW && !split) drow = d_fetch(perm, Ls, b, tw, g, threadIdx.x);
    const size_t pairb = (size_t)g.KC * 256 * RCH;
    RSrc q;
    q.a = __builtin_amdgcn_make_buffer_rsrc(ws_ptr<uint8_t>(wsa, lay.off_Ap) + (size_t)tp * pairb, 0, (int)pairb,
                                            0x00020000);
    q.b = __builtin_amdgcn_make_buffer_rsrc(ws_ptr<uint8_t>(wsbB, lay.off_Bp) + (size_t)tw * pairb, 0, (int)pairb,
                                            0x00020000);
    q.voffA = ((SKIP ? 0 : 128 * rh) + i32) * RCH + grp * 16 + kh * 8;
#pragma unroll
    for (int i = 0; i < 4; ++i) q.boffA[i] = wave_uniform((SKIP ? 32 * r_block(rh, i) : 32 * i) * RCH);
    q.voffB = (wc + i32) * RCH + grp * 16 + kh * 8;
    q.KC = g.KC > 0 ? g.KC : 1;
    // A unit of the 256 x 256 blocks that knows its first chunk step before its tile's length
    // (whole tiles, and the units of the ranges division) loads that step's table entries and
    // chunk data at once, so that their latency overlaps the loads of the length and the rows
    // below.  (A tile of rows of length 0 runs no step; its early loads read data that exist
    // and go unused.  The 256 x 64 blocks measured slower with it: compensator +1.5 %.)
    const u4 *rtab = ws_ptr<u4>(ws, lay.off_rtab);
    const int64_t xs = NARROW ? -1 : lay.vsplit ? ux0 : (S == 1 ? 0 : -1);
    u4 ent[512 / NT];
    RData<NB> cur, nxt;
    if (xs >= 0 && g.KC > 0) {
        r_load_ent<NT>(ent, rtab + (size_t)(xs / q.KC) * 512, tid);
        r_load(q, (int)(xs % q.KC), cur);
    }
    const int ngroups = (int)(round_up(ws_ptr<int32_t>(wsa, lay.off_tileL)[2 * tp], RCH) / RCH);

    const int64_t nch = (int64_t)ngroups * g.KC;
    // the unit's chunk steps (a tile of rows of length 0 has none)
    const int64_t x1 = lay.vsplit ? min(ux1, nch) : (int64_t)(s + 1) * nch / S;
    const int64_t x0 = lay.vsplit ? min(ux0, x1) : (int64_t)s * nch / S;
    // this thread's entries of the group tables (the next group's loaded while the current
    // group runs) and the first chunk, unless loaded above: issued before the row lengths
    // below are waited for
    if (xs < 0 && x0 < x1) {
        r_load_ent<NT>(ent, rtab + (size_t)(x0 / g.KC) * 512, tid);
        r_load(q, (int)(x0 % q.KC), cur);
    }

    // (the layout holds a length for every row, padding rows too, so a row's length is
    // loaded beside its original index rather than after it)
    if (TABLES) {
        if (tid < ngroups) rems[tid] = 0u;
        __syncthreads();
        const int pt = perm[tid], lt = Ls[tid];
        const int Lt = pt >= 0 ? lt : 0;
        if (Lt % RCH != 0) atomicOr(&rems[Lt / RCH], 1u << (Lt % RCH));
        __syncthreads();
    }
    // the lane's A rows' lengths (padding rows: never end), and the longest length of the
    // wave's first two and last two blocks (their first rows; padding: 0)
    int Lr[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int row = r_row0<SKIP>(rh, i) + i32;
        const int pr = perm[row], lr = Ls[row];
        Lr[i] = pr >= 0 ? lr : INT_MAX;
    }
    const int h0 = r_row0<SKIP>(rh, 0), h1 = r_row0<SKIP>(rh, 2), h01 = r_row0<SKIP>(rh, 1);
    const int p0 = perm[h0], l0 = Ls[h0], p1 = perm[h1], l1 = Ls[h1], p01 = perm[h01], l01 = Ls[h01];
    const int Lh0 = wave_uniform(p0 >= 0 ? l0 : 0), Lh1 = wave_uniform(p1 >= 0 ? l1 : 0);
    const int Lh01 = wave_uniform(p01 >= 0 ? l01 : 0);

    const uint32_t lrep = 16u * (uint32_t)(lane & (RREP - 1));
    q.loB = lrep + 16u * RREP;
    q.lut = reinterpret_cast<const char *>(lut);

    v16f acc[4][NB];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int c = 0; c < NB; ++c) acc[i][c] = v16f{};

    RFrags<NB> f[2];
    u4 m[4];
    // One cycle group per trip: the collective table fill between two barriers, then the
    // wave's chunks.  Three phases in turn, as the wave's rows end: all four blocks run, only
    // the first two run, none runs (the wave still takes part in the table fills).  Separate
    // loops, so that a later phase holds none of an earlier one's registers.
    if (NARROW && !split) d_put(dl, drow, tid);   // (read after the epilogue's first barrier)
    int64_t x = x0;
    auto group_start = [&](int G, int64_t xe, bool (&fin)[4]) {
        const uint32_t rm = TABLES ? rems[G] : 0u;
        // every read of the previous group's table is done before it is replaced
        __syncthreads();
        r_fill_lut<NT>(lut, ent, tid, rm);
        if (xe < x1) {
            r_load_ent<NT>(ent, rtab + (size_t)(G + 1) * 512, tid);
        }
        __syncthreads();
        // the lane's A rows: ended, ending inside this group (the masked table of the
        // length's rank among the group's lengths; with MASK a mask instead) or running on
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int rem = Lr[i] - RCH * G;
            fin[i] = rem <= 0;
            q.loA[i] = lrep;
            if (MASK) {
                m[i] = r_len_mask(Lr[i], G);
            } else if (TABLES && rem > 0 && rem < RCH) {
                const uint32_t k = (uint32_t)__popc(rm & ((1u << rem) - 1u));
                q.loA[i] = 0x10000u | (16u * (k * RREP1 + (uint32_t)(lane & (RREP1 - 1))));
            }
        }
        if (!MASK) r_finish(cur, fin);
    };
    for (; x < x1;) {
        const int G = (int)(x / g.KC);
        if (SKIP && Lh1 <= RCH * G) break;
        const int64_t xe = min(x1, (int64_t)(G + 1) * g.KC);
        bool fin[4];
        group_start(G, xe, fin);
        r_frags<0, MASK>(q, cur, m, f[0]);
        r_chunks<MASK>(q, (int)(x - (int64_t)G * g.KC), (int)(xe - (int64_t)G * g.KC), cur, nxt, m, fin, acc, f);
        x = xe;
    }
    for (; SKIP && x < x1;) {
        const int G = (int)(x / g.KC);
        if (Lh01 <= RCH * G) break;
        const int64_t xe = min(x1, (int64_t)(G + 1) * g.KC);
        bool fin[4];
        group_start(G, xe, fin);
        r_frags_h<0, MASK>(q, cur, m, f[0]);
        r_chunks_h<MASK>(q, (int)(x - (int64_t)G * g.KC), (int)(xe - (int64_t)G * g.KC), cur, nxt, m, fin, acc, f);
        x = xe;
    }
    for (; SKIP && x < x1;) {
        const int G = (int)(x / g.KC);
        if (Lh0 <= RCH * G) break;
        const int64_t xe = min(x1, (int64_t)(G + 1) * g.KC);
        bool fin[4];
        group_start(G, xe, fin);
        r_frags_q<0, MASK>(q, cur, m, f[0]);
        r_chunks_q<MASK>(q, (int)(x - (int64_t)G * g.KC), (int)(xe - (int64_t)G * g.KC), cur, nxt, m, fin, acc, f);
        x = xe;
    }
    for (; SKIP && x < x1;) {
        const int G = (int)(x / g.KC);
        const int64_t xe = min(x1, (int64_t)(G + 1) * g.KC);
        __syncthreads();
        r_fill_lut<NT>(lut, ent, tid, TABLES ? rems[G] : 0u);
        if (xe < x1) r_load_ent<NT>(ent, rtab + (size_t)(G + 1) * 512, tid);
        __syncthreads();
        x = xe;
    }

    if (NARROW) {
        // the k-half 1 waves hand their sums to the k-half 0 waves of the same rows
        __syncthreads();   // (every read of the table is done)
        float4 *F = reinterpret_cast<float4 *>(lut) + rh * (4 * NB * 4 * 64);
        if (kh == 1) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int c = 0; c < NB; ++c)
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        F[((i * NB + c) * 4 + e) * 64 + lane] =
                            float4{acc[i][c][4 * e], acc[i][c][4 * e + 1], acc[i][c][4 * e + 2], acc[i][c][4 * e + 3]};
        }
        __syncthreads();
        if (kh == 0) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int c = 0; c < NB; ++c)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float4 t = F[((i * NB + c) * 4 + e) * 64 + lane];
                        acc[i][c][4 * e] += t.x;
                        acc[i][c][4 * e + 1] += t.y;
                        acc[i][c][4 * e + 2] += t.z;
                        acc[i][c][4 * e + 3] += t.w;
                    }
        }
    }
    if (split) {
        if (kh == 0)
            store_part_r<SKIP, NB>(acc,
                                   ws_ptr<uint8_t>(ws, lay.off_part) + (size_t)v * 256 * lay.pcols * (lay.p16 ? 2 : 4),
                                   lay.p16 != 0, rh, wc, lane);
        continue;
    }
    if (!NARROW) d_stage<NT>(dl, perm, Ls, b, tw, g, tid);
    // TR rows per pass: all that fit the table's LDS (64 KB, or 128 KB with the masked tables)
    constexpr int TS = NARROW ? 64 + 4 : 256 + 4, TR = NARROW ? 128 : (TABLES ? 64 : 32);
    static_assert(TR * TS * 4 <= (TABLES ? 2 : 1) * 256 * 16 * 16, "the epilogue transpose must fit the table");
    float *T = reinterpret_cast<float *>(lut);
    for (int h = 0; h < 256 / TR; ++h) {
        __syncthreads();
        // rows TR h .. TR h + TR - 1: the blocks i of each wave with r_row0(rh, i) among them
        // (NARROW: the k-half 0 waves, which hold the sums)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int rr = r_row0<SKIP>(rh, i) - TR * h;
            if (rr < 0 || rr >= TR || kh != 0) continue;
#pragma unroll
            for (int c = 0; c < NB; ++c)
#pragma unroll
                for (int e = 0; e < 16; ++e)
                    T[(rr + 8 * (e >> 2) + 4 * grp + (e & 3)) * TS + wc + 32 * c + i32] = acc[i][c][e];
        }
        __syncthreads();
        d_rows<BIP, NT, NARROW ? 16 : 64, TR, TS>(dl, T, TR * h, tw, b, g, tid);
    }
    }
}

// 256 x 256 blocks: one launch, each block takes the variant the status word names
union RLdsW {
    RLds<true> t;
    RLds<false> m;
};
template <bool BIP>
__global__ __launch_bounds__(256, 1) void k_rgemm(MGemmArgs g, Layout lay, uint8_t *ws) {
    __shared__ RLdsW sh;
    if (ws_ptr<uint32_t>(ws, lay.off_status)[2] != 0u) rgemm_body<BIP, true, false, false>(g, lay, ws, sh.m);
    else rgemm_body<BIP, false, false, true>(g, lay, ws, sh.t);
}

// 256 x 64 blocks: one launch, each block takes the variant the status word names
template <bool BIP>
__global__ __launch_bounds__(256, 2) void k_rgemm_n(MGemmArgs g, Layout lay, uint8_t *ws) {
    __shared__ RLds<false> sh;
    if (ws_ptr<uint32_t>(ws, lay.off_status)[2] != 0u) rgemm_body<BIP, true, true, false>(g, lay, ws, sh);
    else rgemm_body<BIP, false, true, false>(g, lay, ws, sh);
}

template <bool BIP, bool NARROW>
static hipError_t launch_rgemm_w(const MGemmArgs &g, const Layout &lay, uint8_t *ws, hipStream_t st) {
    const unsigned tiles = (unsigned)(g.batch * (lay.MT / 2) * (lay.NT / 2));
    const unsigned tail = tiles - (unsigned)g.F;
    const dim3 grid(lay.vsplit ? (unsigned)lay.sk_slots : (unsigned)g.F + tail * (unsigned)g.S),
        block(256);
    hipError_t e;
    if (NARROW) {
        gemm_launch((k_rgemm_n<BIP>), grid, block, st, tail == 0, g, lay, ws);
    } else {
        gemm_launch((k_rgemm<BIP>), grid, block, st, tail == 0, g, lay, ws);
    }
    e = hipGetLastError();
    if (e != hipSuccess || tail == 0) return e;
    return launch_qreduce<BIP>(g, lay, ws, tail, st);
}

template <bool BIP>
static hipError_t launch_rgemm(const MGemmArgs &g, const Layout &lay, uint8_t *ws, hipStream_t st) {
    return lay.narrow ? launch_rgemm_w<BIP, true>(g, lay, ws, st) : launch_rgemm_w<BIP, false>(g, lay, ws, st);
}

template <bool BIP>
static hipError_t launch_mgemm_pol(const MGemmArgs &g, const Layout &lay, uint8_t *ws,
                                   hipStream_t st) {
    if (lay.mbm == 256) return lay.rgen ? launch_rgemm<BIP>(g, lay, ws, st) : launch_qgemm<BIP>(g, lay, ws, st);
    if (lay.mbn == 256) return launch_mgemm_tile<BIP, 256>(g, lay, ws, st);
    return launch_mgemm_tile<BIP, 128>(g, lay, ws, st);
}

static MGemmArgs make_gemm_args(const sc_gemm_desc &d, const Layout &lay, const float *sA, const float *sB,
                                float *out, int32_t *counts) {
    MGemmArgs g{};
    g.M = d.M;
    g.N = d.N;
    g.K = d.K;
    g.KQP = lay.KQP;
    g.LBS = lay.LBS;
    g.nbB = lay.nbB;
    g.batch = d.batch;
    g.S = lay.S;
    g.F = lay.F;
    g.KC = lay.KC;
    g.sA = sA;
    g.sB = sB;
    g.strideSA = d.strideSA;
    g.strideSB = d.strideSB;
    g.strideO = d.strideO;
    g.ldo = d.ldo;
    g.out = out;
    g.counts = counts;
    g.vec_out = reinterpret_cast<uintptr_t>(out) % 16 == 0 && d.ldo % 4 == 0 && d.strideO % 4 == 0;
    g.vec_cnt = reinterpret_cast<uintptr_t>(counts) % 16 == 0 && d.ldo % 4 == 0 && d.strideO % 4 == 0;
    return g;
}

hipError_t launch_fgemm(const sc_gemm_desc &d, const Layout &lay, const int8_t *A, const int8_t *B,
                        const float *sA, const float *sB, float *out, int32_t *counts, uint8_t *ws,
                        hipStream_t st) {
    const MGemmArgs g = make_gemm_args(d, lay, sA, sB, out, counts);
    FArgs f{};
    f.A = A;
    f.B = B;
    f.lda = d.lda;
    f.ldb = d.ldb;
    f.strideA = d.strideA;
    f.strideB = d.strideB;
    // buffer loads check whole dwords against the extent, so it is rounded up to the dword
    // that holds the last byte (same page; the bytes past it are masked as elements >= K)
    f.bytesA = (uint32_t)round_up(fused_extent(d.M, d.lda, d.K), 4);
    f.bytesB = (uint32_t)round_up(fused_extent(d.N, d.ldb, d.K), 4);
    f.nbB = lay.nbB;
    f.L_max = d.L_max;
    if (d.polarity == SC_BIPOLAR_XNOR) return launch_fgemm_pol<SC_BIPOLAR_XNOR>(g, f, lay, ws, st);
    return launch_fgemm_pol<SC_UNIPOLAR_AND_SM>(g, f, lay, ws, st);
}

hipError_t launch_mgemm(const sc_gemm_desc &d, const Layout &lay, const float *sA, const float *sB,
                        float *out, int32_t *counts, uint8_t *ws, hipStream_t st) {
    const MGemmArgs g = make_gemm_args(d, lay, sA, sB, out, counts);
    if (d.polarity == SC_BIPOLAR_XNOR) return launch_mgemm_pol<true>(g, lay, ws, st);
    return launch_mgemm_pol<false>(g, lay, ws, st);
}

}  // namespace scg
