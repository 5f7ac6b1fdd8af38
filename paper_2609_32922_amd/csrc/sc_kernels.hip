// HIP kernels of libscgemm for gfx950 (MI355X): emulated stochastic-computing GEMM.
//
// Pipeline of one sc_gemm call (all on the caller's stream):
//   k_draws      comparator sequences r^A, r^B (Sec. 3.1 "Bitstream generation",
//                LFSR or scrambled Sobol-8 of Sec. A.1) -- one lane per cycle, the LFSR
//                through jump-ahead; it also clears the status words.  With one batch
//                entry and LFSR sequences k_schedule does both instead (one launch fewer)
//   k_cbsg_table C-BSG only: CA[L][beta] = ones of A's stream in its first L cycles
//   k_schedule   per-row length scheduler: validates L_i, counting-sorts rows by L
//                (descending) so that a 128-row tile runs for the longest length it
//                holds (Sec. 4.2: row i stops after its own l_i cycles; Sec. 4.1: the
//                cost grows with the sum of the l_i)
//   k_marginals  bipolar only: RA_i = sum_d sum_{l<L_i} zA and RB_j(L) for all L
//   k_planes     comparator stream generation into packed bit planes (one word =
//                32 inner-dimension elements at one cycle); 64 lanes compare one
//                row's 64 elements against r_l in one v_cmp, the wave ballot is the
//                packed word.  With C-BSG, A's planes are intervals of B's counter.
//   k_gemm       tiled AND/bitop3 + popcount over (d, l), int32 accumulators, and the
//                Eq. (1) decode epilogue in the original row order
//
// Bipolar XNOR counts use the bitwise identity XNOR(a,b) = 1 - a - b + 2ab summed
// over the valid cycles, X_ij = K L_i - RA_i - RB_j(L_i) + 2 AND_ij, so the hot loop
// is one AND and one popcount per 32 bit pairs and A's planes can be zero beyond L_i.
// Unipolar sign-magnitude counts use popc((a & b) ^ sigma) with sigma = signA ^ signB
// per 32 elements, which equals the signed AND count plus popc(sigma) per cycle.
//
// C-BSG (Sec. 4.2, Eq. (6)): with c = ones of A's stream over the row's L cycles and
// Z_k = [rB_k < beta_B], one element pair contributes
//   sum_k [k < c] Z_k + [k < L - c] (1 - Z_k) = (L - c) + sgn * sum_k D_k Z_k,
// D_k = [min(c, L-c) <= k < max(c, L-c)], sgn = -1 if c < L - c else +1,
// so the bipolar C-BSG counts run the same signed hot loop as unipolar, with A's
// planes holding D and A's signs holding sgn, plus the marginal K L - sum_d c.
// Unipolar C-BSG is the plain signed loop with A's planes holding [k < c].
#include "sc_internal.h"

namespace scg {

// ----------------------------------------------------------------------------
// comparator sequence
// ----------------------------------------------------------------------------
constexpr uint32_t kFeedback = 0x80200003u;   // x^32+x^22+x^2+x+1, Galois right-shift taps
constexpr uint32_t kPolyLow = 0x00400007u;    // the same polynomial minus x^32

constexpr uint32_t lfsr_step_ce(uint32_t s) { return (s >> 1) ^ ((s & 1u) ? kFeedback : 0u); }

// kJump.v[l] is the register state after 8*l steps from state 1.  A right-shift step
// multiplies the state polynomial by x^{-1} modulo p(x), so the state after 8*l steps
// from S_0 is S_0 * kJump.v[l] mod p(x): every cycle's draw is computed independently.
struct JumpTable {
    uint32_t v[SC_L_MAX_LIMIT];
};
constexpr JumpTable make_jump_table() {
    JumpTable t{};
    uint32_t s = 1u;
    for (int l = 0; l < SC_L_MAX_LIMIT; ++l) {
        t.v[l] = s;
        for (int k = 0; k < 8; ++k) s = lfsr_step_ce(s);
    }
    return t;
}
__constant__ JumpTable kJump = make_jump_table();

__device__ __forceinline__ uint64_t splitmix64(uint64_t x) {
    uint64_t z = x + 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// Product of two polynomials of degree < 32 modulo p(x), Horner from the top bit.
__device__ __forceinline__ uint32_t gf2_mulmod(uint32_t a, uint32_t b) {
    uint32_t acc = 0;
#pragma unroll
    for (int k = 31; k >= 0; --k) {
        acc = (acc << 1) ^ ((acc >> 31) ? kPolyLow : 0u);
        acc ^= ((a >> k) & 1u) ? b : 0u;
    }
    return acc;
}

// 8-bit Sobol direction numbers V_j = m_j 2^(8-j), j = 1..8: dimension 1 has m_j = 1;
// dimension 2 comes from the primitive polynomial x + 1, whose recurrence is
// m_j = m_{j-1} xor 2 m_{j-1} from m_1 = 1.
struct SobolDirs {
    uint32_t v[2][8];
};
constexpr SobolDirs make_sobol_dirs() {
    SobolDirs t{};
    uint32_t m = 1u;
    for (int j = 1; j <= 8; ++j) {
        t.v[0][j - 1] = 1u << (8 - j);
        if (j > 1) m = m ^ (m << 1);
        t.v[1][j - 1] = m << (8 - j);
    }
    return t;
}
__constant__ SobolDirs kSobol = make_sobol_dirs();

// Draw l of operand op (0: A, 1: B) of the comparator sequence.
__device__ __forceinline__ uint32_t draw_value(uint64_t seed, int rng, int op, int l) {
    const uint64_t h = splitmix64(2ull * seed + (uint64_t)op);
    uint32_t v = 0;
    if (rng == SC_RNG_SOBOL8_CBSG) {
        // point l (< 256) of dimension op + 1, digitally shifted by the top 8 bits of h
        v = (uint32_t)(h >> 56);
#pragma unroll
        for (int j = 0; j < 8; ++j)
            if ((l >> j) & 1) v ^= kSobol.v[op][j];
    } else {
        uint32_t s0 = (uint32_t)(h >> 32);
        if (s0 == 0u) s0 = 1u;
        uint32_t s = gf2_mulmod(s0, kJump.v[l]);
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            v = (v << 1) | (s & 1u);
            s = (s >> 1) ^ ((s & 1u) ? kFeedback : 0u);
        }
    }
    return v;
}

__global__ __launch_bounds__(256) void k_draws(uint64_t seed, int rng, int n, uint32_t *rA,
                                               uint32_t *rB, uint8_t *bytes_out, int op_only,
                                               uint32_t *status) {
    const int l = blockIdx.x * blockDim.x + threadIdx.x;
    const int op = op_only >= 0 ? op_only : (int)blockIdx.y;
    if (status != nullptr && l == 0 && blockIdx.y == 0) {
        status[0] = 0u;
        status[1] = 0u;   // longest tile pair of the call
        status[2] = 0u;   // some row pair holds more lengths inside a cycle group than tables
    }
    if (l >= n) return;
    const uint32_t v = draw_value(seed, rng, op, l);
    if (bytes_out != nullptr)
        bytes_out[l] = (uint8_t)v;
    else
        (op == 0 ? rA : rB)[l] = v;
}

hipError_t launch_draws(uint64_t seed, int rng, int n, uint32_t *rA, uint32_t *rB,
                        uint8_t *bytes_out, int op_only, uint32_t *status, hipStream_t st) {
    dim3 grid((unsigned)((n + 255) / 256), op_only >= 0 ? 1u : 2u);
    hipLaunchKernelGGL(k_draws, grid, dim3(256), 0, st, seed, rng, n, rA, rB, bytes_out, op_only,
                       status);
    return hipGetLastError();
}

// CA[L][beta] = #{l < L : rA_l < beta} for L = 0..L_max, beta = 0..256 (one thread per
// boundary; L_max <= 256 draws staged in LDS)
__global__ __launch_bounds__(320) void k_cbsg_table(const uint32_t *__restrict__ rA, int L_max,
                                                    uint16_t *__restrict__ CA) {
    __shared__ uint32_t r[CBSG_L_MAX];
    const int beta = threadIdx.x;
    for (int l = threadIdx.x; l < L_max; l += blockDim.x) r[l] = rA[l];
    __syncthreads();
    if (beta >= CA_COLS) return;
    uint32_t c = 0;
    for (int l = 0; l < L_max; ++l) {
        CA[(size_t)l * CA_COLS + beta] = (uint16_t)c;
        c += r[l] < (uint32_t)beta ? 1u : 0u;
    }
    CA[(size_t)L_max * CA_COLS + beta] = (uint16_t)c;
}

hipError_t launch_cbsg_table(const uint32_t *rA, int L_max, uint16_t *CA, hipStream_t st) {
    hipLaunchKernelGGL(k_cbsg_table, dim3(1), dim3(320), 0, st, rA, L_max, CA);
    return hipGetLastError();
}

// ----------------------------------------------------------------------------
// helpers
// ----------------------------------------------------------------------------

// v_writelane_b32 through the compiler intrinsic (not inline asm), so that the backend
// sees the instruction and inserts the wait states it needs after the v_cmp that
// produced the lane value in VCC.
__device__ int writelane_i32(int value, int lane, int old) __asm("llvm.amdgcn.writelane.i32");

// Inclusive scan across a 64-lane wave.
__device__ __forceinline__ int64_t wave_incl_scan(int64_t v, int lane) {
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int64_t t = __shfl_up(v, o, 64);
        if (lane >= o) v += t;
    }
    return v;
}

__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// Exclusive scan over a 1024-thread block; returns the block total in *total.
__device__ int64_t block_excl_scan_1024(int64_t v, int64_t *total) {
    __shared__ int64_t wsum[16];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int64_t inc = wave_incl_scan(v, lane);
    if (lane == 63) wsum[w] = inc;
    __syncthreads();
    if (w == 0) {
        int64_t x = lane < 16 ? wsum[lane] : 0;
        x = wave_incl_scan(x, lane);
        if (lane < 16) wsum[lane] = x;
    }
    __syncthreads();
    const int64_t base = w > 0 ? wsum[w - 1] : 0;
    *total = wsum[15];
    __syncthreads();
    return base + inc - v;
}

// acc += popcount(x) as one v_bcnt_u32_b32 with the accumulator as second source.
// Written out so that unrolled chains keep this one-instruction form instead of
// being reassociated into separate popcounts and three-input adds.  The s_nop ahead
// of each count measurably raises how often gfx950 issues two VALU instructions per
// SIMD in one quad-cycle in this AND/count stream (about 1.23x the single-issue rate
// on the 6304x768x3072 layer at L = 128).
__device__ __forceinline__ void popc_acc(int32_t &acc, uint32_t x) {
    asm("s_nop 0\n\tv_bcnt_u32_b32 %0, %1, %0" : "+v"(acc) : "v"(x));
}


// ----------------------------------------------------------------------------
// per-row length scheduler (one 1024-thread block per batch entry)
// ----------------------------------------------------------------------------
// Adds 1 to hist[l] for every active lane and returns the lane's old value (its place
// in bucket l).  The lanes that share the first active lane's l take one LDS atomic
// together, the others one each: equal lengths (the common case) cost one atomic per
// wave instead of one per row, and mixed lengths cost what single atomics cost.
__device__ int wave_bucket_add(int *hist, int l, bool active) {
    const int lane = threadIdx.x & 63;
    const uint64_t act = __ballot(active);
    if (act == 0) return 0;
    const int leader = __ffsll((unsigned long long)act) - 1;
    const int lv = __builtin_amdgcn_readlane(l, leader);
    const bool mine = active && l == lv;
    const uint64_t grp = __ballot(mine);
    int base = 0;
    if (lane == leader) base = atomicAdd(&hist[lv], __popcll(grp));
    base = __builtin_amdgcn_readlane(base, leader);
    if (mine) return base + __popcll(grp & ((1ull << lane) - 1));
    return active ? atomicAdd(&hist[l], 1) : 0;
}

__global__ __launch_bounds__(1024) void k_schedule(const int32_t *__restrict__ L, int64_t strideL,
                                                   int M, int L_max, Layout lay, uint8_t *ws, uint64_t seed,
                                                   int rng, int ndraws) {
    __shared__ int hist[SC_L_MAX_LIMIT + 1];
    const int b = blockIdx.x, tid = threadIdx.x;
    uint8_t *wsb = ws + (size_t)b * lay.stride_batchA;
    int32_t *perm = ws_ptr<int32_t>(wsb, lay.off_perm);
    int32_t *Ls = ws_ptr<int32_t>(wsb, lay.off_Ls);
    int32_t *RA = ws_ptr<int32_t>(wsb, lay.off_RA);     // zeroed here, summed by C-BSG planes
    int32_t *tileL = ws_ptr<int32_t>(wsb, lay.off_tileL);
    int64_t *tileOff = ws_ptr<int64_t>(wsb, lay.off_tileOff);
    uint32_t *status = ws_ptr<uint32_t>(ws, lay.off_status);
    const int32_t *Lb = L + (size_t)b * strideL;

    if (ndraws > 0) {
        // one batch entry: this block also clears the status words and makes the comparator
        // sequences (the work of k_draws), before any of its own status updates
        if (tid == 0) {
            status[0] = 0u;
            status[1] = 0u;
            status[2] = 0u;
        }
        uint32_t *rA = ws_ptr<uint32_t>(ws, lay.off_rA), *rB = ws_ptr<uint32_t>(ws, lay.off_rB);
        for (int l = tid; l < ndraws; l += 1024) {
            rA[l] = draw_value(seed, rng, 0, l);
            rB[l] = draw_value(seed, rng, 1, l);
        }
    }
    for (int v = tid; v <= L_max; v += 1024) hist[v] = 0;
    __syncthreads();
    // Up to SREG * 1024 rows the lengths are loaded once, all loads in flight together, and
    // kept in registers for the scatter; longer batch entries loop (and load them twice).
    constexpr int SREG = 8;
    const bool cached = M <= SREG * 1024;
    int lv[SREG];
    if (cached) {
#pragma unroll
        for (int k = 0; k < SREG; ++k) {
            const int i = k * 1024 + tid;
            lv[k] = i < M ? Lb[i] : 0;
        }
#pragma unroll
        for (int k = 0; k < SREG; ++k) {
            if (lv[k] < 0 || lv[k] > L_max) {
                atomicOr(status, STATUS_BAD_LENGTH);
                lv[k] = 0;
            }
            if (k * 1024 < M) wave_bucket_add(hist, lv[k], k * 1024 + tid < M);
        }
    } else {
        for (int i0 = 0; i0 < M; i0 += 1024) {
            const int i = i0 + tid;
            int l = i < M ? Lb[i] : 0;
            if (l < 0 || l > L_max) {
                atomicOr(status, STATUS_BAD_LENGTH);
                l = 0;
            }
            wave_bucket_add(hist, l, i < M);
        }
    }
    __syncthreads();
    // start position of each length bucket, longest lengths first
    int64_t carry = 0;
    for (int c = 0; c <= L_max; c += 1024) {
        const int idx = L_max - (c + tid);
        const int64_t v = idx >= 0 ? hist[idx] : 0;
        int64_t tot;
        const int64_t ex = block_excl_scan_1024(v, &tot);
        if (idx >= 0) hist[idx] = (int)(carry + ex);
        carry += tot;
        __syncthreads();
    }
    if (cached) {
#pragma unroll
        for (int k = 0; k < SREG; ++k) {
            const int i = k * 1024 + tid;
            if (k * 1024 >= M) break;
            const int pos = wave_bucket_add(hist, lv[k], i < M);
            if (i < M) {
                perm[pos] = i;
                Ls[pos] = lv[k];
                RA[pos] = 0;
            }
        }
    } else {
        for (int i0 = 0; i0 < M; i0 += 1024) {
            const int i = i0 + tid;
            int l = i < M ? Lb[i] : 0;
            if (l < 0 || l > L_max) l = 0;
            const int pos = wave_bucket_add(hist, l, i < M);
            if (i < M) {
                perm[pos] = i;
                Ls[pos] = l;
                RA[pos] = 0;
            }
        }
    }
    for (int p = M + tid; p < lay.MT * BM; p += 1024) {
        perm[p] = -1;
        Ls[p] = 0;
        RA[p] = 0;
    }
    __syncthreads();
    // After the scatter hist[l] is the end of length l's run of sorted positions (runs in
    // order of decreasing length, ends non-increasing in l): the length at sorted position
    // p < M is the largest l whose run ends after p.
    auto length_at = [&](int p) {
        if (p >= M) return 0;
        int lo = 0, hi = L_max;   // hist[lo] > p holds (hist[0] = M)
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (hist[mid] > p) lo = mid;
            else hi = mid - 1;
        }
        return lo;
    };
    // tile lengths (first sorted row of a tile holds its longest length; a pair of tiles
    // that one 256-row block takes runs at the pair's longest length) and offsets
    carry = 0;
    for (int c = 0; c < lay.MT; c += 1024) {
        const int t = c + tid;
        int tl = 0;
        if (t < lay.MT) {
            const int t0 = lay.mbm == 2 * BM ? (t & ~1) : t;
            tl = (int)round_up(length_at(t0 * BM), lay.tstep);
            tileL[t] = tl;
        }
        int64_t tot;
        const int64_t ex = block_excl_scan_1024((int64_t)tl * lay.words_per_L, &tot);
        if (t < lay.MT) tileOff[t] = carry + ex;
        carry += tot;
    }
    // the first tile pair holds the batch entry's longest rows
    if (tid == 0 && lay.mbm == 2 * BM) atomicMax(status + 1, (uint32_t)round_up(length_at(0), lay.tstep));
    // The int8-chunk GEMM keeps, per cycle group, a table of A masked to each row length
    // that ends inside the group: RSLOTS of them.  Rows are sorted, so the distinct lengths
    // of a pair are the first rows of runs of equal length; a pair with more such lengths
    // that are not multiples of 32 than tables makes the GEMM mask its fragments instead.
    if (lay.rgen) {
        // After the scatter hist[l] is the end of length l's run of sorted positions, and the
        // run starts where the run of l + 1 ends.  Each length that is not a multiple of 32
        // adds one to every pair its run meets (a difference array over pairs, then a scan).
        const int npairs = lay.MT / 2;
        __shared__ int dpair[2048 + 1];
        for (int q0 = 0; q0 < npairs; q0 += 2048) {
            const int nq = min(npairs - q0, 2048);
            __syncthreads();
            for (int q = tid; q <= nq; q += 1024) dpair[q] = 0;
            __syncthreads();
            for (int l = tid; l <= L_max; l += 1024) {
                const int end = hist[l], start = l == L_max ? 0 : hist[l + 1];
                if (l % 32 == 0 || end <= start) continue;
                const int qa = max(start >> 8, q0), qb = min((end - 1) >> 8, q0 + nq - 1);
                if (qa > qb) continue;
                atomicAdd(&dpair[qa - q0], 1);
                atomicAdd(&dpair[qb + 1 - q0], -1);
            }
            __syncthreads();
            int64_t carry = 0;
            bool over = false;
            for (int c = 0; c < nq; c += 1024) {
                const int q = c + tid;
                int64_t tot;
                const int64_t v = q < nq ? dpair[q] : 0;
                const int64_t ex = block_excl_scan_1024(v, &tot);
                over = over || (q < nq && carry + ex + v > lay.rslots);
                carry += tot;
            }
            if (__syncthreads_or(over) && tid == 0) atomicOr(status + 2, 1u);
        }
    }
}

hipError_t launch_schedule(const sc_gemm_desc &d, const Layout &lay, const int32_t *L, uint8_t *ws,
                           bool draws, hipStream_t st) {
    if (draws && d.batch != 1) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_schedule, dim3((unsigned)d.batch), dim3(1024), 0, st, L, d.strideL, d.M,
                       d.L_max, lay, ws, d.seed, d.rng, draws ? lay.LBS : 0);
    return hipGetLastError();
}

// ----------------------------------------------------------------------------
// marginals for the bipolar identity (one wave per row; 4 waves per block)
//   G[v] = #{d : beta_d > v}; the row's ones at cycle l are G[r_l].
// ----------------------------------------------------------------------------
__device__ void row_level_tail_counts(const int8_t *__restrict__ x, int K, int *hist, int lane) {
    // hist has 260 entries; on return hist[v] = #{d : beta(x_d) > v} for v in [0, 255]
    for (int v = lane; v < 260; v += 64) hist[v] = 0;
    __syncthreads();
    for (int dd = lane; dd < K; dd += 64) atomicAdd(&hist[beta_bipolar(x[dd])], 1);
    __syncthreads();
    // inclusive prefix over levels 0..255 (lane owns 4 consecutive levels)
    const int h0 = hist[4 * lane], h1 = hist[4 * lane + 1], h2 = hist[4 * lane + 2];
    const int h3 = hist[4 * lane + 3];
    const int own = h0 + h1 + h2 + h3;
    const int before = (int)wave_incl_scan(own, lane) - own;
    __syncthreads();
    // G[v] = K - #{beta <= v}
    hist[4 * lane] = K - (before + h0);
    hist[4 * lane + 1] = K - (before + h0 + h1);
    hist[4 * lane + 2] = K - (before + h0 + h1 + h2);
    hist[4 * lane + 3] = K - (before + own);
    __syncthreads();
}

// one 64-thread block per sorted row position of A
__global__ __launch_bounds__(64) void k_marginals_A(const int8_t *__restrict__ A, int64_t lda,
                                                    int64_t strideA, int K, Layout lay, uint8_t *ws) {
    __shared__ int hist[260];
    const int lane = threadIdx.x;
    const int p = blockIdx.x, b = blockIdx.y;
    uint8_t *wsb = ws + (size_t)b * lay.stride_batchA;
    const int32_t *perm = ws_ptr<int32_t>(wsb, lay.off_perm);
    const int32_t *Ls = ws_ptr<int32_t>(wsb, lay.off_Ls);
    int32_t *RA = ws_ptr<int32_t>(wsb, lay.off_RA);
    const uint32_t *rA = ws_ptr<uint32_t>(ws, lay.off_rA);
    const int i = perm[p];
    const int Li = Ls[p];
    if (i < 0 || Li == 0) {
        if (lane == 0) RA[p] = 0;
        return;
    }
    row_level_tail_counts(A + (size_t)b * strideA + (size_t)i * lda, K, hist, lane);
    int s = 0;
    for (int l = lane; l < Li; l += 64) s += hist[rA[l]];
    s = wave_sum(s);
    if (lane == 0) RA[p] = s;
}

// one 64-thread block per row of B: RB[j][L] for L = 0..L_max
__global__ __launch_bounds__(64) void k_marginals_B(const int8_t *__restrict__ B, int64_t ldb,
                                                    int64_t strideB, int K, int L_max, Layout lay,
                                                    uint8_t *ws) {
    __shared__ int hist[260];
    const int lane = threadIdx.x;
    const int j = blockIdx.x, b = blockIdx.y;
    uint8_t *wsb = ws + (size_t)b * lay.stride_batchB;
    int32_t *RB = ws_ptr<int32_t>(wsb, lay.off_RB) + (size_t)j * (L_max + 1);
    const uint32_t *rB = ws_ptr<uint32_t>(ws, lay.off_rB);
    row_level_tail_counts(B + (size_t)b * strideB + (size_t)j * ldb, K, hist, lane);
    int64_t carry = 0;
    if (lane == 0) RB[0] = 0;
    for (int l0 = 0; l0 < L_max; l0 += 64) {
        const int l = l0 + lane;
        const int64_t v = l < L_max ? hist[rB[l]] : 0;
        const int64_t inc = wave_incl_scan(v, lane);
        if (l < L_max) RB[l + 1] = (int32_t)(carry + inc);
        carry += __shfl(inc, 63, 64);
    }
}

hipError_t launch_marginals(const sc_gemm_desc &d, const Layout &lay, const int8_t *A, const int8_t *B,
                            uint8_t *ws, hipStream_t st) {
    const int rowsA = lay.MT * BM;
    hipLaunchKernelGGL(k_marginals_A, dim3((unsigned)rowsA, (unsigned)d.batch), dim3(64), 0, st, A,
                       d.lda, d.strideA, d.K, lay, ws);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_marginals_B, dim3((unsigned)d.N, (unsigned)lay.nbB), dim3(64), 0, st, B,
                       d.ldb, d.strideB, d.K, d.L_max, lay, ws);
    return hipGetLastError();
}

// ----------------------------------------------------------------------------
// stream generation into bit planes
// ----------------------------------------------------------------------------
struct PlaneArgs {
    const int8_t *X;
    int64_t ld, strideX;        // row stride, batch stride (elements)
    int rows, K, KB;
    int nchunk;                 // cycle blocks of LCH per tile in the grid
    int uniformL;               // cycles of every row when lengths are not per row
    int tile_rows;              // BM or BN (128)
    size_t stride_batch;        // bytes between batch entries of the workspace block
    size_t off_perm, off_Ls, off_tileL, off_tileOff;   // 0 = not used (B side)
    size_t off_planes, off_signs, off_r;
    size_t off_CA, off_RA;      // C-BSG (A side): count table, row marginal
    int per_row;                // 1: A side (sorted rows, per-row lengths)
    int LBS;                    // B side: cycle stride of the planes
};

// One block covers one 128-row tile, LCH cycles and 64 elements (two plane words per
// row and cycle).  Each wave takes 32 rows; its 64 lanes are the 64 elements.
//
// Comparator mode (CBSG = false): bit of element d at cycle l is [r_l < beta_d] for
// l < L_row.  Sign planes (unipolar) hold [q_d < 0].
//
// C-BSG mode (CBSG = true, A side only): A's planes are indexed by B's draw counter k.
// With c_d = CA[L_row][beta_d] the bit is [lo_d <= k < hi_d]: [0, c_d) for unipolar,
// [min(c_d, L-c_d), max(c_d, L-c_d)) for bipolar, whose sign planes hold [c_d < L - c_d]
// and whose blocks of the first cycle chunk add sum_d c_d into RA.
template <int POL, bool CBSG>
__global__ __launch_bounds__(256) void k_planes(PlaneArgs a, uint8_t *ws) {
    constexpr bool SIGNS = POL == SC_UNIPOLAR_AND_SM || CBSG;
    __shared__ uint32_t T[2][LCH][BM + 1];
    const int t = blockIdx.x / a.nchunk, ch = blockIdx.x % a.nchunk;
    const int dp = blockIdx.y, b = blockIdx.z;
    const int tid = threadIdx.x, lane = tid & 63, w = wave_uniform(tid >> 6);
    uint8_t *wsb = ws + (size_t)b * a.stride_batch;
    const uint32_t *r = ws_ptr<uint32_t>(ws, a.off_r);

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
        off = (int64_t)t * a.KB * a.LBS * BN;
    }
    const int l0 = ch * LCH;
    if (l0 >= Lloop) return;
    const int nl = min(LCH, Lloop - l0);
    uint32_t *planes = ws_ptr<uint32_t>(wsb, a.off_planes) + off;
    uint32_t *signs = SIGNS ? ws_ptr<uint32_t>(wsb, a.off_signs) : nullptr;
    const uint16_t *CA = CBSG ? ws_ptr<uint16_t>(ws, a.off_CA) : nullptr;
    int32_t *RA = CBSG && POL == SC_BIPOLAR_XNOR ? ws_ptr<int32_t>(wsb, a.off_RA) : nullptr;
    const int8_t *Xb = a.X + (size_t)b * a.strideX;
    const int d = dp * 64 + lane;
    // the chunk's 32 comparator draws, loaded once (l0 + 31 < LBS, the draw count)
    int rr[LCH];
    if (!CBSG) {
#pragma unroll
        for (int l = 0; l < LCH; ++l) rr[l] = wave_uniform((int)r[l0 + l]);
    }

    for (int k = 0; k < 32; ++k) {
        const int m = w * 32 + k;
        const int p = t * 128 + m;
        int row, Lr;
        if (a.per_row) {
            row = wave_uniform(perm[p]);
            Lr = row >= 0 ? wave_uniform(Ls[p]) : 0;
        } else {
            row = p < a.rows ? p : -1;
            Lr = row >= 0 ? a.uniformL : 0;
        }
        const bool valid = row >= 0 && d < a.K;
        const int q = valid ? (int)Xb[(size_t)row * a.ld + d] : 0;
        const int beta = valid ? (POL == SC_BIPOLAR_XNOR ? beta_bipolar(q) : beta_unipolar(q)) : 0;
        uint32_t word = 0;
        bool neg = valid && q < 0;
        if (CBSG) {
            const int c = valid ? (int)CA[(size_t)Lr * CA_COLS + beta] : 0;
            int lo = 0, hi = c;
            if (POL == SC_BIPOLAR_XNOR) {
                const int e = Lr - c;
                lo = min(c, e);
                hi = max(c, e);
                neg = valid && c < e;
                if (ch == 0) {
                    const int sc = wave_sum(c);
                    if (lane == 0 && sc != 0) atomicAdd(&RA[p], sc);
                }
            }
            const uint32_t width = (uint32_t)(valid ? hi - lo : 0);
#pragma unroll
            for (int l = 0; l < LCH; ++l) {
                // counter index l0 + l inside [lo, hi); beyond the row's length hi <= L
                const uint64_t m64 = __ballot((uint32_t)(l0 + l - lo) < width);
                word = (uint32_t)writelane_i32((int)(uint32_t)m64, l, (int)word);
                word = (uint32_t)writelane_i32((int)(uint32_t)(m64 >> 32), l + 32, (int)word);
            }
        } else {
            const int lrem = Lr - l0;          // cycles of this row left in the chunk
#pragma unroll
            for (int l = 0; l < LCH; ++l) {
                // a cycle past the row's length compares against 256: never a one
                const int thr = wave_uniform(l < lrem ? rr[l] : 256);
                const uint64_t m64 = __ballot(thr < beta);
                // lane l receives cycle l of the first 32 elements, lane 32+l of the next 32
                word = (uint32_t)writelane_i32((int)(uint32_t)m64, l, (int)word);
                word = (uint32_t)writelane_i32((int)(uint32_t)(m64 >> 32), l + 32, (int)word);
            }
        }
        T[lane >> 5][lane & 31][m] = word;
        if (SIGNS && ch == 0) {
            const uint64_t s64 = __ballot(neg);
            if (lane == 0) {
                const size_t so = ((size_t)t * a.KB + 2 * dp) * 128 + m;
                signs[so] = (uint32_t)s64;
                if (2 * dp + 1 < a.KB) signs[so + 128] = (uint32_t)(s64 >> 32);
            }
        }
    }
    __syncthreads();
    // coalesced copy-out: 2 words-per-cycle blocks x nl cycles x 128 words
    for (int e = tid; e < 2 * LCH * 32; e += 256) {
        const int g = e & 31, row = e >> 5;          // row = kbl * LCH + l
        const int kbl = row / LCH, l = row % LCH;
        const int kb = 2 * dp + kbl;
        if (kb < a.KB && l < nl) {
            uint4 v;
            v.x = T[kbl][l][4 * g];
            v.y = T[kbl][l][4 * g + 1];
            v.z = T[kbl][l][4 * g + 2];
            v.w = T[kbl][l][4 * g + 3];
            uint4 *dst = reinterpret_cast<uint4 *>(planes + ((size_t)kb * Lloop + l0 + l) * 128) + g;
            *dst = v;
        }
    }
}

template <bool CBSG>
static void launch_planes_side(int polarity, dim3 grid, const PlaneArgs &pa, uint8_t *ws,
                               hipStream_t st) {
    if (polarity == SC_BIPOLAR_XNOR)
        hipLaunchKernelGGL((k_planes<SC_BIPOLAR_XNOR, CBSG>), grid, dim3(256), 0, st, pa, ws);
    else
        hipLaunchKernelGGL((k_planes<SC_UNIPOLAR_AND_SM, CBSG>), grid, dim3(256), 0, st, pa, ws);
}

hipError_t launch_planes(const sc_gemm_desc &d, const Layout &lay, const int8_t *A, const int8_t *B,
                         uint8_t *ws, hipStream_t st) {
    const int dpairs = (lay.KB + 1) / 2;
    if (dpairs == 0) return hipSuccess;
    const bool cbsg = d.rng == SC_RNG_SOBOL8_CBSG;
    PlaneArgs pa{};
    pa.X = A;
    pa.ld = d.lda;
    pa.strideX = d.strideA;
    pa.rows = d.M;
    pa.K = d.K;
    pa.KB = lay.KB;
    pa.nchunk = (lay.LP + LCH - 1) / LCH;
    pa.uniformL = 0;
    pa.tile_rows = BM;
    pa.stride_batch = lay.stride_batchA;
    pa.off_perm = lay.off_perm;
    pa.off_Ls = lay.off_Ls;
    pa.off_tileL = lay.off_tileL;
    pa.off_tileOff = lay.off_tileOff;
    pa.off_planes = lay.off_Ap;
    pa.off_signs = lay.off_SA;
    pa.off_r = lay.off_rA;
    pa.off_CA = lay.off_CA;
    pa.off_RA = lay.off_RA;
    pa.per_row = 1;
    pa.LBS = lay.LBS;
    dim3 gA((unsigned)(lay.MT * pa.nchunk), (unsigned)dpairs, (unsigned)d.batch);
    if (cbsg)
        launch_planes_side<true>(d.polarity, gA, pa, ws, st);
    else
        launch_planes_side<false>(d.polarity, gA, pa, ws, st);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;

    PlaneArgs pb = pa;
    pb.X = B;
    pb.ld = d.ldb;
    pb.strideX = d.strideB;
    pb.rows = d.N;
    pb.nchunk = lay.LBS / LCH;
    pb.uniformL = d.L_max;
    pb.tile_rows = BN;
    pb.stride_batch = lay.stride_batchB;
    pb.off_perm = pb.off_Ls = pb.off_tileL = pb.off_tileOff = 0;
    pb.off_planes = lay.off_Bp;
    pb.off_signs = lay.off_SB;
    pb.off_r = lay.off_rB;
    pb.off_CA = pb.off_RA = 0;
    pb.per_row = 0;
    dim3 gB((unsigned)(lay.NT * pb.nchunk), (unsigned)dpairs, (unsigned)lay.nbB);
    launch_planes_side<false>(d.polarity, gB, pb, ws, st);
    return hipGetLastError();
}

// ----------------------------------------------------------------------------
// packed AND/bitop3 + popcount GEMM with the Eq. (1) decode epilogue
//
// The grid is one-dimensional over work units (tile, split): a 128x128 output tile
// of one batch entry, restricted to a contiguous range of the ceil(K/32) element
// blocks.  Units are ordered row-tile major, so the row tiles holding the longest
// streams (row tile 0 after the descending sort) are dispatched first.  With one
// split the decode runs in the GEMM epilogue; with several, each unit writes its
// int32 partial counts and k_gemm_reduce sums them and decodes.
// ----------------------------------------------------------------------------
struct GemmArgs {
    int M, N, K, KB, LBS, L_max, nbB, batch, S;
    const float *sA, *sB;
    int64_t strideSA, strideSB, strideO, ldo;
    float *out;
    int32_t *counts;
};

// counts and Eq. (1) decode of row r (0..7) of one thread's 8x8 block, written in the
// original row order.  acc holds, per mode: MODE_AND the AND count (X = K L - RA - RB +
// 2 acc); MODE_SIGNED the signed count S; MODE_CBSG sum_d sgn D.Z (X = K L - RA + acc).
template <int MODE>
__device__ __forceinline__ void epilogue_row(const int32_t (&acc)[8], int r, int b, int tm, int tn,
                                             int tx, int ty, const GemmArgs &g, const Layout &lay,
                                             uint8_t *ws) {
    const int bB = g.nbB == 1 ? 0 : b;
    uint8_t *wsa = ws + (size_t)b * lay.stride_batchA;
    uint8_t *wsbB = ws + (size_t)bB * lay.stride_batchB;
    const int rl = r < 4 ? 4 * ty + r : 64 + 4 * ty + (r - 4);
    const int p = tm * BM + rl;
    const int i = ws_ptr<int32_t>(wsa, lay.off_perm)[p];
    if (i < 0) return;
    const int Li = ws_ptr<int32_t>(wsa, lay.off_Ls)[p];
    const int ra = MODE != MODE_SIGNED ? ws_ptr<int32_t>(wsa, lay.off_RA)[p] : 0;
    const int32_t *RB = ws_ptr<int32_t>(wsbB, lay.off_RB);
    const float sa = g.sA[(size_t)b * g.strideSA + i];
    const float *sBb = g.sB + (size_t)b * g.strideSB;
    float *orow = g.out + (size_t)b * g.strideO + (size_t)i * g.ldo;
    int32_t *crow = g.counts ? g.counts + (size_t)b * g.strideO + (size_t)i * g.ldo : nullptr;
    const float scale = sa * 16129.0f;
    const int KL = g.K * Li;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int j0 = tn * BN + h * 64 + 4 * tx;       // four adjacent columns
        if (j0 >= g.N) continue;
        int rb[4] = {0, 0, 0, 0};
        if (MODE == MODE_AND) {
#pragma unroll
            for (int c = 0; c < 4; ++c)
                if (j0 + c < g.N) rb[c] = RB[(size_t)(j0 + c) * (g.L_max + 1) + Li];
        }
        float o[4];
        int32_t cnt[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int j = j0 + c < g.N ? j0 + c : j0;
            int32_t num;
            if (MODE == MODE_AND) {
                cnt[c] = KL - ra - rb[c] + 2 * acc[4 * h + c];
                num = 2 * cnt[c] - KL;
            } else if (MODE == MODE_CBSG) {
                cnt[c] = KL - ra + acc[4 * h + c];
                num = 2 * cnt[c] - KL;
            } else {
                cnt[c] = acc[4 * h + c];
                num = cnt[c];
            }
            o[c] = 0.0f;
            if (Li > 0) o[c] = (float)num / (float)Li * (scale * sBb[j]);
            else cnt[c] = 0;
        }
        float *op = orow + j0;
        if (j0 + 3 < g.N && (reinterpret_cast<uintptr_t>(op) & 15) == 0) {
            *reinterpret_cast<float4 *>(op) = make_float4(o[0], o[1], o[2], o[3]);
        } else {
#pragma unroll
            for (int c = 0; c < 4; ++c)
                if (j0 + c < g.N) op[c] = o[c];
        }
        if (crow) {
            int32_t *cp = crow + j0;
            if (j0 + 3 < g.N && (reinterpret_cast<uintptr_t>(cp) & 15) == 0) {
                *reinterpret_cast<int4 *>(cp) = make_int4(cnt[0], cnt[1], cnt[2], cnt[3]);
            } else {
#pragma unroll
                for (int c = 0; c < 4; ++c)
                    if (j0 + c < g.N) cp[c] = cnt[c];
            }
        }
    }
}

template <int MODE, bool SPLIT>
__global__ __launch_bounds__(256) void k_gemm(GemmArgs g, Layout lay, uint8_t *ws) {
    __shared__ uint4 As[LCH * BM / 4];
    __shared__ uint4 Bs[LCH * BN / 4];
    // unit -> (row tile, batch entry, column tile, split), row tile slowest
    const int u = blockIdx.x;
    const int s = u % g.S;
    const int tile = u / g.S;              // = (tm * batch + b) * NT + tn
    const int tn = tile % lay.NT;
    const int tb = tile / lay.NT;
    const int b = tb % g.batch, tm = tb / g.batch;
    const int kb0 = (int)((int64_t)s * g.KB / g.S), kb1 = (int)((int64_t)(s + 1) * g.KB / g.S);
    const int bB = g.nbB == 1 ? 0 : b;
    const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
    uint8_t *wsa = ws + (size_t)b * lay.stride_batchA;
    uint8_t *wsbB = ws + (size_t)bB * lay.stride_batchB;
    const int Lloop = ws_ptr<int32_t>(wsa, lay.off_tileL)[tm];
    const int64_t offA = ws_ptr<int64_t>(wsa, lay.off_tileOff)[tm];
    const uint32_t *Ap = ws_ptr<uint32_t>(wsa, lay.off_Ap) + offA;
    const uint32_t *Bp = ws_ptr<uint32_t>(wsbB, lay.off_Bp);

    int32_t acc[8][8];
#pragma unroll
    for (int r = 0; r < 8; ++r)
#pragma unroll
        for (int c = 0; c < 8; ++c) acc[r][c] = 0;

    for (int kb = kb0; kb < kb1 && Lloop > 0; ++kb) {
        uint32_t sig[8][8];
        if (MODE != MODE_AND) {
            const uint4 *sa4 = reinterpret_cast<const uint4 *>(ws_ptr<uint32_t>(wsa, lay.off_SA) +
                                                               ((size_t)tm * g.KB + kb) * BM);
            const uint4 a0 = sa4[ty], a1 = sa4[16 + ty];
            uint4 b0 = make_uint4(0u, 0u, 0u, 0u), b1 = b0;
            if (MODE == MODE_SIGNED) {
                const uint4 *sb4 = reinterpret_cast<const uint4 *>(
                    ws_ptr<uint32_t>(wsbB, lay.off_SB) + ((size_t)tn * g.KB + kb) * BN);
                b0 = sb4[tx];
                b1 = sb4[16 + tx];
            }
            const uint32_t sa[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
            const uint32_t sb[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
#pragma unroll
            for (int r = 0; r < 8; ++r)
#pragma unroll
                for (int c = 0; c < 8; ++c) {
                    sig[r][c] = sa[r] ^ sb[c];
                    acc[r][c] -= Lloop * __builtin_popcount(sig[r][c]);
                }
        }
        const uint4 *gA = reinterpret_cast<const uint4 *>(Ap + (size_t)kb * Lloop * BM);
        const uint4 *gB = reinterpret_cast<const uint4 *>(Bp + ((size_t)tn * g.KB + kb) * g.LBS * BN);
        for (int l0 = 0; l0 < Lloop; l0 += LCH) {
            const int nl = min(LCH, Lloop - l0);
            __syncthreads();
            for (int e = tid; e < nl * 32; e += 256) {
                As[e] = gA[l0 * 32 + e];
                Bs[e] = gB[l0 * 32 + e];
            }
            __syncthreads();
            for (int l = 0; l < nl; l += LSTEP) {
#pragma unroll
                for (int v = 0; v < LSTEP; ++v) {
                    const uint4 a0 = As[(l + v) * 32 + ty], a1 = As[(l + v) * 32 + 16 + ty];
                    const uint4 b0 = Bs[(l + v) * 32 + tx], b1 = Bs[(l + v) * 32 + 16 + tx];
                    const uint32_t av[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
                    const uint32_t bv[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
#pragma unroll
                    for (int r = 0; r < 8; ++r)
#pragma unroll
                        for (int c = 0; c < 8; ++c) {
                            if (MODE != MODE_AND)
                                popc_acc(acc[r][c], (av[r] & bv[c]) ^ sig[r][c]);
                            else
                                popc_acc(acc[r][c], av[r] & bv[c]);
                        }
                }
            }
        }
    }

    if (SPLIT) {
        // partial counts of this split: [tile][split][thread][64] int32, 256 B per thread
        int4 *dst = reinterpret_cast<int4 *>(ws_ptr<int32_t>(ws, lay.off_part) +
                                             (((size_t)tile * g.S + s) * 256 + tid) * 64);
#pragma unroll
        for (int r = 0; r < 8; ++r) {
            dst[2 * r] = make_int4(acc[r][0], acc[r][1], acc[r][2], acc[r][3]);
            dst[2 * r + 1] = make_int4(acc[r][4], acc[r][5], acc[r][6], acc[r][7]);
        }
    } else {
#pragma unroll
        for (int r = 0; r < 8; ++r) epilogue_row<MODE>(acc[r], r, b, tm, tn, tx, ty, g, lay, ws);
    }
}

// sums the partial counts of every split of a tile and decodes.  Four blocks per
// tile; reduce thread (g, q) owns rows 2q and 2q+1 of GEMM thread g's 8x8 block, so
// the four threads of one g read adjacent 64-byte pieces of its partials.
template <int MODE>
__global__ __launch_bounds__(256) void k_gemm_reduce(GemmArgs g, Layout lay, uint8_t *ws) {
    const int tile = blockIdx.x >> 2;
    const int tn = tile % lay.NT;
    const int tb = tile / lay.NT;
    const int b = tb % g.batch, tm = tb / g.batch;
    const int gt = (blockIdx.x & 3) * 64 + (threadIdx.x >> 2);   // GEMM thread
    const int q = threadIdx.x & 3;
    const int tx = gt & 15, ty = gt >> 4;
    int32_t acc0[8], acc1[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) acc0[c] = acc1[c] = 0;
    const int4 *base = reinterpret_cast<const int4 *>(ws_ptr<int32_t>(ws, lay.off_part)) +
                       ((size_t)tile * g.S * 256 + gt) * 16 + 4 * q;
    for (int s = 0; s < g.S; ++s) {
        const int4 *src = base + (size_t)s * 256 * 16;
        const int4 u0 = src[0], v0 = src[1], u1 = src[2], v1 = src[3];
        acc0[0] += u0.x; acc0[1] += u0.y; acc0[2] += u0.z; acc0[3] += u0.w;
        acc0[4] += v0.x; acc0[5] += v0.y; acc0[6] += v0.z; acc0[7] += v0.w;
        acc1[0] += u1.x; acc1[1] += u1.y; acc1[2] += u1.z; acc1[3] += u1.w;
        acc1[4] += v1.x; acc1[5] += v1.y; acc1[6] += v1.z; acc1[7] += v1.w;
    }
    epilogue_row<MODE>(acc0, 2 * q, b, tm, tn, tx, ty, g, lay, ws);
    epilogue_row<MODE>(acc1, 2 * q + 1, b, tm, tn, tx, ty, g, lay, ws);
}

template <int MODE>
static hipError_t launch_gemm_mode(const GemmArgs &g, const Layout &lay, uint8_t *ws, hipStream_t st) {
    const unsigned tiles = (unsigned)(g.batch * lay.MT * lay.NT);
    if (g.S == 1) {
        hipLaunchKernelGGL((k_gemm<MODE, false>), dim3(tiles), dim3(256), 0, st, g, lay, ws);
        return hipGetLastError();
    }
    hipLaunchKernelGGL((k_gemm<MODE, true>), dim3(tiles * (unsigned)g.S), dim3(256), 0, st, g, lay, ws);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((k_gemm_reduce<MODE>), dim3(tiles * 4u), dim3(256), 0, st, g, lay, ws);
    return hipGetLastError();
}

hipError_t launch_gemm(const sc_gemm_desc &d, const Layout &lay, const float *sA, const float *sB,
                       float *out, int32_t *counts, uint8_t *ws, hipStream_t st) {
    GemmArgs g{};
    g.M = d.M;
    g.N = d.N;
    g.K = d.K;
    g.KB = lay.KB;
    g.LBS = lay.LBS;
    g.L_max = d.L_max;
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
    if (lay.mode == MODE_AND) return launch_gemm_mode<MODE_AND>(g, lay, ws, st);
    if (lay.mode == MODE_CBSG) return launch_gemm_mode<MODE_CBSG>(g, lay, ws, st);
    return launch_gemm_mode<MODE_SIGNED>(g, lay, ws, st);
}

}  // namespace scg
