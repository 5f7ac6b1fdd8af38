// HIP kernels of libscgemm for gfx950 (MI355X) that precede the counting GEMM of an SC
// GEMM call (the GEMM itself is in sc_mfma.hip).  All run on the caller's stream:
//   k_draws      comparator sequences r^A, r^B (Sec. 3.1 "Bitstream generation",
//                LFSR or scrambled Sobol-8 of Sec. A.1) -- one lane per cycle, the LFSR
//                through jump-ahead; it also clears the status words.  With one batch
//                entry and LFSR sequences k_schedule does both instead (one launch fewer)
//   k_cbsg_table C-BSG only: CA[L][beta] = ones of A's stream in its first L cycles
//   k_schedule   per-row length scheduler: validates L_i, counting-sorts rows by L
//                (descending) so that a 128-row tile runs for the longest length it
//                holds (Sec. 4.2: row i stops after its own l_i cycles; Sec. 4.1: the
//                cost grows with the sum of the l_i)
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

// Inclusive scan across a 64-lane wave.
__device__ __forceinline__ int64_t wave_incl_scan(int64_t v, int lane) {
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int64_t t = __shfl_up(v, o, 64);
        if (lane >= o) v += t;
    }
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
    __shared__ int hstart[SC_L_MAX_LIMIT + 1];
    __shared__ int dpair[2048 + 1];
    __shared__ int lmin, lmax;
    const int b = blockIdx.x, tid = threadIdx.x;
    uint8_t *wsb = ws + (size_t)b * lay.stride_batchA;
    int32_t *perm = ws_ptr<int32_t>(wsb, lay.off_perm);
    int32_t *Ls = ws_ptr<int32_t>(wsb, lay.off_Ls);
    int32_t *tileL = ws_ptr<int32_t>(wsb, lay.off_tileL);
    int64_t *tileOff = ws_ptr<int64_t>(wsb, lay.off_tileOff);
    uint32_t *status = ws_ptr<uint32_t>(ws, lay.off_status);
    const int32_t *Lb = L + (size_t)b * strideL;

    // Up to SREG * 1024 rows the lengths are loaded once, all loads in flight together (issued
    // first, so that their latency overlaps the sequences and the clearing below), and kept in
    // registers for the scatter; longer batch entries loop (and load them twice).
    constexpr int SREG = 20;
    const bool cached = M <= SREG * 1024;
    int lv[SREG];
    if (cached) {
#pragma unroll
        for (int k = 0; k < SREG; ++k) {
            const int i = k * 1024 + tid;
            lv[k] = i < M ? Lb[i] : 0;
        }
    }
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
    if (tid == 0) {
        lmin = INT_MAX;
        lmax = INT_MIN;
    }
    __syncthreads();
    // the lengths held in registers: validated, and their range over the batch entry
    if (cached) {
        int lo = INT_MAX, hi = INT_MIN;
#pragma unroll
        for (int k = 0; k < SREG; ++k) {
            if (lv[k] < 0 || lv[k] > L_max) {
                atomicOr(status, STATUS_BAD_LENGTH);
                lv[k] = 0;
            }
            if (k * 1024 + tid < M) {
                lo = min(lo, lv[k]);
                hi = max(hi, lv[k]);
            }
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
            lo = min(lo, __shfl_xor(lo, o, 64));
            hi = max(hi, __shfl_xor(hi, o, 64));
        }
        if ((tid & 63) == 0) {
            atomicMin(&lmin, lo);
            atomicMax(&lmax, hi);
        }
        __syncthreads();
    }
    // One length for every row (M > 0): the sort keeps the row order, and the counts below
    // are set directly.
    const bool one = cached && M > 0 && lmin == lmax;
    if (one) {
        const int l = lmin;
        // as after the scatter of the general path: hist[v] = end and hstart[v] = start of
        // length v's run of sorted positions (lengths above l: empty runs at 0, below: at M)
        for (int v = tid; v <= L_max; v += 1024) {
            hist[v] = v <= l ? M : 0;
            hstart[v] = v < l ? M : 0;
        }
#pragma unroll
        for (int k = 0; k < SREG; ++k) {
            const int i = k * 1024 + tid;
            if (i < M) {
                perm[i] = i;
                Ls[i] = l;
            }
        }
        // every pair meets one length; it is not a multiple of 32 only when l is not
        if (tid == 0 && lay.rgen && l % 32 != 0 && lay.rslots < 1) atomicOr(status + 2, 1u);
    } else if (cached) {
#pragma unroll
        for (int k = 0; k < SREG; ++k)
            if (k * 1024 < M) wave_bucket_add(hist, lv[k], k * 1024 + tid < M);
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
    // start position of each length bucket, longest lengths first (also kept in hstart: the
    // scatter below moves hist[l] on to the end of l's run)
    int64_t carry = 0;
    for (int c = 0; !one && c <= L_max; c += 1024) {
        const int idx = L_max - (c + tid);
        const int64_t v = idx >= 0 ? hist[idx] : 0;
        int64_t tot;
        const int64_t ex = block_excl_scan_1024(v, &tot);
        if (idx >= 0) {
            hist[idx] = (int)(carry + ex);
            hstart[idx] = (int)(carry + ex);
        }
        carry += tot;
        __syncthreads();
    }
    if (one) {
        // (done above)
    } else if (cached) {
#pragma unroll
        for (int k = 0; k < SREG; ++k) {
            const int i = k * 1024 + tid;
            if (k * 1024 >= M) break;
            const int pos = wave_bucket_add(hist, lv[k], i < M);
            if (i < M) {
                perm[pos] = i;
                Ls[pos] = lv[k];
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
            }
        }
    }
    for (int p = M + tid; p < lay.MT * BM; p += 1024) {
        perm[p] = -1;
        Ls[p] = 0;
    }
    // The int8-chunk GEMM keeps, per cycle group, a table of A masked to each row length
    // that ends inside the group: rslots of them.  Rows are sorted, so the distinct lengths of
    // a pair are the runs of equal length that meet it; a pair that more lengths which are not
    // multiples of 32 meet than there are tables makes the GEMM mask its fragments instead.
    // Each such length adds one to every pair its run [hstart[l], end) meets (a difference
    // array over pairs, then a scan); end = hstart[l - 1] (runs in order of decreasing
    // length), or M.  (Up to 2048 pairs per pass; the first pass runs beside the scatter.)
    const int npairs = lay.rgen && !one ? lay.MT / 2 : 0;
    for (int q0 = 0; q0 < npairs; q0 += 2048) {
        const int nq = min(npairs - q0, 2048);
        if (q0 > 0) __syncthreads();
        for (int q = tid; q <= nq; q += 1024) dpair[q] = 0;
        __syncthreads();
        for (int l = tid; l <= L_max; l += 1024) {
            const int start = hstart[l], end = l == 0 ? M : hstart[l - 1];
            if (l % 32 == 0 || end <= start) continue;
            const int qa = max(start >> 8, q0), qb = min((end - 1) >> 8, q0 + nq - 1);
            if (qa > qb) continue;
            atomicAdd(&dpair[qa - q0], 1);
            atomicAdd(&dpair[qb + 1 - q0], -1);
        }
        __syncthreads();
        int64_t pc = 0;
        bool over = false;
        for (int c = 0; c < nq; c += 1024) {
            const int q = c + tid;
            int64_t tot;
            const int64_t v = q < nq ? dpair[q] : 0;
            const int64_t ex = block_excl_scan_1024(v, &tot);
            over = over || (q < nq && pc + ex + v > lay.rslots);
            pc += tot;
        }
        if (__syncthreads_or(over) && tid == 0) atomicOr(status + 2, 1u);
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
    // that one 256-row block takes runs at the pair's longest length) and, for the GEMMs that
    // read planes, the tiles' plane offsets
    carry = 0;
    for (int c = 0; c < lay.MT; c += 1024) {
        const int t = c + tid;
        int tl = 0;
        if (t < lay.MT) {
            const int t0 = lay.mbm == 2 * BM ? (t & ~1) : t;
            tl = (int)round_up(length_at(t0 * BM), MSTEP);
            tileL[t] = tl;
        }
        if (!lay.rgen) {
            int64_t tot;
            const int64_t ex = block_excl_scan_1024((int64_t)tl * lay.words_per_L, &tot);
            if (t < lay.MT) tileOff[t] = carry + ex;
            carry += tot;
        }
    }
    // the first tile pair holds the batch entry's longest rows
    if (tid == 0 && lay.mbm == 2 * BM) atomicMax(status + 1, (uint32_t)round_up(length_at(0), MSTEP));
}

// Work division of the int8-chunk GEMM when row lengths vary (Layout::vsplit).  Tile t (pair
// tp of batch entry b x B pair tw, in the GEMM's tile order: longest pairs first) runs
// ceil(tileL / 32) x KC chunk steps (32-cycle groups x 32-element chunks) and then decodes.
// Its cost, in units of the time of one step: W1 per step while every row block of the
// block runs, W2 per step once the 256 x 64 blocks run only the first half of each wave's
// row blocks (from the group where sorted row 128 of the pair has ended: rows are sorted by
// length, and the blocks {2, 3} and {6, 7} of the waves' row halves hold rows 128 .. 255),
// W3 once they run only row block 0 (from the group where sorted row 32 has ended),
// at least 1 (a tile of rows of length 0 still writes its zeros), plus E for its decode and
// prologue (measured: 13.6 + 3.7 us against 3.6 us per step for 256 x 256 blocks; 13.4 us
// against 1.65 us per step for 256 x 64 blocks, whose best E measured 5 steps of 3, 5 and 8).
// The tiles' costs are laid end to end and the total cut into sk_slots ranges of about
// T = ceil(W / sk_slots) (see cut() below), range s for GEMM block s: every block
// gets the same share of the MFMA work, which follows the sum of the row lengths (Sec. 4.1),
// and of the decodes.  A tile inside one range runs whole and is decoded by its block; a
// tile that c cuts cross through its steps runs as c + 1 pieces (a cut maps to the first
// step whose cost ends after it), whose partial sums the split-sum pass adds (a cut through
// the decode's share leaves the steps to one piece).  Written: units {tile, first step, end
// step, partial index or -1} in tile order, which is range order; slot[s] = the first unit
// of range s (slot[sk_slots] = the unit count); tinfo[t] = {pieces, partial index of piece
// 0}.  One block.
__global__ __launch_bounds__(1024) void k_units(Layout lay, int batch, uint8_t *ws) {
    const int tid = threadIdx.x;
    const int NTW = lay.NT / 2, npairs = lay.MT / 2, slots = lay.sk_slots;
    const int tiles = batch * npairs * NTW;
    const int64_t W1 = lay.narrow ? RW1_NARROW : 1, W2 = lay.narrow ? RW2_NARROW : 1;
    const int64_t W3 = lay.narrow ? RW3_NARROW : 1;
    const int64_t E = 5 * W1;
    // tile t's steps at weight W1, W2 and W3 (the 256 x 64 blocks: from the group after which
    // sorted row 128, then row 32, of the pair has ended)
    auto steps = [&](int t) -> int4 {
        const int tb = t / NTW, b = tb % batch, tp = tb / batch;
        uint8_t *wsb = ws + (size_t)b * lay.stride_batchA;
        const int g0 = (ws_ptr<int32_t>(wsb, lay.off_tileL)[2 * tp] + 31) / 32;
        int g1 = g0, g2 = g0;
        if (lay.narrow) {
            auto ends = [&](int r) {
                const int L1 = ws_ptr<int32_t>(wsb, lay.off_perm)[r] >= 0 ? ws_ptr<int32_t>(wsb, lay.off_Ls)[r] : 0;
                return min((L1 + 31) / 32, g0);
            };
            g1 = ends(tp * 256 + 128);
            g2 = max(ends(tp * 256 + 32), g1);
        }
        return make_int4(g1 * lay.KC, (g2 - g1) * lay.KC, (g0 - g2) * lay.KC, 0);
    };
    auto cost = [&](int4 n) -> int64_t {
        const int64_t c = (int64_t)n.x * W1 + (int64_t)n.y * W2 + (int64_t)n.z * W3;
        return c > 0 ? c : 1;
    };
    // the steps whose cost ends at or before c (0 <= c <= cost(n); c = cost(n): every step)
    auto step_at = [&](int4 n, int64_t c) -> int64_t {
        const int64_t c1 = (int64_t)n.x * W1, c2 = c1 + (int64_t)n.y * W2;
        return c < c1 ? c / W1 : c < c2 ? n.x + (c - c1) / W2 : n.x + n.y + (c - c2) / W3;
    };
    int64_t W = 0;
    for (int c = 0; c < tiles; c += 1024) {
        int64_t tot;
        block_excl_scan_1024(c + tid < tiles ? cost(steps(c + tid)) + E : 0, &tot);
        W += tot;
    }
    const int64_t T = (W + slots - 1) / slots;
    // Range s covers the costs [cut(s), cut(s + 1)).  The 256 x 64 blocks take the ranges in
    // pairs, 2p for the first block of a CU and 2p + 1 for the second, the first
    // (16 + RLEAD_NARROW) / 16 T long (cut(slots) = slots T >= W either way).
    const bool lead = lay.narrow && slots % 2 == 0;
    const int64_t TL = lead ? T + T * RLEAD_NARROW / 16 : T;
    auto cut = [&](int64_t s) -> int64_t { return lead ? (s >> 1) * 2 * T + (s & 1) * TL : s * T; };
    auto range_of = [&](int64_t c) -> int64_t {
        if (!lead) return c / T;
        const int64_t p = c / (2 * T);
        return 2 * p + (c - p * 2 * T >= TL ? 1 : 0);
    };
    int4 *units = ws_ptr<int4>(ws, lay.off_units);
    int2 *tinfo = ws_ptr<int2>(ws, lay.off_tinfo);
    uint32_t *slot = ws_ptr<uint32_t>(ws, lay.off_slot);
    int64_t ccarry = 0, ucarry = 0, pcarry = 0;
    for (int c = 0; c < tiles; c += 1024) {
        const int t = c + tid;
        const int4 n = t < tiles ? steps(t) : make_int4(0, 0, 0, 0);
        const int64_t w = t < tiles ? cost(n) : 0, cw = t < tiles ? w + E : 0;
        int64_t ctot, utot, ptot;
        const int64_t C = ccarry + block_excl_scan_1024(cw, &ctot);
        // ranges meeting the tile's cost; the last one starts inside the decode's share when
        // the last cut lies past the steps: it gets no piece
        const int nr = t < tiles ? (int)(range_of(C + cw - 1) - range_of(C) + 1) : 0;
        const int np = nr > 1 && cut(range_of(C + cw - 1)) >= C + w ? nr - 1 : nr;
        const int64_t U = ucarry + block_excl_scan_1024(np, &utot);
        const int64_t P = pcarry + block_excl_scan_1024(np > 1 ? np : 0, &ptot);
        if (t < tiles) {
            tinfo[t] = make_int2(np, np > 1 ? (int)P : -1);
            for (int p = 0; p < nr; ++p) {
                const int64_t s0 = range_of(C) + p;
                const int64_t a = p == 0 ? C : cut(s0), e = p == np - 1 ? C + w : cut(s0 + 1);
                if (p < np)
                    units[U + p] = make_int4(t, (int)step_at(n, a - C), (int)step_at(n, e - C),
                                             np > 1 ? (int)(P + p) : -1);
                // (a range starting inside the decode's share starts with the next tile's first unit)
                if (cut(s0) == a) slot[s0] = (uint32_t)(U + p);
            }
        }
        ccarry += ctot;
        ucarry += utot;
        pcarry += ptot;
    }
    // ranges past the end of the work hold no unit
    for (int64_t s = (W > 0 ? range_of(W - 1) + 1 : 0) + tid; s <= slots; s += 1024) slot[s] = (uint32_t)ucarry;
}

hipError_t launch_units(const sc_gemm_desc &d, const Layout &lay, uint8_t *ws, hipStream_t st) {
    hipLaunchKernelGGL(k_units, dim3(1), dim3(1024), 0, st, lay, d.batch, ws);
    return hipGetLastError();
}

hipError_t launch_schedule(const sc_gemm_desc &d, const Layout &lay, const int32_t *L, uint8_t *ws,
                           bool draws, hipStream_t st) {
    if (draws && d.batch != 1) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_schedule, dim3((unsigned)d.batch), dim3(1024), 0, st, L, d.strideL, d.M,
                       d.L_max, lay, ws, d.seed, d.rng, draws ? lay.LBS : 0);
    return hipGetLastError();
}

}  // namespace scg
