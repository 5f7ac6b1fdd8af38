// Internal definitions shared by the kernels and the host API of libscgemm.
//
// Data layout in device memory (all inside the caller's workspace):
//
//   status     one uint32 (bit 0: some L_i out of range), then one uint32: the longest
//              tile-pair cycle count of the call (256-row GEMM), then one uint32: nonzero
//              when some 256-row pair holds more distinct lengths that are not multiples of
//              32 than the int8-chunk GEMM has masked tables (rslots; it then masks its
//              fragments); all cleared by k_draws (or k_schedule); then one uint32: the
//              work units of the 256-row GEMM when their division follows the tile lengths
//              (written by k_units)
//   draws      rA[LBS], rB[LBS]                   uint32, comparator sequences
//   CA         C-BSG only: CA[L][beta] = #{l < L : rA_l < beta}, uint16 [L_max+1][257]
//   rtab       int8-chunk GEMM only: for each 32-cycle group G, the fp4 slot row of every
//              int8 byte for A and for B: uint4 [LBS/32][2][256] (built once per call)
//   per batch entry b of A (batch entries):
//     perm[MT*BM]      sorted position -> original row (or -1 for padding)
//     Ls[MT*BM]        stream length at each sorted position
//     tileL[MT]        cycles the GEMM runs for row tile t: the longest L of the tile (of
//                      the tile pair with 256-row blocks), rounded up to 8
//     tileOff[MT]      word offset of tile t's planes inside Ap
//     Ap               fp4 planes of A (or int8 chunks, below)
//   part       partial counts when GEMM tiles are split along the inner (element, cycle) range
//   units      vsplit only (k_units): the 256-row GEMM's work units {tile, first chunk step,
//              end chunk step, partial index or -1} (int4), per tile {pieces, partial index
//              of piece 0} (int2), and per GEMM block the first of its units (uint32,
//              sk_slots + 1 of them)
//   per batch entry of B (1 if B is broadcast, else batch entries):
//     Bp               fp4 planes of B (or int8 chunks)
//
// Each stream bit is an fp4 (e2m1) value in {-1, 0, +1} ("nibble planes").  A slot is
// (octet o of 8 cycles, element quad dq of 4 elements) and holds 16 bytes: dword e =
// element 4*dq+e, nibble c = cycle 8*o+c, with value +1 (0x2), -1 (0xA) or 0.  Slots are
// ordered s = o * KQP + dq and each slot stores its 128 rows contiguously: A tile t is
// uint4 [Lloop/8 * KQP][128], B tile is uint4 [LBS/8 * KQP][128].  A row of length L has
// zero nibbles at cycles >= L.
//
// 256 x 256 GEMM blocks with comparator streams (rgen): no planes.  Ap and Bp hold the int8
// operands in 32-element chunks instead: pair t of 256 rows (A in the scheduler's order) is
// bytes [KC][256][32], byte e of row r of chunk c = element 32c + e, with -128 read as -127
// (the same comparator boundaries) and 0x80 (-128) marking an element >= K or a padding
// row.  The GEMM builds the fp4 fragments from them.
//
// N <= 128 with comparator streams (fused): no planes either; the GEMM builds its fragments
// from the int8 rows themselves.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/scgemm.h"

static_assert(SC_KL_LIMIT == 8ll << 24, "K * L_max limit: MAX_SPLIT parts of 2^24 products");

namespace scg {

constexpr int BM = 128;          // rows of A per GEMM tile
constexpr int BN = 128;          // rows of B per GEMM tile
constexpr int LCH = 32;          // cycle granularity of the draw arrays and B's planes
constexpr uint32_t STATUS_BAD_LENGTH = 1u;
constexpr int DEFAULT_CUS = 256; // compute units of an MI355X, when no device can be queried
constexpr int MAX_SPLIT = 8;     // most parts a GEMM tile is split into along its inner range
constexpr int CBSG_L_MAX = 256;  // one period of the 8-bit Sobol sequences
constexpr int CA_COLS = 257;     // boundaries 0..256

constexpr int MSTEP = 8;         // cycles per octet (tile lengths padded to it)
constexpr int MSTAGE = 4;        // slots per LDS stage of the MFMA GEMM (2 MFMA k-steps)
constexpr int MFMA_BLOCKS_PER_CU = 2;   // resident 128-row MFMA GEMM blocks per CU (LDS bound)
constexpr double MFMA_QUAD_RATE = 1.1e13;  // products/s of one 256 x 256 GEMM block (one per CU)
constexpr double PART_BW = 3e12;           // bytes/s of writing and summing partial sums

// Estimated time of the 256-row GEMM with every tile split s ways (F = 0): the larger of
// the load per block slot and the longest unit, plus writing and summing the partial sums.  With
// one row length the units are equal and the load is whole rounds of them; with varying
// lengths the tiles come longest first, so the blocks fill in behind the long units and
// the load is the total over the CUs.  The host evaluates it with L_max, the GEMM kernels
// again with the longest tile pair of the call (both pick the same way among s).
__host__ __device__ inline double quad_split_time(int64_t tiles, int s, double perL, double Lmean,
                                                  double Lmax, bool one_length, int slots, double part_bytes) {
    const double avgT = perL * Lmean, maxT = perL * Lmax;
    const double load = one_length ? (double)((tiles * s + slots - 1) / slots) * avgT / s
                                   : (double)tiles * avgT / slots;
    const double red = s > 1 ? (double)tiles * (2 * s) * part_bytes / PART_BW + 5e-6 : 0.0;
    return (load > maxT / s ? load : maxT / s) + red;
}
constexpr int OCH = 8;           // octets per block of the nibble-plane generator
constexpr int RSLOTS = 4;        // int8-chunk GEMM: tables masked to a row length, per cycle group
constexpr int64_t MFMA_EXACT = 1ll << 24;   // products one fp32 accumulator sums exactly
// chunk steps whose counts fit int16: a step adds at most 32 x 32 products of magnitude 1 to a count
constexpr int64_t P16_STEPS = 32767 / (32 * 32);
constexpr int64_t RSTEP_EXACT = MFMA_EXACT / (32 * 32);   // int8-chunk GEMM chunk steps (32 cycles x
                                                          // 32 elements) one accumulator sums exactly
// Cost of a chunk step of the 256 x 64 int8-chunk GEMM in the work division, while all of a
// wave's row blocks run (RW1) and once only the first two do (RW2): half the MFMAs and two
// thirds of the table reads (measured on attention-V: 9/16 of a full step's time, against
// 8/16, 10/16 and 11/16); the 256 x 256 blocks weigh every step 1
constexpr int64_t RW1_NARROW = 16, RW2_NARROW = 9;
// ... and once only the first one does (RW3: one A read and two MFMAs per k-step, beside two B
// reads; measured on attention-V: 5/16 against 3, 4, 7 and 9); the smallest of the three
constexpr int64_t RW3_NARROW = 5;
// The 256 x 64 blocks run two per CU, and the one dispatched first issues first: of the two
// ranges of a CU's pair of blocks, the first one's is RLEAD_NARROW / 16 longer than the
// average and the second one's as much shorter, so that both end together
constexpr int64_t RLEAD_NARROW = 4;

__host__ __device__ inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

// comparator boundaries of an int8 value (bipolar, and unipolar magnitude).  -128 lies
// outside the quantiser's range; its boundaries equal those of -127 (0 bipolar, and a
// magnitude boundary at or above 256 unipolar: a one on every cycle), so the magnitude is
// capped at 127 and every boundary stays in [0, 256].
__device__ __forceinline__ int beta_bipolar(int q) { return (256 * (q + 127) + 127) / 254; }
__device__ __forceinline__ int beta_unipolar(int q) {
    const int a = q < 0 ? (q < -127 ? 127 : -q) : q;
    return (256 * a + 63) / 127;
}

__device__ __forceinline__ int wave_uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

template <typename T>
__device__ __forceinline__ T *ws_ptr(uint8_t *ws, size_t off) {
    return reinterpret_cast<T *>(ws + off);
}

struct Layout {
    int MT, NT;        // row tiles of A and B (NT rounded up to a multiple of mbn / 128, the
                       // B tiles one GEMM block takes)
    int LBS;           // cycle stride of B planes and length of draw arrays (L_max rounded to LCH)
    int nbB;           // batch entries of B planes (1 when B is broadcast)
    int KQP;           // element quads per octet, ceil(K/4) rounded up to 4
    int mbn;           // columns of B per GEMM block (256, or 128 when N <= 128)
    int fused;         // N <= 128, comparator streams: the GEMM builds its fp4 fragments from
                       // the int8 operands (no planes in the workspace)
    int mbm;           // rows of A per GEMM block: 256 (row tiles taken in pairs that run at
                       // the pair's longest length; MT even) when mbn = 256 and MT > 1, else 128
    int rgen;          // 256-row GEMM with comparator streams: fragments built in the GEMM
                       // from int8 chunks and a per-group table (no planes)
    int narrow;        // rgen with N <= 64: blocks of 256 rows x 64 columns
    int rslots;        // rgen: tables masked to a row length per cycle group (0 when narrow)
    int KC;            // 32-element chunks per row, ceil(K/32)
    int cus;           // compute units of the device the call runs on
    int64_t words_per_L;   // plane words of one 128-row tile per cycle of its length
    size_t off_rA, off_rB, off_status, off_CA, off_rtab;
    size_t off_perm, off_Ls, off_tileL, off_tileOff, off_Ap;
    size_t stride_batchA;          // bytes per A batch entry block
    size_t off_Bp;
    size_t stride_batchB;          // bytes per B batch entry block
    int S;             // splits of the inner range per GEMM tile (1 = no split)
    int Smin;          // fewest splits that keep every part's fp32 sums exact (<= 2^24 products)
    int F;             // 256-row GEMM: tiles 0 .. F-1 run whole, tiles F.. in S parts each
    double q_perL, q_Lmean;   // 256-row GEMM split model: seconds per cycle of one tile, mean L
    int q_one;                // 256-row GEMM split model: all rows have one length
    int q_slots;              // 256-row GEMM split model: blocks that run at once
    double q_pbytes;          // 256-row GEMM split model: partial-sum bytes of one part (the
                              // columns a block computes: 256, or 64 with N <= 64)
    size_t off_part;   // partial counts of split tiles: [pieces][256 rows][pcols columns] int32
    int pcols;         // columns of a piece of partial counts: 256, or 64 for the 256 x 64 blocks
    int p16;           // int8-chunk GEMM split into parts of at most P16_STEPS chunk steps: the
                       // partial counts are int16 ([pieces][256 rows][pcols columns])
    int vsplit;        // int8-chunk GEMM with varying lengths: the tiles' chunk steps, end to
                       // end, are cut into sk_slots equal ranges, one per GEMM block (k_units)
    int sk_slots;      // vsplit: GEMM blocks, each running one range of the work
    size_t off_units, off_tinfo, off_slot;
    size_t total;
};

// Host-side layout computation for a device with `cus` compute units (no HIP calls).
// Returns false on overflow or when no split count up to MAX_SPLIT keeps the counts exact.
bool make_layout(const sc_gemm_desc &d, int cus, Layout *lay);

// Kernel launchers (sc_kernels.hip).  All return hipSuccess or the launch error.
hipError_t launch_draws(uint64_t seed, int rng, int n, uint32_t *rA, uint32_t *rB,
                        uint8_t *bytes_out, int op_only, uint32_t *status, hipStream_t st);
hipError_t launch_cbsg_table(const uint32_t *rA, int L_max, uint16_t *CA, hipStream_t st);
// draws: also clear the status words and make the comparator sequences (one batch entry only)
hipError_t launch_schedule(const sc_gemm_desc &d, const Layout &lay, const int32_t *L,
                           uint8_t *ws, bool draws, hipStream_t st);
// the 256-row GEMM's work units from the scheduled tile lengths (Layout::vsplit)
hipError_t launch_units(const sc_gemm_desc &d, const Layout &lay, uint8_t *ws, hipStream_t st);

// counting GEMM (sc_mfma.hip)
// Profiling events of the next launch_mgemm / launch_fgemm on this host thread (sc_gemm's
// prof_event_begin / end, NULL = none): its first kernel records begin when it starts and
// every kernel records end when it ends (the last one's stays), so the events time the GEMM
// kernels themselves, with no marker of their own in the stream.  gemm_events_taken() tells
// whether a kernel took them since set_gemm_events.
void set_gemm_events(hipEvent_t begin, hipEvent_t end);
bool gemm_events_taken();
hipError_t launch_mplanes(const sc_gemm_desc &d, const Layout &lay, const int8_t *A,
                          const int8_t *B, uint8_t *ws, hipStream_t st);
hipError_t launch_mgemm(const sc_gemm_desc &d, const Layout &lay, const float *sA, const float *sB,
                        float *out, int32_t *counts, uint8_t *ws, hipStream_t st);
hipError_t launch_fgemm(const sc_gemm_desc &d, const Layout &lay, const int8_t *A, const int8_t *B,
                        const float *sA, const float *sB, float *out, int32_t *counts, uint8_t *ws,
                        hipStream_t st);
hipError_t launch_rchunks(const sc_gemm_desc &d, const Layout &lay, const int8_t *A, const int8_t *B,
                          uint8_t *ws, hipStream_t st);

// bytes of one batch entry of an operand from its first byte: (rows - 1) * ld + K
__host__ __device__ inline int64_t fused_extent(int rows, int64_t ld, int K) {
    return rows > 0 && K > 0 ? (int64_t)(rows - 1) * ld + K : 0;
}

// thresholds and ladder of the per-row length policy, passed by value to the kernel
struct MpParams {
    float tau[SC_MP_MAX_LEVELS];
    int32_t ladder[SC_MP_MAX_LEVELS];
    int32_t n;
};

// front end (sc_frontend.hip)
hipError_t launch_quantize(int batch, int rows, int K, const float *X, int64_t ldx, int64_t strideX,
                           int per_tensor, int8_t *Q, int64_t ldq, int64_t strideQ, float *scale,
                           float *rowmax, int64_t strideS, hipStream_t st);
hipError_t launch_mp_lengths(int batch, int M, const float *metric, int64_t strideM,
                             const MpParams &p, int32_t *L_out, int64_t strideL, hipStream_t st);

}  // namespace scg
