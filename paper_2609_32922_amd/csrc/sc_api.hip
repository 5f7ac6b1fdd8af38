// Host side of libscgemm: argument checks, workspace layout and the launch sequence.
// Every check runs before anything is enqueued; the library allocates nothing.
#include <limits.h>
#include <math.h>

#include <atomic>
#include <mutex>

#include "sc_internal.h"

namespace scg {

namespace {

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

// checked size arithmetic: returns false on overflow of size_t
bool mul_ok(size_t a, size_t b, size_t *r) {
    if (a != 0 && b > SIZE_MAX / a) return false;
    *r = a * b;
    return true;
}

}  // namespace

// Compute units of the current device (the width over which the GEMM's work is divided),
// cached per device; DEFAULT_CUS when no device can be queried (e.g. sizing a workspace on
// a host without a GPU).
static int device_cus() {
    static std::atomic<int> cache[64];
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) {
        (void)hipGetLastError();
        return DEFAULT_CUS;
    }
    if (dev < 64) {
        const int c = cache[dev].load(std::memory_order_relaxed);
        if (c > 0) return c;
    }
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) {
        (void)hipGetLastError();
        return DEFAULT_CUS;
    }
    if (dev < 64) cache[dev].store(n, std::memory_order_relaxed);
    return n;
}

bool make_layout(const sc_gemm_desc &d, int cus, Layout *lay) {
    Layout l{};
    l.cus = cus > 0 ? cus : DEFAULT_CUS;
    l.KQP = (int)round_up((d.K + 3) / 4, 4);
    l.words_per_L = (int64_t)l.KQP * 64;
    l.MT = (d.M + BM - 1) / BM;
    l.NT = (d.N + BN - 1) / BN;
    // N <= 64 with comparator streams and M > 128: the int8-chunk GEMM in blocks of
    // 256 rows x 64 columns (the B side still laid out as one 256-row pair)
    l.narrow = d.rng == SC_RNG_LFSR32 && d.N <= 64 && d.M > BM;
    l.mbn = (l.NT > 1 || l.narrow) ? 2 * BN : BN;
    l.NT = (int)round_up(l.NT, l.mbn / BN);
    // N <= 128 (one B tile): every A plane would be used once, so the GEMM generates the
    // fragments itself (comparator streams; operand offsets must fit 31 bits)
    l.fused = l.mbn == BN && d.rng == SC_RNG_LFSR32 && fused_extent(d.M, d.lda, d.K) < INT_MAX - 4 &&
              fused_extent(d.N, d.ldb, d.K) < INT_MAX - 4;
    l.mbm = (l.MT > 1 && l.mbn == 2 * BN) ? 2 * BM : BM;
    if (l.mbm == 2 * BM) l.MT = (int)round_up(l.MT, 2);
    // 256 x 256 blocks with comparator streams: fragments from int8 chunks and a table of
    // each 32-cycle group, so the operands are read as bytes instead of fp4 planes
    l.rgen = l.mbm == 2 * BM && d.rng == SC_RNG_LFSR32;
    l.rslots = l.narrow ? 0 : RSLOTS;
    l.KC = (d.K + 31) / 32;
    l.LBS = (int)round_up(d.L_max, LCH);
    l.nbB = (d.strideB == 0) ? 1 : d.batch;
    if (l.nbB < 1) l.nbB = 1;
    const bool cbsg = d.rng == SC_RNG_SOBOL8_CBSG;

    // the status word is always the first word of the workspace
    size_t off = 0;
    l.off_status = off;
    off = align256(off + 4 * 4);
    l.off_rA = off;
    off = align256(off + (size_t)l.LBS * 4);
    l.off_rB = off;
    off = align256(off + (size_t)l.LBS * 4);
    l.off_CA = off;
    if (cbsg) off = align256(off + (size_t)(d.L_max + 1) * CA_COLS * 2);
    l.off_rtab = off;
    if (l.rgen) off = align256(off + (size_t)(l.LBS / 32) * 512 * 16);

    // one A block per batch entry
    const size_t rowsA = (size_t)l.MT * BM;
    size_t a = 0, sz;
    l.off_perm = a;
    a = align256(a + rowsA * 4);
    l.off_Ls = a;
    a = align256(a + rowsA * 4);
    l.off_tileL = a;
    a = align256(a + (size_t)l.MT * 4);
    l.off_tileOff = a;
    a = align256(a + (size_t)l.MT * 8);
    l.off_Ap = a;
    // largest planes of one batch entry: every tile at L_max rounded up to an octet
    if (!mul_ok((size_t)l.MT * (size_t)l.words_per_L, (size_t)round_up(d.L_max, MSTEP) * 4, &sz))
        return false;
    if (l.fused) sz = 0;
    if (l.rgen && !mul_ok(rowsA, (size_t)l.KC * 32, &sz)) return false;
    a = align256(a + sz);
    l.stride_batchA = a;
    const size_t baseA = off;
    size_t totA;
    if (!mul_ok(a, (size_t)(d.batch > 0 ? d.batch : 0), &totA)) return false;
    off += totA;

    // one B block per distinct B batch entry
    const size_t rowsB = (size_t)l.NT * BN;
    size_t bb = 0;
    l.off_Bp = bb;
    if (!mul_ok((size_t)l.NT * (size_t)l.words_per_L, (size_t)l.LBS * 4, &sz)) return false;
    if (l.fused) sz = 0;
    if (l.rgen && !mul_ok(rowsB, (size_t)l.KC * 32, &sz)) return false;
    bb = align256(bb + sz);
    l.stride_batchB = bb;
    const size_t baseB = off;
    size_t totB;
    if (!mul_ok(bb, (size_t)l.nbB, &totB)) return false;
    off += totB;

    // Exactness of the counts: a GEMM part sums its products into fp32 accumulators, which
    // stay exact integers while a part holds at most 2^24 products per output.  Units of the
    // inner range and products per unit of each GEMM: (32-cycle group, 32-element chunk) =
    // 1024 (int8-chunk GEMM); stage of 4 slots = 128 (fused GEMM); k-step of 2 slots = 64.
    // A part takes at most ceil(units / S) units, so S is at least Smin; the parts' int32
    // partial sums are then added exactly.
    const int64_t octs = round_up(d.L_max, MSTEP) / MSTEP;
    const int64_t units = l.rgen ? (int64_t)(l.LBS / 32) * l.KC
                                 : l.fused ? octs * (l.KQP / MSTAGE) : octs * (l.KQP / 2);
    const int64_t per_unit = l.rgen ? 32 * 32 : l.fused ? 128 : 64;
    l.Smin = 1;
    while (l.Smin <= MAX_SPLIT && (units + l.Smin - 1) / l.Smin * per_unit > MFMA_EXACT) l.Smin *= 2;
    if (l.Smin > MAX_SPLIT) return false;

    // Division of the GEMM tiles into work units.
    const bool quad = l.mbm == 2 * BM;
    const int64_t tiles = (int64_t)(d.batch > 0 ? d.batch : 0) * (l.MT / (l.mbm / BM)) * (l.NT / (l.mbn / BN));
    // indivisible steps along the inner range per cycle (chunks of every 32-cycle group with rgen)
    const int kunits = l.rgen ? l.KC * (l.LBS / 32) : l.KQP / 2;
    const int smax = kunits > l.Smin ? kunits : l.Smin;
    // partial-sum bytes of one part (256-row blocks of N <= 64 compute 64 columns)
    const double tile_bytes = (double)l.mbm * (l.narrow ? 64 : l.mbn) * 4.0;
    const double Lmean = d.L_hint > 0 ? d.L_hint : d.L_max;
    l.S = l.Smin;
    l.F = 0;
    if (quad && tiles > 0) {
        // 256 x 256 tiles, one block per CU, taking whole tiles or parts of tiles
        // (quad_split_time).  Candidates: every tile split s ways (F = 0), or whole tiles in
        // full rounds with the tiles of a last partial round split to fill one round.  Split
        // counts are powers of two: units are dealt to the eight XCDs round-robin, so each
        // XCD then holds units of one k-range, whose operand slots its blocks read
        // together from its L2 (three-way splits measured slower than four-way).  With
        // F = 0 the GEMM kernels may lower s again with the actual longest tile pair
        // (measured: 6304 x 768 x 3072 with L in [16, 256], mean 64, longest 172: the GEMM
        // takes 0.49 ms split two ways against 0.61 ms three ways), never below Smin.
        // (the 64-column blocks of N <= 64 do a quarter of the work and run two per CU)
        l.q_perL = (double)l.mbm * (l.narrow ? 64 : l.mbn) * 4.0 * l.KQP / MFMA_QUAD_RATE;
        l.q_slots = l.narrow ? 2 * l.cus : l.cus;
        l.q_Lmean = Lmean;
        l.q_pbytes = tile_bytes;
        l.q_one = Lmean >= d.L_max;
        const double avgT = l.q_perL * Lmean, maxT = l.q_perL * d.L_max;
        double best = 0.0;
        for (int s = l.Smin; s <= MAX_SPLIT && s <= smax; s *= 2) {
            const double est = quad_split_time(tiles, s, l.q_perL, Lmean, d.L_max, l.q_one != 0, l.q_slots,
                                               l.q_pbytes);
            if (s == l.Smin || est < best * 0.97) {
                best = est;
                l.S = s;
            }
        }
        // (the tail's split fills the last round as closely as it can: its units are few
        // and short, so balance counts for more there than a shared k-range per XCD)
        const int64_t R = tiles % l.q_slots;
        int s2 = R > 0 ? (int)(l.q_slots / R) : 1;
        s2 = s2 > MAX_SPLIT ? MAX_SPLIT : s2;
        if (s2 > kunits) s2 = kunits;
        if (l.Smin == 1 && tiles >= l.q_slots && R > 0 && s2 > 1) {
            const double red = (double)R * (2 * s2) * tile_bytes / PART_BW + 5e-6;
            const double est = fmax((double)(tiles / l.q_slots) * avgT + avgT / s2, maxT) + red;
            if (est < best * 0.97) {
                best = est;
                l.F = (int)(tiles - R);
                l.S = s2;
            }
        }
        if (l.S == 1) l.F = (int)tiles;
    } else if (tiles > 0 && kunits > 1) {
        // 128-row tiles: every tile split s ways.  Estimated time of split s: the busiest
        // slot (a resident block) runs ceil(units/slots) units of average work, plus the
        // excess of the heaviest unit over the average, plus, for s > 1, writing and summing
        // s partial tiles.  Units are dealt to the eight XCDs round-robin, so s is a power of
        // two: each XCD then keeps one k-range of its tiles, and its L2 serves that range to
        // all of them.  Rates are the measured order of magnitude: 4.8e12 products/s per
        // resident block (two per CU); partial sums at 3e12 B/s.
        const int slots = l.cus * MFMA_BLOCKS_PER_CU;
        const double rate = 4.8e12;
        const double per_L = (double)BM * l.mbn * 4.0 * l.KQP;
        double best = 0.0;
        for (int s = l.Smin; s <= MAX_SPLIT && s <= smax; s *= 2) {
            const int64_t nunits = tiles * s;
            const double avg_u = per_L * Lmean / s, max_u = per_L * d.L_max / s;
            const double gemm = ((double)((nunits + slots - 1) / slots) * avg_u + (max_u - avg_u)) / rate;
            const double red = s > 1 ? (double)tiles * (2 * s) * tile_bytes / 3e12 + 5e-6 : 0.0;
            if (s == l.Smin || gemm + red < best * 0.97) {
                best = gemm + red;
                l.S = s;
            }
        }
    }
    // Int8-chunk GEMM with varying lengths: the work of a tile follows its rows' lengths
    // (Sec. 4.1: the cost follows the sum of the l_i), known only on the device.  There the
    // tiles' chunk steps are laid end to end and cut into sk_slots equal ranges, one per GEMM
    // block (k_units): a tile inside a range runs whole, one that a cut crosses runs in
    // pieces that the split-sum pass adds.  A range holds at most RSTEP_EXACT steps, so every
    // whole tile and piece sums exactly.
    // (Short tiles, a few chunk steps each, keep the division below: their pieces' partial sums
    // and their in-GEMM decodes would cost as much as the steps; ViT-L/14 Q.K^T heads with
    // K = 64 took 0.61 ms cut into ranges against 0.41 ms split alike.)
    l.pcols = l.narrow ? 64 : l.mbn;
    l.vsplit = quad && l.rgen && tiles > 0 && !l.q_one &&
               (int64_t)l.KC * ((int64_t)(Lmean + 31) / 32) >= 16;
    l.off_units = off;
    int64_t pieces = quad ? (tiles - l.F) * (int64_t)l.S : tiles * (int64_t)l.S;
    if (l.vsplit) {
        // (k_units weighs a step at most w1 and at least w2 and adds at most 7 w1 per tile for
        // its decode and a minimum step: W <= w1 wmax.  A range of cost T = ceil(W / sl) <=
        // w1 wmax / sl + 1 holds at most T / w2 + 1 steps, which must stay below RSTEP_EXACT;
        // the 256 x 64 blocks' ranges hold up to twice T.)
        const int64_t w1 = l.narrow ? RW1_NARROW : 1, w2 = l.narrow ? RW3_NARROW : 1;   // (w2: the lightest step)
        const int64_t wmax = tiles * ((int64_t)l.KC * (l.LBS / 32) + 7);
        const int64_t den = (w2 * (RSTEP_EXACT - 2) - 1) / (l.narrow ? 2 : 1);
        int64_t sl = l.q_slots;
        if (w1 * wmax > sl * den) sl = (w1 * wmax + den - 1) / den;
        if (sl > (1 << 20)) return false;
        l.sk_slots = (int)sl;
        l.F = 0;
        l.S = 1;
        off = align256(off + (size_t)(tiles + sl) * 16);
        l.off_tinfo = off;
        off = align256(off + (size_t)tiles * 8);
        l.off_slot = off;
        off = align256(off + (size_t)(sl + 1) * 4);
        // a cut inside a tile adds one piece to it and may make it a split tile: at most two
        // pieces per cut
        pieces = 2 * sl;
    }
    // Parts of the int8-chunk GEMM's split tiles of at most P16_STEPS chunk steps store int16
    // partial counts (half the partial-sum traffic).  A part of S has at most ceil(steps / S)
    // of a tile's steps; with F = 0 the GEMM may lower S to Smin.
    if (l.rgen && !l.vsplit && l.S > 1) {
        const int64_t smin = l.F > 0 ? l.S : l.Smin;
        const int64_t steps = (int64_t)l.KC * (l.LBS / 32);
        l.p16 = (steps + smin - 1) / smin <= P16_STEPS;
    }
    l.off_part = off;
    if (pieces > 0 && (l.S > 1 || l.vsplit)) {
        size_t partb;
        // every piece is [mbm rows][pcols columns] of int32 (int16 with p16)
        if (!mul_ok((size_t)pieces, (size_t)l.mbm * (size_t)l.pcols * (l.p16 ? 2 : 4), &partb)) return false;
        off = align256(off + partb);
    }

    // make every offset absolute for batch entry 0
    l.off_perm += baseA;
    l.off_Ls += baseA;
    l.off_tileL += baseA;
    l.off_tileOff += baseA;
    l.off_Ap += baseA;
    l.off_Bp += baseB;
    l.total = off;
    *lay = l;
    return true;
}

static int check_desc(const sc_gemm_desc *d) {
    if (d == nullptr) return SC_ERR_NULL;
    if (d->batch < 0 || d->M < 0 || d->N < 0 || d->K < 0 || d->K > SC_K_LIMIT) return SC_ERR_SHAPE;
    if (d->L_max < 1 || d->L_max > SC_L_MAX_LIMIT) return SC_ERR_LEN;
    // the counts stay exact: at most MAX_SPLIT parts of at most 2^24 products each
    if ((int64_t)d->K * d->L_max > SC_KL_LIMIT) return SC_ERR_SHAPE;
    if (d->polarity != SC_BIPOLAR_XNOR && d->polarity != SC_UNIPOLAR_AND_SM) return SC_ERR_POLARITY;
    if (d->rng != SC_RNG_LFSR32 && d->rng != SC_RNG_SOBOL8_CBSG) return SC_ERR_RNG;
    if (d->rng == SC_RNG_SOBOL8_CBSG && d->L_max > CBSG_L_MAX) return SC_ERR_LEN;
    if (d->L_hint < 0 || d->L_hint > d->L_max) return SC_ERR_LEN;
    if (d->reserved != 0) return SC_ERR_RESERVED;
    if (d->lda < d->K || d->ldb < d->K || d->ldo < d->N) return SC_ERR_STRIDE;
    if (d->strideA < 0 || d->strideB < 0 || d->strideO < 0 || d->strideSA < 0 || d->strideSB < 0 ||
        d->strideL < 0)
        return SC_ERR_STRIDE;
    // distinct batch entries must not overlap in the output: either each entry's block
    // lies before the next one (blocked), or the entries sit side by side in the columns
    // of one row stride (interleaved, e.g. per-head outputs of one token matrix)
    if (d->batch > 1 && d->M > 0 && d->N > 0) {
        const bool blocked = d->strideO >= (int64_t)(d->M - 1) * d->ldo + d->N;
        const bool interleaved = d->strideO >= d->N && (int64_t)(d->batch - 1) * d->strideO + d->N <= d->ldo;
        if (!blocked && !interleaved) return SC_ERR_STRIDE;
    }
    return SC_OK;
}

// Checks of one call (before anything is enqueued) and its workspace layout.
static int check_call(const sc_gemm_desc *desc, const int8_t *A, const float *sA, const int8_t *B,
                      const float *sB, const int32_t *L_per_row, const float *out, Layout *lay) {
    const int rc = check_desc(desc);
    if (rc != SC_OK) return rc;
    const sc_gemm_desc &d = *desc;
    // a descriptor whose workspace cannot be laid out is refused as sc_gemm_workspace_size refuses it
    if (!make_layout(d, device_cus(), lay)) return SC_ERR_SHAPE;
    // a pointer may be NULL only when the array it points to has no elements
    const bool anyM = d.batch > 0 && d.M > 0, anyN = d.batch > 0 && d.N > 0;
    if ((anyM && d.K > 0 && A == nullptr) || (anyN && d.K > 0 && B == nullptr) ||
        (anyM && (sA == nullptr || L_per_row == nullptr)) || (anyN && sB == nullptr) ||
        (anyM && anyN && out == nullptr))
        return SC_ERR_NULL;
    return SC_OK;
}

// The launch sequence of one call on workspace ws (lay.total bytes, 256-byte aligned).
static int enqueue(const sc_gemm_desc &d, const Layout &lay, const int8_t *A, const float *sA, const int8_t *B,
                   const float *sB, const int32_t *L_per_row, float *out, int32_t *counts, uint8_t *ws,
                   hipStream_t st) {
    uint32_t *rA = reinterpret_cast<uint32_t *>(ws + lay.off_rA);
    // one batch entry with LFSR sequences: the scheduler's single block also clears the
    // status and makes the sequences (one launch fewer); otherwise k_draws does, first
    const bool empty = d.batch == 0 || d.M == 0 || d.N == 0;
    const bool fuse = !empty && d.batch == 1 && d.rng == SC_RNG_LFSR32;
    hipError_t e = hipSuccess;
    if (!fuse) {
        e = launch_draws(d.seed, d.rng, lay.LBS, rA, reinterpret_cast<uint32_t *>(ws + lay.off_rB), nullptr, -1,
                         reinterpret_cast<uint32_t *>(ws + lay.off_status), st);
        if (e != hipSuccess) return SC_ERR_HIP;
    }
    if (empty) return SC_OK;

    if (d.rng == SC_RNG_SOBOL8_CBSG &&
        launch_cbsg_table(rA, d.L_max, reinterpret_cast<uint16_t *>(ws + lay.off_CA), st) != hipSuccess)
        return SC_ERR_HIP;
    if ((e = launch_schedule(d, lay, L_per_row, ws, fuse, st)) != hipSuccess) return SC_ERR_HIP;
    if (lay.vsplit && (e = launch_units(d, lay, ws, st)) != hipSuccess) return SC_ERR_HIP;
    if (lay.rgen) {
        if ((e = launch_rchunks(d, lay, A, B, ws, st)) != hipSuccess) return SC_ERR_HIP;
    } else if (!lay.fused) {
        if ((e = launch_mplanes(d, lay, A, B, ws, st)) != hipSuccess) return SC_ERR_HIP;
    }
    // the profiling events ride on the GEMM kernels' own dispatches (a marker of their own
    // in the stream left an idle gap of several microseconds after it); recorded as markers
    // only if no GEMM kernel was launched
    hipEvent_t ev0 = reinterpret_cast<hipEvent_t>(d.prof_event_begin);
    hipEvent_t ev1 = reinterpret_cast<hipEvent_t>(d.prof_event_end);
    set_gemm_events(ev0, ev1);
    e = lay.fused ? launch_fgemm(d, lay, A, B, sA, sB, out, counts, ws, st)
                  : launch_mgemm(d, lay, sA, sB, out, counts, ws, st);
    const bool taken = gemm_events_taken();
    set_gemm_events(nullptr, nullptr);
    if (e != hipSuccess) return SC_ERR_HIP;
    if (!taken && ev0 != nullptr && hipEventRecord(ev0, st) != hipSuccess) return SC_ERR_HIP;
    if (!taken && ev1 != nullptr && hipEventRecord(ev1, st) != hipSuccess) return SC_ERR_HIP;
    return SC_OK;
}

// The workspace of sc_gemm_noalloc: a static device array, one copy per device, held until
// the process ends.  Host code never uses its name as an address: the device address of
// each device's copy is looked up once (hipGetSymbolAddress, with that device current) and
// kept per device.
static __device__ __align__(256) uint8_t scratch[SC_NOALLOC_WORKSPACE_BYTES];

static bool scratch_address(uint8_t **ptr) {
    constexpr int MAXDEV = 64;
    static std::mutex mu;
    static uint8_t *addr[MAXDEV] = {};
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAXDEV) return false;
    std::lock_guard<std::mutex> lock(mu);
    if (addr[dev] == nullptr) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr ||
            (reinterpret_cast<uintptr_t>(p) & 255u) != 0)
            return false;
        addr[dev] = static_cast<uint8_t *>(p);
    }
    *ptr = addr[dev];
    return true;
}

}  // namespace scg

using namespace scg;

extern "C" {

int sc_version(void) { return 10200; }

const char *sc_strerror(int code) {
    switch (code) {
        case SC_OK: return "SC_OK";
        case SC_ERR_NULL: return "SC_ERR_NULL: a required pointer is NULL";
        case SC_ERR_SHAPE: return "SC_ERR_SHAPE: bad batch/M/N/K (or K*L_max above 2^27)";
        case SC_ERR_LEN:
            return "SC_ERR_LEN: L_max outside [1, SC_L_MAX_LIMIT] ([1, 256] for C-BSG) or L_hint "
                   "outside [0, L_max]";
        case SC_ERR_POLARITY: return "SC_ERR_POLARITY: unknown polarity";
        case SC_ERR_RNG: return "SC_ERR_RNG: unknown rng or operand index";
        case SC_ERR_WORKSPACE: return "SC_ERR_WORKSPACE: workspace missing or too small";
        case SC_ERR_HIP: return "SC_ERR_HIP: a HIP call or kernel launch failed";
        case SC_ERR_DEVICE_STATUS: return "SC_ERR_DEVICE_STATUS: some L_i outside [0, L_max]";
        case SC_ERR_STRIDE: return "SC_ERR_STRIDE: a stride is too small or negative";
        case SC_ERR_RESERVED: return "SC_ERR_RESERVED: the reserved descriptor field is not 0";
        default: return "unknown status code";
    }
}

int sc_gemm_workspace_size(const sc_gemm_desc *desc, size_t *bytes) {
    if (bytes == nullptr) return SC_ERR_NULL;
    const int rc = check_desc(desc);
    if (rc != SC_OK) return rc;
    Layout lay;
    if (!make_layout(*desc, device_cus(), &lay)) return SC_ERR_SHAPE;
    *bytes = lay.total;
    return SC_OK;
}

int sc_gemm(const sc_gemm_desc *desc, const int8_t *A, const float *sA, const int8_t *B,
            const float *sB, const int32_t *L_per_row, float *out, int32_t *counts, void *workspace,
            size_t workspace_bytes, void *stream) {
    Layout lay;
    const int rc = check_call(desc, A, sA, B, sB, L_per_row, out, &lay);
    if (rc != SC_OK) return rc;
    if (workspace == nullptr || workspace_bytes < lay.total ||
        (reinterpret_cast<uintptr_t>(workspace) & 255u) != 0)
        return SC_ERR_WORKSPACE;
    return enqueue(*desc, lay, A, sA, B, sB, L_per_row, out, counts, reinterpret_cast<uint8_t *>(workspace),
                   reinterpret_cast<hipStream_t>(stream));
}

int sc_gemm_noalloc(const sc_gemm_desc *desc, const int8_t *A, const float *sA, const int8_t *B,
                    const float *sB, const int32_t *L_per_row, float *out, int32_t *counts,
                    int32_t *status_out, void *stream) {
    Layout lay;
    const int rc = check_call(desc, A, sA, B, sB, L_per_row, out, &lay);
    if (rc != SC_OK) return rc;
    if (lay.total > SC_NOALLOC_WORKSPACE_BYTES) return SC_ERR_WORKSPACE;
    uint8_t *ws = nullptr;
    if (!scratch_address(&ws)) return SC_ERR_HIP;
    hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    const int e = enqueue(*desc, lay, A, sA, B, sB, L_per_row, out, counts, ws, st);
    if (e != SC_OK) return e;
    // the status word (offset 0 of every workspace) of this call, for the caller
    if (status_out != nullptr &&
        hipMemcpyAsync(status_out, ws, sizeof(int32_t), hipMemcpyDeviceToDevice, st) != hipSuccess)
        return SC_ERR_HIP;
    return SC_OK;
}

int sc_gemm_status(const void *workspace, void *stream) {
    if (workspace == nullptr) return SC_ERR_NULL;
    hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    if (hipStreamSynchronize(st) != hipSuccess) return SC_ERR_HIP;
    uint32_t word = 0;
    if (hipMemcpy(&word, workspace, sizeof(word), hipMemcpyDeviceToHost) != hipSuccess)
        return SC_ERR_HIP;
    return (word & STATUS_BAD_LENGTH) ? SC_ERR_DEVICE_STATUS : SC_OK;
}

int sc_quantize(int32_t batch, int32_t rows, int32_t K, const float *X, int64_t ldx,
                int64_t strideX, int32_t per_tensor, int8_t *Q, int64_t ldq, int64_t strideQ,
                float *scale, float *rowmax, int64_t strideS, void *stream) {
    if (batch < 0 || rows < 0 || K < 0 || K > SC_K_LIMIT) return SC_ERR_SHAPE;
    if (per_tensor != 0 && per_tensor != 1) return SC_ERR_SHAPE;
    if (ldx < K || ldq < K || strideX < 0 || strideQ < 0 || strideS < 0) return SC_ERR_STRIDE;
    if (batch > 1 && rows > 0 && strideS < rows) return SC_ERR_STRIDE;
    if (batch == 0 || rows == 0) return SC_OK;
    if ((K > 0 && (X == nullptr || Q == nullptr)) || scale == nullptr) return SC_ERR_NULL;
    hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    if (launch_quantize(batch, rows, K, X, ldx, strideX, per_tensor, Q, ldq, strideQ, scale, rowmax,
                        strideS, st) != hipSuccess)
        return SC_ERR_HIP;
    return SC_OK;
}

int sc_mp_lengths(int32_t batch, int32_t M, const float *metric, int64_t strideM,
                  const float *tau, const int32_t *ladder, int32_t n_levels, int32_t *L_out,
                  int64_t strideL, void *stream) {
    if (batch < 0 || M < 0) return SC_ERR_SHAPE;
    if (n_levels < 1 || n_levels > SC_MP_MAX_LEVELS) return SC_ERR_LEN;
    if (ladder == nullptr || (n_levels > 1 && tau == nullptr)) return SC_ERR_NULL;
    MpParams p{};
    p.n = n_levels;
    for (int k = 0; k < n_levels; ++k) {
        if (ladder[k] < 0 || ladder[k] > SC_L_MAX_LIMIT || (k > 0 && ladder[k] >= ladder[k - 1]))
            return SC_ERR_LEN;
        p.ladder[k] = ladder[k];
    }
    for (int k = 0; k + 1 < n_levels; ++k) {
        if (!(tau[k] >= 0.0f && tau[k] <= 1.0f) || (k > 0 && tau[k] > tau[k - 1])) return SC_ERR_LEN;
        p.tau[k] = tau[k];
    }
    if (strideM < 0 || strideL < 0 || (batch > 1 && M > 0 && (strideM < M || strideL < M)))
        return SC_ERR_STRIDE;
    if (batch == 0 || M == 0) return SC_OK;
    if (metric == nullptr || L_out == nullptr) return SC_ERR_NULL;
    if (launch_mp_lengths(batch, M, metric, strideM, p, L_out, strideL,
                          reinterpret_cast<hipStream_t>(stream)) != hipSuccess)
        return SC_ERR_HIP;
    return SC_OK;
}

int sc_comparator_sequence(uint64_t seed, int32_t op, int32_t rng, int32_t n, uint8_t *out,
                           void *stream) {
    if (out == nullptr) return SC_ERR_NULL;
    if ((op != 0 && op != 1) || (rng != SC_RNG_LFSR32 && rng != SC_RNG_SOBOL8_CBSG))
        return SC_ERR_RNG;
    if (n < 1 || n > (rng == SC_RNG_SOBOL8_CBSG ? CBSG_L_MAX : SC_L_MAX_LIMIT)) return SC_ERR_LEN;
    hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    if (launch_draws(seed, rng, n, nullptr, nullptr, out, op, nullptr, st) != hipSuccess)
        return SC_ERR_HIP;
    return SC_OK;
}

}  // extern "C"
