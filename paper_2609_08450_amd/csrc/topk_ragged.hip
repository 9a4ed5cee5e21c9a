// Exact Top-K over ragged FP32 rows for gfx950 (wave64): kernels and C-ABI.
//
// One kernel launch per call.  Work item = (row r, segment p); blockIdx.x =
// p * n_rows + r, so every row's first segment is dispatched before any
// second segment.  Each item is one 512-thread workgroup.  A call whose rows
// each take one workgroup and outnumber the resident workgroups (at most
// 16384 rows) first runs a one-workgroup pre-pass that orders the rows
// longest first; blockIdx.x then indexes that order.
//
//   L <= K            segment 0 writes the direct layout (Section 2.1).
//   not sampled       segment 0 runs exact coarse recovery alone
//                     (eq:method:exact-init): coarse histogram pass, classify
//                     pass, refinement.
//   sampled, 1 seg    Phase 1 (view histogram, eq:method:sample-hist and
//                     eq:method:primary-threshold) -> Phase 2 (complete-row
//                     certify + compact, eq:method:candidate-set) -> band or
//                     exact recovery when underfilled -> Phase 3 refinement.
//   sampled, P segs   segment 0 runs Phase 1 and publishes the endpoints
//                     (a large view is shared: each segment histograms its
//                     own part, the last to add publishes); every segment
//                     certifies and compacts its contiguous part of the row
//                     (eq:method:split-local); the last segment to arrive
//                     merges the candidate ranges (eq:method:split-reduce)
//                     and finishes the row.
//
// Keys: asc = order-preserving uint32 of the FP32 bits; the descending key
// kappa32 = ~asc (Section 4.3) is what the radix digits are taken from.  The
// refinement orders the composite key (kappa32, index), so ties at rank K go
// to the lowest index: the result is the K smallest composite keys.

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <climits>
#include <cstdlib>
#include <mutex>
#include <type_traits>

#include "../../include/topk_ragged.h"

namespace {

constexpr int kBlock = 512;                 // threads per workgroup (8 waves)
constexpr int kBins = 2048;                 // 11-bit digits and coarse bins
constexpr int kWaves = kBlock / 64;
constexpr int kCap = TOPK_FRONTIER_CAP;     // largest policy frontier (pairs)
constexpr int kFront = 7168;                // LDS frontier storage (pairs)
// Phase 2 region of a wave: kWaveCap entries, one spill slot, and 64 slots
// (one per lane) that take the writes of lanes without a hit
constexpr int kWaveStride = kFront / kWaves;
constexpr int kWaveCap = kWaveStride - 1 - 64;
static_assert(kCap <= kFront, "policy capacity must fit the storage");
constexpr int kVec = 4;                     // 16-byte loads per thread per chunk
static_assert(kVec * 4 <= 64, "per-thread element masks are 64-bit");
static_assert(kFront % kBlock == 0 && kFront % kWaves == 0, "frontier layout");
constexpr int kPer = kFront / kBlock;       // frontier slots per thread
constexpr int kChunkVecs = kBlock * kVec;   // 16-byte vectors per chunk
constexpr int kMaxSplit = 64;               // most segments per row
constexpr int kSegMin = 8192;               // shortest segment, elements
constexpr uint32_t kMagic = 0x544F504Bu;    // workspace header tag
constexpr int kSpinLimit = 1 << 15;         // polls before recomputing the view
constexpr int kSpinMicros = 100;            // and the longest wait for the boundaries
constexpr size_t kHeaderBytes = 1024;
constexpr size_t kRowStateBytes = 256;
constexpr uintptr_t kWorkspaceAlign = 256; // 64-bit atomics and 16-byte header loads
// a split row's merged view histogram; its merged coarse histogram of the
// segments whose candidates overflowed has the same size and sits in a
// region of its own after the row blocks (so that the blocks keep their
// 64 KB + 256 B stride: with the histogram inside them the decode batch ran
// 10 % slower)
constexpr size_t kViewHistBytes = kBins * sizeof(uint32_t);
constexpr size_t kRowBlockBytes = kRowStateBytes + kViewHistBytes + 2 * kFront * sizeof(uint32_t);
// Views of at least this many samples are shared by a split row's segments
// (each histograms the samples inside its own range and the histograms are
// merged): one workgroup gathering them all is bound by its cache-line
// fills (one 128-byte line per 4-byte sample).
constexpr int64_t kCoopView = 4096;
// The same for rows the item table cuts: their segments start among a whole
// call's first loads, where segment 0 alone took 15-20 us to gather a view of
// 1000-2000 samples (edge mix 76.9 -> 74.8 us per call from 1024; from 512
// 75.7, from 2048 unchanged).
constexpr int64_t kCoopViewTable = 1024;
// Most segments a row may have for its segments to publish per wave.
constexpr int64_t kWavePublishMaxSegs = 16;
// Calls with more rows than can be resident run their rows longest first: a
// pre-pass writes the work items, one 16-byte entry (row, segment, segments,
// length, offset, row-state slot) each, into a fixed region after the header,
// for calls of up to kOrderMaxRows rows.  Among the kOrderBlock longest rows,
// those much longer than the call's mean work per resident workgroup are cut
// into segments, at most kOrderExtra more items per call.
constexpr int kOrderMaxRows = 16384;
constexpr int kOrderExtra = 1024;
constexpr size_t kOrderBytes = (size_t)(kOrderMaxRows + kOrderExtra) * 16;
constexpr int kOrderBlock = 1024;
constexpr int kOrderPer = kOrderMaxRows / kOrderBlock;

typedef float f4 __attribute__((ext_vector_type(4)));

// Per-row state of a split row.  The row in slot k (its index r when every
// row may be split, else the slot the item table gives it) owns the workspace
// block at kHeaderBytes + kOrderBytes + k * kRowBlockBytes: this state, padded
// to 256 bytes, the 2048-bin view histogram that segments sharing the view add
// into, then kFront candidates as 64-bit (index | FP32 bits << 32) words
// (the segments' A(tau1) entries, concatenated); and the 2048-bin coarse
// histogram at kHeaderBytes + kOrderBytes + split_rows * kRowBlockBytes +
// k * kViewHistBytes.  Every field and entry is written and read with
// agent-scope atomic accesses (see the arrive step).
struct RowState {
    uint64_t sa;         // entries reserved in the candidate buffer (low 32
                         // bits) | segments done with Phase 2 << 32: the last
                         // arrival's atomic returns the final reserved count
    uint64_t counts;     // C(tau1) | C(tau0) << 32 of the row (exact)
    uint32_t taus;       // segment 0's tau0 | tau1 << 16 | 1 << 31 once known
    uint32_t incomplete; // a segment could not keep all of its A(tau1): with
                         // per-wave publishing 1, else the number of such
                         // segments (each adds its coarse histogram)
    uint32_t amax;       // largest ascending key among the stored entries
    uint32_t varrive;    // segments that have added their part of a shared view
    // The split exact route (segments that added a histogram wait for the
    // finisher's tau_star, classify their own ranges and arrive again):
    uint32_t ocnt;       // outputs reserved (entries with c < tau_star)
    uint32_t qcnt;       // kept entries (c == tau_star) reserved in the candidate buffer
    uint32_t arrive2;    // second arrivals
    uint64_t xtau;       // the route word: tau_star | arrivals expected << 11 |
                         // abandoned << 30 | 1 << 31 | |Q0| << 32 | |E0| << 48
    uint64_t xmask;      // segments that stopped waiting
};

// Workspace header (first kHeaderBytes of the workspace).
struct WsHeader {
    uint32_t magic;
    uint32_t split_rows; // rows with per-row state
    uint32_t max_rows;
    uint32_t cap;
    uint32_t pad[12];
    uint32_t stats[16]; // [0..5] routes, [6] reread, [7] wait fallback, [8] errors
};

enum { kStatReread = 6, kStatWaitFallback = 7, kStatErrors = 8 };

struct KArgs {
    const float *scores;
    const int64_t *offs;
    const int32_t *lens;
    int32_t *out_idx;
    float *out_val;
    int32_t *trace;
    WsHeader *hdr;
    char *rows;     // per-row blocks of kRowBlockBytes
    const uint4 *order; // rows longest first (row, length, offset), or NULL: item = row
    int32_t n_rows;
    int32_t K;
    int32_t pmax;
    int32_t seg_items; // split rows: aim for about this many (row, segment) items
    int32_t s_log2;
    int32_t q0, q1;
    int32_t l_samp_min;
    int32_t cap;
    int32_t spin_limit; // polls of the boundary word before a segment builds the view itself
    uint32_t spin_ticks; // and the most constant-rate clock ticks it waits for them
#ifdef TOPK_PHASE_TIMERS
    uint64_t *timers; // 32 words per workgroup, see PHASE_MARK
#endif
};

// Optional phase timers (built only with -DTOPK_PHASE_TIMERS): thread 0 of
// each workgroup stamps the constant-rate clock at fixed points of the row
// pipeline: 0 start, 1 endpoints known, 2 Phase 2 done, 3 arrived, 4 finisher
// has the merged frontier, 5 row done; word 6 = hardware id, 7 = role;
// 8 finish entered, 9 frontier ready, 10..12 after refinement rounds 0..2,
// 13 refinement done, 14 live entries entering refinement, 15 rounds run.
// The stamps go to LDS and are copied out when the workgroup exits, so that
// no global store of the instrumentation delays the loads being timed.
#ifdef TOPK_PHASE_TIMERS
__shared__ uint64_t g_tmarks[32];
#define PHASE_MARK(a, k)                                                                 \
    do {                                                                                 \
        if ((a).timers && threadIdx.x == 0) g_tmarks[k] = wall_clock64();                \
    } while (0)
#define PHASE_WORD(a, k, v)                                                              \
    do {                                                                                 \
        if ((a).timers && threadIdx.x == 0) g_tmarks[k] = (v);                           \
    } while (0)
struct TimerFlush {
    uint64_t *t;
    __device__ ~TimerFlush() {
        if (t && threadIdx.x == 0)
            for (int k = 0; k < 32; k++) t[(size_t)blockIdx.x * 32 + k] = g_tmarks[k];
    }
};
#else
#define PHASE_MARK(a, k) do {} while (0)
#define PHASE_WORD(a, k, v) do {} while (0)
#endif

// ------------------------------------------------------------- keys ----

// FP32 bit pattern of a value.  Takes the float by value: a bit cast applied
// directly to an element of an ext_vector_type lvalue does not read the
// subscripted element with this compiler.
__device__ __forceinline__ uint32_t fbits(float v) { return __builtin_bit_cast(uint32_t, v); }

__device__ __forceinline__ uint32_t asc_key(uint32_t b) {
    return b ^ ((uint32_t)((int32_t)b >> 31) | 0x80000000u);
}

__device__ __forceinline__ uint32_t bits_from_asc(uint32_t u) {
    return u ^ ((uint32_t)((int32_t)(~u) >> 31) | 0x80000000u);
}

// Coarse bin c(x) = floor(kappa16(fp16_rn(x)) / 32) (eq:method:coarse-map).
// For a negative FP16 pattern kappa16 = h, for a non-negative one 0x7FFF - h.
__device__ __forceinline__ uint32_t coarse_bin(float x) {
    const uint32_t h = __builtin_bit_cast(uint16_t, (_Float16)x);
    const uint32_t k16 = (h & 0x8000u) ? h : (0x7FFFu - h);
    return k16 >> 5;
}

__device__ __forceinline__ uint32_t f16_from_asc16(uint32_t a) {
    return (a & 0x8000u) ? (a & 0x7FFFu) : (~a & 0xFFFFu);
}

__device__ __forceinline__ uint32_t asc16_of(uint32_t h) {
    return (h & 0x8000u) ? (~h & 0xFFFFu) : (h | 0x8000u);
}

// Inclusive FP32 endpoint of coarse bin tau, as an ascending key: the
// smallest non-NaN value whose FP16 rounding lands in a bin <= tau.  The
// first admitted FP16 value v has ascending key hlo; every FP32 value above
// the midpoint between v and its FP16 predecessor rounds to >= v, and the
// midpoint itself goes wherever the hardware's round-to-nearest-even sends it.
__device__ __forceinline__ uint32_t bin_cutoff(uint32_t tau) {
    const int32_t hlo = 65504 - 32 * (int32_t)tau;   // 0xFFFF - (32 tau + 31)
    if (hlo <= 0x03FF) return 0x007FFFFFu;          // every value, -inf included
    if (hlo > 0xFC00) return 0xFFFFFFFFu;           // not even +inf qualifies
    const uint32_t v16 = f16_from_asc16((uint32_t)hlo);
    const uint32_t w16 = f16_from_asc16((uint32_t)hlo - 1u);
    float m;
    if (w16 == 0xFC00u) {
        m = -65520.0f;                              // lower overflow threshold
    } else if (v16 == 0x7C00u) {
        m = 65520.0f;                               // upper overflow threshold
    } else {
        const float w = (float)__builtin_bit_cast(_Float16, (uint16_t)w16);
        const float v = (float)__builtin_bit_cast(_Float16, (uint16_t)v16);
        m = (w + v) * 0.5f;                         // exact: adjacent FP16 values
    }
    uint32_t cut = asc_key(__builtin_bit_cast(uint32_t, m));
    const uint32_t hm = __builtin_bit_cast(uint16_t, (_Float16)m);
    if ((int32_t)asc16_of(hm) < hlo) cut += 1u;     // midpoint rounds down
    return cut;
}

// ------------------------------------------------------ wave helpers ----

__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & 63u); }

// Inclusive wave64 prefix sum with DPP row shifts and row broadcasts (no LDS
// round trips).
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v) {
    v += __builtin_amdgcn_update_dpp(0u, v, 0x111, 0xf, 0xf, false); // row_shr:1
    v += __builtin_amdgcn_update_dpp(0u, v, 0x112, 0xf, 0xf, false); // row_shr:2
    v += __builtin_amdgcn_update_dpp(0u, v, 0x114, 0xf, 0xf, false); // row_shr:4
    v += __builtin_amdgcn_update_dpp(0u, v, 0x118, 0xf, 0xf, false); // row_shr:8
    v += __builtin_amdgcn_update_dpp(0u, v, 0x142, 0xa, 0xf, false); // row_bcast:15
    v += __builtin_amdgcn_update_dpp(0u, v, 0x143, 0xc, 0xf, false); // row_bcast:31
    return v;
}

// Wave64 minimum / maximum; the result is valid in lane 63.
__device__ __forceinline__ uint32_t wave_min_to63(uint32_t v) {
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp(~0u, v, 0x111, 0xf, 0xf, false));
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp(~0u, v, 0x112, 0xf, 0xf, false));
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp(~0u, v, 0x114, 0xf, 0xf, false));
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp(~0u, v, 0x118, 0xf, 0xf, false));
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp(~0u, v, 0x142, 0xa, 0xf, false));
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp(~0u, v, 0x143, 0xc, 0xf, false));
    return v;
}

__device__ __forceinline__ uint32_t wave_max_to63(uint32_t v) {
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0u, v, 0x111, 0xf, 0xf, false));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0u, v, 0x112, 0xf, 0xf, false));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0u, v, 0x114, 0xf, 0xf, false));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0u, v, 0x118, 0xf, 0xf, false));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0u, v, 0x142, 0xa, 0xf, false));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0u, v, 0x143, 0xc, 0xf, false));
    return v;
}

struct Find {
    uint32_t bin;   // first bin whose inclusive prefix reaches the target
    uint32_t below; // prefix before that bin
    uint32_t eq;    // count in that bin
};

// Executed by one whole wave: locate min{b : H(b) >= k} over the 2048-bin
// histogram (eq:method:primary-threshold, eq:method:digit-boundary).  Level 1:
// lane l sums bins [32 l, 32 l + 32) and a wave scan finds the owning lane;
// level 2: 32 lanes scan the owner's bins.  Lane 0 writes *out.  A target of 0
// or above the total yields bin = 2048.
__device__ __forceinline__ void wave_find_level2(const uint32_t *hist, uint32_t incl, uint32_t tot,
                                                 uint32_t total, uint32_t k, Find *out) {
    const int lane = lane_id();
    if (k == 0 || k > total) {
        if (lane == 0) { out->bin = kBins; out->below = total; out->eq = 0; }
        return;
    }
    const int owner = __ffsll((unsigned long long)__ballot(incl >= k)) - 1;
    const uint32_t base = __builtin_amdgcn_readlane(incl - tot, owner);
    const uint32_t v = (lane < 32) ? hist[owner * 32 + lane] : 0u;
    const uint32_t incl2 = wave_incl_scan(v);
    const int l2 = __ffsll((unsigned long long)__ballot(lane < 32 && base + incl2 >= k)) - 1;
    const uint32_t below = base + __builtin_amdgcn_readlane(incl2 - v, l2);
    const uint32_t eq = __builtin_amdgcn_readlane(v, l2);
    if (lane == 0) { out->bin = (uint32_t)(owner * 32 + l2); out->below = below; out->eq = eq; }
}

// wave_find_level2 with the result returned (wave-uniform) instead of
// stored, so that every wave can locate the bin itself.
__device__ __forceinline__ Find wave_find_reg(const uint32_t *hist, uint32_t incl, uint32_t tot,
                                              uint32_t total, uint32_t k) {
    const int lane = lane_id();
    Find f;
    if (k == 0 || k > total) {
        f.bin = kBins; f.below = total; f.eq = 0;
        return f;
    }
    const int owner = __ffsll((unsigned long long)__ballot(incl >= k)) - 1;
    const uint32_t base = __builtin_amdgcn_readlane(incl - tot, owner);
    const uint32_t v = (lane < 32) ? hist[owner * 32 + lane] : 0u;
    const uint32_t incl2 = wave_incl_scan(v);
    const int l2 = __ffsll((unsigned long long)__ballot(lane < 32 && base + incl2 >= k)) - 1;
    f.bin = (uint32_t)(owner * 32 + l2);
    f.below = base + __builtin_amdgcn_readlane(incl2 - v, l2);
    f.eq = __builtin_amdgcn_readlane(v, l2);
    return f;
}

// wave_find_reg for two targets at once (bins only): both owner groups are
// read from LDS together, so the two searches share their latencies.
__device__ __forceinline__ void wave_find_bins2(const uint32_t *hist, uint32_t incl, uint32_t tot,
                                                uint32_t total, uint32_t k0, uint32_t k1,
                                                uint32_t &b0, uint32_t &b1) {
    const int lane = lane_id();
    const bool ok0 = k0 != 0 && k0 <= total, ok1 = k1 != 0 && k1 <= total;
    const int own0 = ok0 ? __ffsll((unsigned long long)__ballot(incl >= k0)) - 1 : 0;
    const int own1 = ok1 ? __ffsll((unsigned long long)__ballot(incl >= k1)) - 1 : 0;
    const uint32_t base0 = __builtin_amdgcn_readlane(incl - tot, own0);
    const uint32_t base1 = __builtin_amdgcn_readlane(incl - tot, own1);
    const uint32_t v0 = (lane < 32) ? hist[own0 * 32 + lane] : 0u;
    const uint32_t v1 = (lane < 32) ? hist[own1 * 32 + lane] : 0u;
    const uint32_t i0 = wave_incl_scan(v0), i1 = wave_incl_scan(v1);
    const int l0 = __ffsll((unsigned long long)__ballot(lane < 32 && base0 + i0 >= k0)) - 1;
    const int l1 = __ffsll((unsigned long long)__ballot(lane < 32 && base1 + i1 >= k1)) - 1;
    b0 = ok0 ? (uint32_t)(own0 * 32 + l0) : (uint32_t)kBins;
    b1 = ok1 ? (uint32_t)(own1 * 32 + l1) : (uint32_t)kBins;
}

__device__ __forceinline__ void wave_find(const uint32_t *hist, uint32_t k0, uint32_t k1, int nk, Find *out) {
    const int lane = lane_id();
    const uint4 *h4 = reinterpret_cast<const uint4 *>(hist + lane * 32);
    uint32_t tot = 0;
#pragma unroll
    for (int i = 0; i < 8; i++) {
        const uint4 t = h4[i];
        tot += t.x + t.y + t.z + t.w;
    }
    const uint32_t incl = wave_incl_scan(tot);
    const uint32_t total = __builtin_amdgcn_readlane(incl, 63);
    wave_find_level2(hist, incl, tot, total, k0, &out[0]);
    if (nk > 1) wave_find_level2(hist, incl, tot, total, k1, &out[1]);
}

// Sums of the 64 groups of 32 bins of a 2048-bin histogram into out[64], by
// the whole block: thread t adds bins [4 t, 4 t + 4), then each group of 8
// lanes is summed with DPP row shifts (lane 8 g + 7 holds group g's sum).
// Needs the histogram complete (caller's barrier); out is complete after the
// next barrier.
static_assert(kBlock * 4 == kBins, "group_sums: one uint4 of bins per thread");
__device__ __forceinline__ void group_sums(const uint32_t *hist, uint32_t *out) {
    const uint4 h = reinterpret_cast<const uint4 *>(hist)[threadIdx.x];
    uint32_t v = h.x + h.y + h.z + h.w;
    v += __builtin_amdgcn_update_dpp(0u, v, 0x111, 0xf, 0xf, false); // row_shr:1
    v += __builtin_amdgcn_update_dpp(0u, v, 0x112, 0xf, 0xf, false); // row_shr:2
    v += __builtin_amdgcn_update_dpp(0u, v, 0x114, 0xf, 0xf, false); // row_shr:4
    if ((threadIdx.x & 7u) == 7u) out[threadIdx.x >> 3] = v;
}

// ------------------------------------------------- shared state ----

struct alignas(16) Smem {
    uint32_t hist[kBins];
    uint32_t hist2[kBins]; // refinement alternates between hist and hist2
    uint32_t ci[kFront]; // frontier indices (row-relative)
    uint32_t ck[kFront]; // frontier keys: FP32 bits after Phase 2, kappa32 after compaction
    uint32_t wcnt[kWaves]; // Phase 2 hits per wave (exact, may exceed kWaveCap)
    uint32_t red[4];       // refinement: min/max kappa32, min/max index of the live keys
    uint32_t coarse[2][64]; // refinement: 32-bin group sums of hist / hist2
    Find find[2];
    uint32_t cnt;       // C(tau1), or the append counter of the current pass
    uint32_t cnt0;      // C(tau0)
    uint32_t incomplete;
    uint32_t opos;      // outputs written for the current row
    uint32_t knext;       // refinement: rank-table entries appended
    uint32_t wc[kWaves];  // refinement: entries committed by each wave in a pass
    uint32_t wk[kWaves];  // refinement: entries kept by each wave in a pass
    uint32_t cut0, cut1, tau0, tau1;
    uint32_t flag;
    uint32_t base;
    int64_t lsum[kWaves]; // per-wave partial sums of the row lengths
    uint32_t amax;        // largest ascending key among the stored entries
    uint64_t xword;       // split exact route: a route word
};

__device__ __forceinline__ void clear_hist(Smem &sm) {
    uint4 *h4 = reinterpret_cast<uint4 *>(sm.hist);
    for (int i = threadIdx.x; i < kBins / 4; i += kBlock) h4[i] = make_uint4(0, 0, 0, 0);
    if (threadIdx.x < 64) sm.coarse[0][threadIdx.x] = 0u;
}

// ---------------------------------------------------- row streaming ----
//
// Streams row elements [beg, end) (row-relative) of the row at element offset
// `off` with 16-byte loads.  The loads are aligned to the 16-byte grid of the
// allocation; the up to three elements on either side of the range that share
// a vector with valid ones are loaded and masked out (a 16-byte aligned block
// never straddles a page, so the access is always mapped).  Each chunk gives
// every thread kVec vectors; fn(x[16], i0[kVec], lo, hi) is called with the
// 16 values, the row index of each vector's first element, and the valid
// row-index window [lo, hi).  Two chunks are in flight (ping-pong registers).

typedef __attribute__((address_space(1))) const f4 gf4; // global, not flat

template <bool kNonTemporal>
__device__ __forceinline__ f4 load4(const f4 *p) {
    const gf4 *g = (const gf4 *)p;
    if constexpr (kNonTemporal) return __builtin_nontemporal_load(g);
    else return *g;
}

struct NoPrologue {
    __device__ void operator()() const {}
};

struct NeverStop {
    __device__ constexpr bool operator()() const { return false; }
};

// A row range as 16-byte vectors: [beg, end) of the row at element offset
// off, covered by nvec vectors from vbase (the start of the 128-byte line
// holding element beg; ibase is the row index of vbase's first element), in
// nch chunks of kChunkVecs.
struct RowVecs {
    const char *vbase;
    int32_t ibase, nvec, nch;
};

__device__ __forceinline__ RowVecs row_vecs(const float *scores, int64_t off, int32_t beg,
                                            int32_t end) {
    const uintptr_t sp = reinterpret_cast<uintptr_t>(scores);
    const int64_t sh = (int64_t)((sp & 15) >> 2);
    // The first vector is that of the 128-byte line holding element beg, so
    // each wave's 64 vectors of a chunk cover eight whole lines, not parts
    // of nine (the elements before beg are masked by the window test; the
    // line holds a valid element, so it lies in mapped memory).
    const int64_t v0 = ((off + beg + sh) >> 2) & ~(int64_t)7;
    RowVecs g;
    g.nvec = (int32_t)(((off + end + sh + 3) >> 2) - v0);
    g.vbase = reinterpret_cast<const char *>(sp & ~(uintptr_t)15) + v0 * 16;
    g.ibase = (int32_t)(v0 * 4 - sh - off);
    g.nch = (g.nvec + kChunkVecs - 1) / kChunkVecs;
    return g;
}

// Loads of chunk c are unconditional: lanes and chunks past the end re-read
// the last vector of the range (one cache line per wave), masked later by
// the window test, so that the in-order load counter lets each consume wait
// for its own chunk only.
template <bool kNT>
__device__ __forceinline__ void issue_chunk(const RowVecs &g, f4 *dst, int32_t c) {
    const int32_t cb = c * kChunkVecs;
#pragma unroll
    for (int m = 0; m < kVec; m++) {
        const int32_t vi = min(cb + m * kBlock + (int32_t)threadIdx.x, g.nvec - 1);
        dst[m] = load4<kNT>(reinterpret_cast<const f4 *>(g.vbase + (uint32_t)vi * 16u));
    }
}

template <class F>
__device__ __forceinline__ void consume_chunk(const RowVecs &g, const f4 *src, int32_t c,
                                              int32_t beg, int32_t end, F &fn) {
    if (c >= g.nch) return;
    const int32_t cb = c * kChunkVecs;
    // vectors of this chunk per thread (block-uniform)
    const int32_t mv = min(kVec, (g.nvec - cb + kBlock - 1) / kBlock);
    int32_t i0[kVec];
#pragma unroll
    for (int m = 0; m < kVec; m++) i0[m] = g.ibase + (cb + m * kBlock + (int32_t)threadIdx.x) * 4;
    // interior chunks need no per-element window test
    const bool edge = g.ibase + cb * 4 < beg || g.ibase + (cb + mv * kBlock) * 4 > end;
    fn(src, i0, beg, end, edge, mv);
}

// Double-buffered chunks: while one chunk (kVec 16-byte loads per thread) is
// consumed, the next one is in flight.  prologue() runs once, by every
// thread, with the first chunk in flight (loads it waits for must have been
// issued before the call, or they would queue behind the chunk).  A wave
// leaves the loop after any chunk for which stop() (wave-uniform) holds.
template <bool kNT, class F, class Pro = NoPrologue, class Stop = NeverStop>
__device__ __forceinline__ void stream_row(const float *scores, int64_t off, int32_t beg,
                                           int32_t end, F &&fn, Pro &&prologue = Pro(),
                                           Stop &&stop = Stop()) {
    if (beg >= end) {
        prologue();
        return;
    }
    const RowVecs g = row_vecs(scores, off, beg, end);
    f4 xa[kVec], xb[kVec];
    issue_chunk<kNT>(g, xa, 0);
    prologue();
    for (int32_t c = 0; c < g.nch; c += 2) {
        issue_chunk<kNT>(g, xb, c + 1);
        consume_chunk(g, xa, c, beg, end, fn);
        if (stop()) break;
        issue_chunk<kNT>(g, xa, c + 2);
        consume_chunk(g, xb, c + 1, beg, end, fn);
        if (stop()) break;
    }
}

// Largest range resident_row takes, in chunks.
constexpr int kResidentChunks = 2;

// A range of at most kResidentChunks chunks held in registers: both chunks
// are loaded once and passed to fn1, then mid() runs (every thread, may
// synchronise), then the same registers are passed to fn2 -- a two-pass
// computation that reads the range from memory once.
template <class F1, class M, class F2>
__device__ __forceinline__ void resident_row(const RowVecs &g, int32_t beg, int32_t end, F1 &&fn1,
                                             M &&mid, F2 &&fn2) {
    static_assert(kResidentChunks == 2, "two register chunks");
    f4 xa[kVec], xb[kVec];
    issue_chunk<false>(g, xa, 0);
    issue_chunk<false>(g, xb, 1);
    consume_chunk(g, xa, 0, beg, end, fn1);
    consume_chunk(g, xb, 1, beg, end, fn1);
    mid();
    consume_chunk(g, xa, 0, beg, end, fn2);
    consume_chunk(g, xb, 1, beg, end, fn2);
}

__device__ __forceinline__ bool in_window(int32_t i, int32_t lo, int32_t hi) {
    return i >= lo && i < hi;
}

// Appends every element of the range whose ascending key u satisfies
// lo_key <= u < hi_key to the LDS frontier (index, kappa32); sm.cnt counts all
// of them even past the capacity.  Phase 2 of Section 4.3 with hi_key = ~0
// (plus the top key itself, see below); the band of eq:method:rescue-band
// with [cut1, cut0).
template <bool kNT>
__device__ __forceinline__ void collect_range(Smem &sm, const float *scores, int64_t off, int32_t beg,
                              int32_t end, uint32_t lo_key, uint32_t hi_key, bool hi_inclusive,
                              uint32_t cap) {
    stream_row<kNT>(scores, off, beg, end, [&](const f4 *x, const int32_t *i0, int32_t lo,
                                               int32_t hi, bool, int32_t mv) {
        uint64_t mask = 0; // one bit per element of the chunk (kVec * 4 <= 64)
#pragma unroll
        for (int m = 0; m < kVec; m++) if (m < mv) {
#pragma unroll
            for (int c = 0; c < 4; c++) {
                const uint32_t u = asc_key(fbits(x[m][c]));
                const bool ok = u >= lo_key && (hi_inclusive ? u <= hi_key : u < hi_key) &&
                                in_window(i0[m] + c, lo, hi);
                mask |= (ok ? 1ull : 0ull) << (m * 4 + c);
            }
        }
        if (mask) {
            uint32_t pos = atomicAdd(&sm.cnt, (uint32_t)__popcll(mask));
#pragma unroll
            for (int m = 0; m < kVec; m++) if (m < mv) {
#pragma unroll
                for (int c = 0; c < 4; c++) {
                    if (mask & (1ull << (m * 4 + c))) {
                        if (pos < cap) {
                            sm.ci[pos] = (uint32_t)(i0[m] + c);
                            sm.ck[pos] = ~asc_key(fbits(x[m][c]));
                        }
                        pos++;
                    }
                }
            }
        }
    });
}

// Phase 2 over [beg, end) (Section 4.3): certify against cut0 and keep the
// admitted tail.  Every value with ascending key u >= cut1 (the nested
// boundary, so a C(tau0) < K proposal can take the band of
// eq:method:rescue-band without a second traversal) is stored as (index, FP32
// bits) in the private region of its wave: sm.ci/ck[w * kWaveStride ..).
// Each element costs one compare; a wave-wide ballot places the hits with no
// atomics, and sm.cnt gets C(tau1).  A wave whose region overflows sets
// sm.incomplete and stops (sm.cnt is then partial; the caller re-counts by
// re-reading) -- or, with kHistOver, goes on to the end of the range adding
// each hit its region cannot keep into the coarse histogram sm.hist2 (clear
// before a barrier that precedes the first chunk's consumption): the stored
// entries and sm.hist2 then count every hit, so sm.cnt is exact and the
// coarse histogram of the range is exact in bins 0..tau1 without a re-read.
// The endpoints are read from sm after prologue() has run.
template <bool kHistOver, class Pro>
__device__ __forceinline__ void phase2_collect(Smem &sm, const float *scores, int64_t off,
                                               int32_t beg, int32_t end, Pro &&prologue) {
    const int w = threadIdx.x >> 6;
    uint32_t cur = 0; // wave-uniform: hits so far
    stream_row<true>(
        scores, off, beg, end,
        [&](const f4 *x, const int32_t *i0, int32_t lo, int32_t hi, bool edge, int32_t mv) {
            const uint32_t cut1 = sm.cut1;
            uint32_t *wi = sm.ci + w * kWaveStride;
            uint32_t *wk = sm.ck + w * kWaveStride;
            auto run = [&](auto positive, auto edge_chunk) {
                constexpr bool kPos = decltype(positive)::value;
                constexpr bool kEdge = decltype(edge_chunk)::value;
                // A positive endpoint v: x >= v iff the raw FP32 bits, read as
                // signed integers, compare >= (one integer compare).
                const int32_t t1 = (int32_t)bits_from_asc(cut1);
                // Branch-free append: every lane writes every element, a hit
                // to its slot (running count + rank among the vector
                // element's hits), any other to its own dummy slot.
                const uint32_t dummy = (uint32_t)kWaveCap + 1u + (uint32_t)lane_id();
#pragma unroll
                for (int m = 0; m < kVec; m++) if (m < mv) {
                    bool hit[4];
                    uint64_t mk[4];
#pragma unroll
                    for (int c = 0; c < 4; c++) {
                        const uint32_t b = fbits(x[m][c]);
                        const bool h1 = kPos ? (int32_t)b >= t1 : asc_key(b) >= cut1;
                        hit[c] = h1;
                        if constexpr (kEdge) hit[c] = h1 && in_window(i0[m] + c, lo, hi);
                        mk[c] = __ballot(hit[c]);
                    }
                    if constexpr (kHistOver) {
                        if (cur >= (uint32_t)kWaveCap) { // (wave-uniform)
                            // region full: the hits are only counted
#pragma unroll
                            for (int c = 0; c < 4; c++) {
                                if (hit[c]) atomicAdd(&sm.hist2[coarse_bin(x[m][c])], 1u);
                                cur += (uint32_t)__popcll(mk[c]);
                            }
                            continue;
                        }
                    }
                    const uint32_t cur0 = cur;
#pragma unroll
                    for (int c = 0; c < 4; c++) {
                        // slot kWaveCap of the region absorbs hits past its
                        // capacity (the count stays exact)
                        const uint32_t q = min(__builtin_amdgcn_mbcnt_hi((uint32_t)(mk[c] >> 32),
                                                   __builtin_amdgcn_mbcnt_lo((uint32_t)mk[c], cur)),
                                               (uint32_t)kWaveCap);
                        const uint32_t d = hit[c] ? q : dummy;
                        wi[d] = (uint32_t)(i0[m] + c);
                        wk[d] = fbits(x[m][c]);
                        cur += (uint32_t)__popcll(mk[c]);
                    }
                    if constexpr (kHistOver) {
                        if (cur > (uint32_t)kWaveCap) { // (wave-uniform, once per wave)
                            // the hits of this vector past the capacity
                            uint32_t run_c = cur0;
#pragma unroll
                            for (int c = 0; c < 4; c++) {
                                const uint32_t rk = __builtin_amdgcn_mbcnt_hi(
                                    (uint32_t)(mk[c] >> 32),
                                    __builtin_amdgcn_mbcnt_lo((uint32_t)mk[c], run_c));
                                if (hit[c] && rk >= (uint32_t)kWaveCap)
                                    atomicAdd(&sm.hist2[coarse_bin(x[m][c])], 1u);
                                run_c += (uint32_t)__popcll(mk[c]);
                            }
                        }
                    }
                }
            };
            // four specialisations, chosen once per chunk
            if (cut1 > 0x80000000u) {
                if (edge) run(std::true_type{}, std::true_type{});
                else run(std::true_type{}, std::false_type{});
            } else {
                if (edge) run(std::false_type{}, std::true_type{});
                else run(std::false_type{}, std::false_type{});
            }
        },
        prologue,
        // a wave whose region has overflowed stops: the segment's entries
        // will not be used, and both counts are then taken by a re-read
        // (with kHistOver no wave stops)
        [&]() { return !kHistOver && cur > (uint32_t)kWaveCap; });
    if ((threadIdx.x & 63) == 0) {
        sm.wcnt[w] = cur;
        atomicAdd(&sm.cnt, cur);
        if (cur > (uint32_t)kWaveCap) sm.incomplete = 1u;
    }
}

// C(tau0) from the stored entries of Phase 2 (all of A(tau1) when complete,
// in the per-wave regions), and into sm.amax the largest ascending key
// stored.  sm.cnt0 and sm.amax must be zero on entry.  Ends with a barrier.
__device__ __forceinline__ uint32_t count_tail(Smem &sm, uint32_t kmin) {
    const uint32_t w = threadIdx.x >> 6;
    const uint32_t beg = w * kWaveStride, end = beg + min(sm.wcnt[w], (uint32_t)kWaveCap);
    uint32_t c = 0, mx = 0;
    for (uint32_t e = beg + (uint32_t)lane_id(); e < end; e += 64) {
        const uint32_t u = asc_key(sm.ck[e]);
        c += u >= kmin ? 1u : 0u;
        mx = max(mx, u);
    }
    c = wave_incl_scan(c);
    mx = wave_max_to63(mx);
    if ((threadIdx.x & 63) == 63) {
        if (c) atomicAdd(&sm.cnt0, c);
        atomicMax(&sm.amax, mx);
    }
    __syncthreads();
    return sm.cnt0;
}

// C(tau0) and C(tau1) (.x, .y, wave-uniform) of the row elements [beg, end)
// that this wave's lanes stream (stream_row's positions of these threads).
__device__ __forceinline__ uint2 count_range_wave(const float *scores, int64_t off, int32_t beg,
                                                  int32_t end, uint32_t cut0, uint32_t cut1) {
    uint32_t c0 = 0, c1 = 0;
    stream_row<false>(scores, off, beg, end, [&](const f4 *x, const int32_t *i0, int32_t lo,
                                                 int32_t hi, bool, int32_t mv) {
#pragma unroll
        for (int m = 0; m < kVec; m++) if (m < mv) {
#pragma unroll
            for (int cc = 0; cc < 4; cc++) {
                const uint32_t u = asc_key(fbits(x[m][cc]));
                const bool in = in_window(i0[m] + cc, lo, hi);
                c0 += (in && u >= cut0) ? 1u : 0u;
                c1 += (in && u >= cut1) ? 1u : 0u;
            }
        }
    });
    return make_uint2(__builtin_amdgcn_readlane(wave_incl_scan(c0), 63),
                      __builtin_amdgcn_readlane(wave_incl_scan(c1), 63));
}

// C(tau0) and C(tau1) of row elements [beg, end) by re-reading them (after a
// wave region overflowed), into sm.cnt0 and sm.cnt (zero on entry).  Ends
// with a barrier.
__device__ __forceinline__ void count_range(Smem &sm, const float *scores, int64_t off,
                                            int32_t beg, int32_t end, uint32_t cut0,
                                            uint32_t cut1) {
    const uint2 c = count_range_wave(scores, off, beg, end, cut0, cut1);
    if ((threadIdx.x & 63) == 0) {
        if (c.x) atomicAdd(&sm.cnt0, c.x);
        if (c.y) atomicAdd(&sm.cnt, c.y);
    }
    __syncthreads();
}

// ----------------------------------------------------------- outputs ----

__device__ __forceinline__ void emit(const KArgs a, int r, uint32_t pos, uint32_t idx,
                                     uint32_t kappa) {
    if (pos >= (uint32_t)a.K) return; // never taken for a consistent selection
    const int64_t o = (int64_t)r * a.K + pos;
    a.out_idx[o] = (int32_t)idx;
    a.out_val[o] = __builtin_bit_cast(float, bits_from_asc(~kappa));
}

__device__ __forceinline__ void write_direct(const KArgs a, int r, const float *row, int64_t L) {
    for (int j = threadIdx.x; j < a.K; j += kBlock) {
        const int64_t o = (int64_t)r * a.K + j;
        if (j < L) {
            a.out_idx[o] = j;
            a.out_val[o] = row[j];
        } else {
            a.out_idx[o] = -1;
            a.out_val[o] = -__builtin_huge_valf();
        }
    }
}

__device__ __forceinline__ void write_error_row(const KArgs a, int r) {
    for (int j = threadIdx.x; j < a.K; j += kBlock) {
        const int64_t o = (int64_t)r * a.K + j;
        a.out_idx[o] = -1;
        a.out_val[o] = -__builtin_huge_valf();
    }
}

// ------------------------------------------------------- refinement ----

// Phase 3 (Section 4.4).  The frontier Q0 (quota k; sm.opos outputs already
// written) stays in sm.ci/ck, as FP32 bits filtered by ascending key >= kmin
// (`raw`) or as kappa32 keys, in per-wave ranges: the wave regions of Phase
// 2 (`segmented`) or eighths of [0, n).  Entries are ordered by the composite
// key z = (kappa32 << 32) | index (ties broken toward the lowest index).
// Each round histograms an 11-bit digit of z over the live entries, finds
// b = min{b : H(b) >= k} (eq:method:digit-boundary), commits the groups
// before b (eq:method:committed-group), keeps group b
// (eq:method:refine-recurrence) and stops once the kept group exactly fills
// the quota.  The paper's digits are fixed 11/11/10-bit fields of kappa32.
// Here the first digit is taken from the live keys' range instead:
// d(z) = (z - lo) >> w, with lo the smallest live key and w the smallest
// shift that maps the range into 2048 bins; every later round takes the next
// 11 bits of the same offset key inside the kept bin.  Bins are contiguous
// key ranges in key order, as radix digits are, so the selected set is the
// same, in fewer rounds: a frontier between 1.9 and 5.0 spans four exponent
// values, which fixed digits would split into a handful of bins.  The live
// entries of a round are exactly those whose key lies in the kept key range
// [lo, hi], so no per-entry state is kept.  Once at most kSmall entries are
// live, the rest is settled by ranking them against each other.  Every pass
// is a loop of each wave over its own range.
__device__ __forceinline__ uint64_t zkey(uint32_t kappa, uint32_t idx) {
    return ((uint64_t)kappa << 32) | idx;
}

__device__ __forceinline__ void reset_range(Smem &sm) {
    if (threadIdx.x < 4) sm.red[threadIdx.x] = (threadIdx.x & 1) ? 0u : ~0u;
}

// Ranking costs each of the ceil(n / 64) working waves n lane reads, so it
// settles only small sets; a digit round is cheaper beyond about 64.
constexpr uint32_t kSmall = 64;

// The live key range of a round, [lo, hi] over composite keys, digit
// d(z) = (z - lo) >> w.  When the range covers whole kappa32 values and the
// digit lies above the index bits (w >= 32), keys and digits are taken from
// kappa32 alone (klo, khi, wf = w - 32): the common case, with half the work.
struct Window {
    uint64_t lo, hi;
    uint32_t w;
    bool fast;
    uint32_t klo, kspan, wf;
    uint32_t imin, imax; // bounds of the live entries' indices
};

// A window of keys [lo >> 32, hi >> 32] with digit shift w (the register
// finish's single round).
__device__ __forceinline__ Window key_window(uint64_t lo, uint64_t hi, uint32_t w) {
    Window v;
    v.lo = lo; v.hi = hi; v.w = w;
    v.fast = w >= 32 && (uint32_t)lo == 0u && (uint32_t)hi == 0xFFFFFFFFu;
    v.klo = (uint32_t)(lo >> 32);
    v.kspan = (uint32_t)(hi >> 32) - v.klo;
    v.wf = v.fast ? w - 32 : 0u;
    v.imin = 0u; v.imax = 0xFFFFFFFFu;
    return v;
}

// The window [lo, hi] of composite keys (kappa32 << 32 | index) with the
// smallest shift w that fits 2048 bins.  A window inside one key is first
// narrowed to the live indices [imin, imax], so that ties (equal keys,
// settled by index) take as few digit rounds as the indices need.
__device__ __forceinline__ Window make_window(uint64_t lo, uint64_t hi, uint32_t imin,
                                              uint32_t imax) {
    if ((lo >> 32) == (hi >> 32)) {
        const uint64_t key = lo & 0xFFFFFFFF00000000ull;
        lo = max(lo, key | imin);
        hi = min(hi, key | imax);
    }
    const uint64_t span = hi - lo;
    const int bits = span ? 64 - __clzll((long long)span) : 0;
    Window v;
    v.lo = lo; v.hi = hi;
    v.w = bits > 11 ? (uint32_t)(bits - 11) : 0u;
    v.fast = v.w >= 32 && (uint32_t)lo == 0u && (uint32_t)hi == 0xFFFFFFFFu;
    v.klo = (uint32_t)(lo >> 32);
    v.kspan = (uint32_t)(hi >> 32) - v.klo;
    v.wf = v.fast ? v.w - 32 : 0u;
    v.imin = imin; v.imax = imax;
    return v;
}

// Frontier entry e of the refinement: its kappa32 and FP32 bits.
struct Ent {
    uint32_t kk, bits;
};

__device__ __forceinline__ Ent read_ent(const Smem &sm, uint32_t e, bool raw) {
    const uint32_t word = sm.ck[e];
    Ent x;
    x.kk = raw ? ~asc_key(word) : word;
    x.bits = raw ? word : bits_from_asc(~word);
    return x;
}

// Per-entry classes against the window and boundary bin b: live, below b,
// in b.  kFast: 32-bit keys (index bits not part of the digit).
template <bool kFast>
struct Classifier {
    Window v;
    uint32_t cb, ce; // fast: below iff t < cb, in b iff cb <= t <= ce (t = kk - klo)
    uint32_t b;
    __device__ __forceinline__ Classifier(const Window &win, uint32_t bin) : v(win), b(bin) {
        cb = bin << win.wf;
        const uint32_t top = cb + (((uint32_t)1 << win.wf) - 1u);
        ce = min(top, win.kspan);
    }
    __device__ __forceinline__ bool live(const Smem &sm, uint32_t e, const Ent &x) const {
        if constexpr (kFast) return x.kk - v.klo <= v.kspan;
        const uint64_t z = zkey(x.kk, sm.ci[e]);
        return z >= v.lo && z <= v.hi;
    }
    __device__ __forceinline__ uint32_t digit(const Smem &sm, uint32_t e, const Ent &x) const {
        if constexpr (kFast) return (x.kk - v.klo) >> v.wf;
        return (uint32_t)((zkey(x.kk, sm.ci[e]) - v.lo) >> v.w);
    }
    // below b / in b, both implying live
    __device__ __forceinline__ void cls(const Smem &sm, uint32_t e, const Ent &x, bool &below,
                                        bool &inb) const {
        if constexpr (kFast) {
            const uint32_t t = x.kk - v.klo;
            below = t < cb && t <= v.kspan;
            inb = t >= cb && t <= ce;
        } else {
            const uint64_t z = zkey(x.kk, sm.ci[e]);
            const bool lv = z >= v.lo && z <= v.hi;
            const uint32_t d = lv ? (uint32_t)((z - v.lo) >> v.w) : 0u;
            below = lv && d < b;
            inb = lv && d == b;
        }
    }
};

// Writes output slot pos of this refinement (entry e, class known).
__device__ __forceinline__ void put_out(const KArgs a, int64_t out0, uint32_t pos, uint32_t idx,
                                        uint32_t bits) {
    // pos < K <= 16384: a 32-bit byte offset from the row's (uniform) base
    const uint32_t boff = pos << 2;
    *reinterpret_cast<int32_t *>(reinterpret_cast<char *>(a.out_idx + out0) + boff) = (int32_t)idx;
    *reinterpret_cast<float *>(reinterpret_cast<char *>(a.out_val + out0) + boff) =
        __builtin_bit_cast(float, bits);
}

// Ranks the nk keys of the LDS table zs against each other and writes the k
// lowest to output slots placed + rank.  Wave v ranks table entries
// [64 v, 64 v + 64) against the whole table, 64 keys at a time read across
// lanes.  Needs the table complete (caller's barrier).
template <class Sink>
__device__ __forceinline__ void rank_small_to(const uint64_t *zs, uint32_t nk, uint32_t k,
                                              uint32_t placed, Sink &&sink) {
    const uint32_t w8 = threadIdx.x >> 6, lane = (uint32_t)lane_id();
    if (64 * w8 >= nk) return;
    const uint32_t i = 64 * w8 + lane;
    // keys are below 2^64 - 1 (indices are below 2^31): ~0 pads never count
    const uint64_t z = i < nk ? zs[i] : ~0ull;
    uint32_t rank = 0;
    for (uint32_t c = 0; c < nk; c += 64) {
        const uint64_t y = (c + lane < nk) ? zs[c + lane] : ~0ull;
        const uint32_t ylo = (uint32_t)y, yhi = (uint32_t)(y >> 32);
        const uint32_t m = min(64u, nk - c);
        for (uint32_t l = 0; l < m; l++) {
            const uint64_t v = ((uint64_t)(uint32_t)__builtin_amdgcn_readlane(yhi, l) << 32) |
                               (uint32_t)__builtin_amdgcn_readlane(ylo, l);
            rank += (v < z) ? 1u : 0u;
        }
    }
    if (i < nk && rank < k) sink(placed + rank, (uint32_t)z, bits_from_asc(~(uint32_t)(z >> 32)));
}

__device__ __forceinline__ void rank_small(const KArgs a, int64_t out0, const uint64_t *zs,
                                           uint32_t nk, uint32_t k, uint32_t placed) {
    rank_small_to(zs, nk, k, placed, [&](uint32_t pos, uint32_t idx, uint32_t bits) {
        put_out(a, out0, pos, idx, bits);
    });
}

// Per-wave exclusive prefix and total of sm.wc / sm.wk (after a barrier).
__device__ __forceinline__ void wave_bases(const Smem &sm, uint32_t &cbase, uint32_t &kbase,
                                           uint32_t &ctotal) {
    const uint32_t w8 = threadIdx.x >> 6;
    cbase = 0; kbase = 0; ctotal = 0;
#pragma unroll
    for (uint32_t v = 0; v < (uint32_t)kWaves; v++) {
        const uint32_t c = sm.wc[v], q = sm.wk[v];
        if (v < w8) { cbase += c; kbase += q; }
        ctotal += c;
    }
}

// One refinement round over the live entries of window win (quota k):
// histogram, boundary bin, count and place.  Returns true when the row is
// complete; otherwise win, n_live and k describe the next round.
template <bool kFast>
__device__ __forceinline__ bool refine_round(const KArgs a, Smem &sm, uint32_t beg, uint32_t end,
                                             bool raw, int64_t out0, uint32_t &placed,
                                             Window &win, uint32_t &n_live, uint32_t &k,
                                             int par) {
    const int tid = threadIdx.x;
    const uint32_t lane = (uint32_t)lane_id(), w8 = (uint32_t)tid >> 6;
    uint32_t *H = par ? sm.hist2 : sm.hist;
    uint32_t *C = sm.coarse[par];
    {
        uint4 *h4 = reinterpret_cast<uint4 *>(par ? sm.hist : sm.hist2);
        for (int i = tid; i < kBins / 4; i += kBlock) h4[i] = make_uint4(0, 0, 0, 0);
        if (tid < 64) sm.coarse[par ^ 1][tid] = 0u;
        if (tid == 0) sm.knext = 0u;
    }
    {
        const Classifier<kFast> q(win, 0u);
        for (uint32_t e = beg + lane; e < end; e += 64) {
            const Ent x = read_ent(sm, e, raw);
            if (q.live(sm, e, x)) {
                const uint32_t d = q.digit(sm, e, x);
                atomicAdd(&H[d], 1u);
                atomicAdd(&C[d >> 5], 1u);
            }
        }
    }
    __syncthreads();
    if (tid < 64) {
        // two levels: 64 coarse groups of 32 bins, then the owner's bins
        const uint32_t c = C[tid];
        const uint32_t incl = wave_incl_scan(c);
        const uint32_t total = __builtin_amdgcn_readlane(incl, 63);
        wave_find_level2(H, incl, c, total, k, &sm.find[par]);
    }
    __syncthreads();
    const Find f = sm.find[par];
    const uint32_t need = k - f.below; // > 0 and <= f.eq
    const bool take_all = f.eq == need;
    const bool rank_next = !take_all && f.eq <= kSmall;
    const Classifier<kFast> q(win, f.bin);
    uint64_t *zs = reinterpret_cast<uint64_t *>(par ? sm.hist : sm.hist2);
    if (take_all || rank_next) {
        // Last round: each wave moves its committed entries (below b, or up
        // to b with take_all) to the front of its own range, in place (an
        // entry is only written over after it has been read), and appends
        // the kept ones (bin b) to the rank table; then the committed
        // entries go out in consecutive slots.
        uint32_t cw = 0;
        for (uint32_t e = beg + lane; e < end; e += 64) {
            const Ent x = read_ent(sm, e, raw);
            bool below, inb;
            q.cls(sm, e, x, below, inb);
            const bool commit = below || (take_all && inb);
            const bool keep = rank_next && inb;
            const uint64_t mc = __ballot(commit);
            const uint64_t mk = __ballot(keep);
            uint32_t kb = 0;
            if (mk) {
                const uint32_t first = (uint32_t)__ffsll((unsigned long long)mk) - 1u;
                if (lane == first) kb = atomicAdd(&sm.knext, (uint32_t)__popcll(mk));
                kb = __builtin_amdgcn_readlane(kb, first);
            }
            if (commit || keep) {
                const uint32_t idx = sm.ci[e];
                if (commit) {
                    const uint32_t d = beg + cw + __builtin_amdgcn_mbcnt_hi((uint32_t)(mc >> 32),
                                              __builtin_amdgcn_mbcnt_lo((uint32_t)mc, 0u));
                    sm.ci[d] = idx;
                    sm.ck[d] = x.bits;
                } else {
                    zs[kb + __builtin_amdgcn_mbcnt_hi((uint32_t)(mk >> 32),
                                __builtin_amdgcn_mbcnt_lo((uint32_t)mk, 0u))] = zkey(x.kk, idx);
                }
            }
            cw += (uint32_t)__popcll(mc);
        }
        if (lane == 0) sm.wc[w8] = cw;
        __syncthreads();
        // (lanes that left the loop early hold a partial cw: use the wave's)
        uint32_t cbase = placed, committed = 0;
#pragma unroll
        for (uint32_t v = 0; v < (uint32_t)kWaves; v++) {
            const uint32_t c = sm.wc[v];
            cbase += v < w8 ? c : 0u;
            committed += c;
        }
        const uint32_t ncw = sm.wc[w8];
        for (uint32_t e = lane; e < ncw; e += 64)
            put_out(a, out0, cbase + e, sm.ci[beg + e], sm.ck[beg + e]);
        placed += committed;
        if (take_all) return true;
        k -= committed;
        rank_small(a, out0, zs, f.eq, k, placed);
        return true;
    }
    // Another round follows: count pass (entries below b per wave), then the
    // place pass; the entries stay where they are.
    uint32_t cw = 0;
    for (uint32_t e = beg + lane; e < end; e += 64) {
        const Ent x = read_ent(sm, e, raw);
        bool below, inb;
        q.cls(sm, e, x, below, inb);
        cw += (uint32_t)__popcll(__ballot(below));
    }
    if (lane == 0) { sm.wc[w8] = cw; sm.wk[w8] = 0u; }
    __syncthreads();
    uint32_t cbase, kbase, committed;
    wave_bases(sm, cbase, kbase, committed);
    cbase += placed;
    // place pass: committed entries to consecutive output slots of each wave
    for (uint32_t e = beg + lane; e < end; e += 64) {
        const Ent x = read_ent(sm, e, raw);
        bool below, inb;
        q.cls(sm, e, x, below, inb);
        const uint64_t mc = __ballot(below);
        if (below)
            put_out(a, out0, cbase + __builtin_amdgcn_mbcnt_hi((uint32_t)(mc >> 32),
                                     __builtin_amdgcn_mbcnt_lo((uint32_t)mc, 0u)),
                    sm.ci[e], x.bits);
        cbase += (uint32_t)__popcll(mc);
    }
    placed += committed;
    k -= committed;
    // next round inside the kept bin: the 11 bits below w
    n_live = f.eq;
    const uint64_t blo = win.lo + ((uint64_t)f.bin << win.w);
    win = make_window(blo, min(blo + (((uint64_t)1 << win.w) - 1), win.hi), win.imin, win.imax);
    __syncthreads(); // sm.wc is rewritten by the next count pass
    return false;
}

// imax: the largest index an entry can have (the row length less one).
__device__ __forceinline__ void refine(const KArgs a, Smem &sm, int r, bool segmented, uint32_t n,
                                       bool raw, uint32_t amin, uint32_t amax, uint32_t n_live,
                                       uint32_t k, uint32_t imax) {
    const int tid = threadIdx.x;
    const uint32_t w8 = (uint32_t)tid >> 6, lane = (uint32_t)lane_id();
    // this wave's entries: [beg, end)
    uint32_t beg, end;
    if (segmented) {
        beg = w8 * kWaveStride;
        end = beg + min(sm.wcnt[w8], (uint32_t)kWaveCap);
    } else {
        const uint32_t per = (n + kWaves - 1) / kWaves;
        beg = min(n, w8 * per);
        end = min(n, beg + per);
    }
    PHASE_WORD(a, 14, n_live);
    const int64_t out0 = (int64_t)r * a.K + (a.K - k); // first output of this refinement
    uint32_t placed = 0;                                // outputs written so far
    // Live keys: ascending key in [amin, amax], i.e. kappa32 in [~amax, ~amin]
    // (amax = 0: not known, measured by a pass over the entries).
    uint32_t klo = amax ? ~amax : 0u, khi = ~amin;
    if (k == 0) return;
    if (n_live == k || n_live <= kSmall) {
        // every live entry is in, or rank the live ones against each other
        const bool all = n_live == k;
        uint32_t cw = 0;
        for (uint32_t e = beg + lane; e < end; e += 64) {
            const Ent x = read_ent(sm, e, raw);
            cw += (uint32_t)__popcll(__ballot(x.kk - klo <= khi - klo));
        }
        if (lane == 0) { sm.wc[w8] = cw; sm.wk[w8] = cw; }
        __syncthreads();
        uint32_t base, kbase, total;
        wave_bases(sm, base, kbase, total);
        uint64_t *zs = reinterpret_cast<uint64_t *>(sm.hist2);
        for (uint32_t e = beg + lane; e < end; e += 64) {
            const Ent x = read_ent(sm, e, raw);
            const bool lv = x.kk - klo <= khi - klo;
            const uint64_t m = __ballot(lv);
            if (lv) {
                const uint32_t pos = base + __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                            __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
                if (all) put_out(a, out0, pos, sm.ci[e], x.bits);
                else zs[pos] = zkey(x.kk, sm.ci[e]);
            }
            base += (uint32_t)__popcll(m);
        }
        if (!all) {
            __syncthreads();
            rank_small(a, out0, zs, n_live, k, 0u);
        }
        __syncthreads();
        return;
    }
    if (tid < 64) sm.coarse[0][tid] = 0u;
    uint32_t imin = 0u;
    if (amax == 0u) {
        // range pass: min/max kappa32 and index of the live entries
        // (sm.red was reset by the caller before its barrier)
        uint32_t kmn = ~0u, kmx = 0u, imn = ~0u, imx = 0u;
        for (uint32_t e = beg + lane; e < end; e += 64) {
            const uint32_t kk = read_ent(sm, e, raw).kk;
            if (kk <= khi) {
                const uint32_t ix = sm.ci[e];
                kmn = min(kmn, kk); kmx = max(kmx, kk);
                imn = min(imn, ix); imx = max(imx, ix);
            }
        }
        kmn = wave_min_to63(kmn);
        kmx = wave_max_to63(kmx);
        imn = wave_min_to63(imn);
        imx = wave_max_to63(imx);
        if (lane == 63) {
            atomicMin(&sm.red[0], kmn);
            atomicMax(&sm.red[1], kmx);
            atomicMin(&sm.red[2], imn);
            atomicMax(&sm.red[3], imx);
        }
    }
    __syncthreads();
    if (amax == 0u) {
        klo = sm.red[0];
        khi = sm.red[1];
        imin = sm.red[2];
        imax = sm.red[3];
    }
    // first window: all live keys
    Window win = make_window((uint64_t)klo << 32, ((uint64_t)khi << 32) | 0xFFFFFFFFull, imin, imax);
    int rounds_run = 0;
    for (;;) {
        const int par = rounds_run & 1;
        const bool done = win.fast
            ? refine_round<true>(a, sm, beg, end, raw, out0, placed, win, n_live, k, par)
            : refine_round<false>(a, sm, beg, end, raw, out0, placed, win, n_live, k, par);
        rounds_run++;
        if (done) break;
    }
    PHASE_WORD(a, 15, (uint64_t)rounds_run);
    __syncthreads();
}

// ------------------------------------------------------ exact routes ----

// Resolves an exact boundary bin that exceeds the frontier capacity without
// materialising it; every pass re-reads the row.  The bin is a contiguous
// range of ascending FP32 keys, [bin_cutoff(t*), bin_cutoff(t* - 1) - 1].
// Digit rounds narrow a window on the key, largest keys first, until the
// k-th largest key uT of the bin is known; when more elements hold uT than
// are still needed, rounds over the row index narrow a window on the index,
// lowest first (the composite order (kappa32, index)).  A last pass commits
// every bin element above uT and those at uT with index <= iT.  A pass costs
// a range test per element; only elements inside the window go further.
__device__ __forceinline__ void reread_select(const KArgs a, Smem &sm, int r, int64_t off, int64_t L,
                              uint32_t tstar, uint32_t k) {
    const int tid = threadIdx.x;
    const float *scores = a.scores;
    const int32_t n = (int32_t)L;
    const uint32_t bhi = tstar == 0u ? 0xFFFFFFFFu : bin_cutoff(tstar - 1u) - 1u;
    uint32_t wlo = bin_cutoff(tstar), whi = bhi;  // key window
    uint32_t ilo = 0u, ihi = (uint32_t)(n - 1);   // index window at key uT
    uint32_t uT = wlo, iT = 0xFFFFFFFFu;
    bool by_key = wlo != whi;
    // every round narrows its window to fewer than 2^11 parts of it, so the
    // key takes at most three rounds and the index three more
    for (int round = 0; round < 6; round++) {
        const uint32_t span = by_key ? whi - wlo : ihi - ilo;
        if (span == 0u) break;                     // one key / one index left
        const int s = max(0, 21 - (int)__builtin_clz(span)); // span >> s < 2^11
        clear_hist(sm);
        __syncthreads();
        if (by_key) {
            stream_row<false>(scores, off, 0, n, [&](const f4 *x, const int32_t *i0, int32_t lo,
                                                     int32_t hi, bool edge, int32_t mv) {
#pragma unroll
                for (int m = 0; m < kVec; m++) if (m < mv) {
#pragma unroll
                    for (int c = 0; c < 4; c++) {
                        const uint32_t u = asc_key(fbits(x[m][c]));
                        if (u - wlo <= span && (!edge || in_window(i0[m] + c, lo, hi)))
                            atomicAdd(&sm.hist[(whi - u) >> s], 1u);
                    }
                }
            });
        } else {
            stream_row<false>(scores, off, 0, n, [&](const f4 *x, const int32_t *i0, int32_t lo,
                                                     int32_t hi, bool edge, int32_t mv) {
#pragma unroll
                for (int m = 0; m < kVec; m++) if (m < mv) {
#pragma unroll
                    for (int c = 0; c < 4; c++) {
                        const uint32_t u = asc_key(fbits(x[m][c]));
                        const uint32_t di = (uint32_t)(i0[m] + c) - ilo;
                        if (u == uT && di <= span && (!edge || in_window(i0[m] + c, lo, hi)))
                            atomicAdd(&sm.hist[di >> s], 1u);
                    }
                }
            });
        }
        __syncthreads();
        if (tid < 64) wave_find(sm.hist, k, 0, 1, sm.find);
        __syncthreads();
        const Find f = sm.find[0];
        __syncthreads();
        const uint32_t need = k - f.below;
        if (by_key) {
            // digit b holds keys whi - u in [b << s, (b + 1) << s)
            const uint64_t b0 = (uint64_t)f.bin << s, b1 = ((uint64_t)f.bin + 1u) << s;
            const uint32_t nlo = b1 > (uint64_t)span ? wlo : whi - (uint32_t)(b1 - 1u);
            whi = whi - (uint32_t)b0;
            wlo = nlo;
            uT = wlo;
            if (f.eq == need) break;               // the whole digit is taken
            by_key = wlo != whi;                   // else ties at uT: index rounds
        } else {
            ilo += f.bin << s;
            ihi = min(ihi, ilo + ((1u << s) - 1u));
            iT = ihi;
            if (f.eq == need) break;
        }
        k = need;
    }
    // Output pass: bin elements with key above uT, and those at uT with index <= iT.
    const uint32_t tspan = bhi - uT;
    stream_row<false>(scores, off, 0, n, [&](const f4 *x, const int32_t *i0, int32_t lo,
                                             int32_t hi, bool edge, int32_t mv) {
#pragma unroll
        for (int m = 0; m < kVec; m++) if (m < mv) {
#pragma unroll
            for (int c = 0; c < 4; c++) {
                const uint32_t u = asc_key(fbits(x[m][c]));
                const int32_t i = i0[m] + c;
                const bool sel = u - uT <= tspan && (u != uT || (uint32_t)i <= iT) &&
                                 (!edge || in_window(i, lo, hi));
                const uint64_t em = __ballot(sel);
                if (em == 0) continue;
                // one position claim per wave (the output order is free)
                const int lead = __builtin_ctzll(em);
                uint32_t op = 0u;
                if (lane_id() == lead) op = atomicAdd(&sm.opos, (uint32_t)__popcll(em));
                op = __builtin_amdgcn_readlane(op, lead);
                if (sel)
                    emit(a, r, op + __builtin_amdgcn_mbcnt_hi((uint32_t)(em >> 32),
                                         __builtin_amdgcn_mbcnt_lo((uint32_t)em, 0u)),
                         (uint32_t)i, ~u);
            }
        }
    });
    __syncthreads();
}

// Coarse bins of one streamed chunk added into sm.hist.
__device__ __forceinline__ void coarse_hist_chunk(Smem &sm, const f4 *x, const int32_t *i0,
                                                  int32_t lo, int32_t hi, bool edge, int32_t mv) {
#pragma unroll
    for (int m = 0; m < kVec; m++) if (m < mv) {
#pragma unroll
        for (int c = 0; c < 4; c++)
            if (!edge || in_window(i0[m] + c, lo, hi))
                atomicAdd(&sm.hist[coarse_bin(x[m][c])], 1u);
    }
}

// Coarse histogram of row elements [beg, end) into sm.hist (clear before a
// preceding barrier); ends with a barrier.
__device__ __forceinline__ void exact_hist(const KArgs a, Smem &sm, int64_t off, int32_t beg,
                                           int32_t end) {
    stream_row<false>(a.scores, off, beg, end,
                      [&](const f4 *x, const int32_t *i0, int32_t lo, int32_t hi, bool edge,
                          int32_t mv) { coarse_hist_chunk(sm, x, i0, lo, hi, edge, mv); });
    __syncthreads();
}

// C(b0) and C(b1) from the complete coarse histogram in sm.hist (elements
// in bins 0..b), into sm.cnt0 and sm.cnt (zero on entry).  Ends with a
// barrier.
__device__ __forceinline__ void hist_counts(Smem &sm, uint32_t b0, uint32_t b1) {
    const uint32_t t4 = 4u * (uint32_t)threadIdx.x;
    const uint4 h = reinterpret_cast<const uint4 *>(sm.hist)[threadIdx.x];
    auto upto = [&](uint32_t b) {
        return (t4 <= b ? h.x : 0u) + (t4 + 1u <= b ? h.y : 0u) + (t4 + 2u <= b ? h.z : 0u) +
               (t4 + 3u <= b ? h.w : 0u);
    };
    const uint32_t c0 = wave_incl_scan(upto(b0));
    const uint32_t c1 = wave_incl_scan(upto(b1));
    if ((threadIdx.x & 63) == 63) {
        if (c0) atomicAdd(&sm.cnt0, c0);
        if (c1) atomicAdd(&sm.cnt, c1);
    }
    __syncthreads();
}

// Exact coarse recovery (eq:method:exact-init) over the whole row by this
// workgroup: a coarse histogram pass finds tau_star = min{b : C(b) >= K}; a
// classify pass commits c < tau_star to the output (E0) and keeps
// c == tau_star as the frontier Q0 when it fits the capacity.  A row of at
// most kResidentChunks chunks is read once and both passes run from
// registers; a longer one is streamed twice.  Returns (tau_star, |E0|, |Q0|)
// in sm.find[0]; ends with a barrier, sm.hist cleared.  With have_hist the
// coarse histogram is already in sm.hist (exact_hist) and only the classify
// pass runs.
__device__ __forceinline__ void exact_classify(const KArgs a, Smem &sm, int r, int64_t off, int64_t L,
                                               bool have_hist) {
    const int tid = threadIdx.x;
    auto hist = [&](const f4 *x, const int32_t *i0, int32_t lo, int32_t hi, bool edge,
                    int32_t mv) { coarse_hist_chunk(sm, x, i0, lo, hi, edge, mv); };
    // After the find: c < tau_star iff u >= key_hi, c == tau_star iff
    // key_lo <= u < key_hi (the bins' ascending-key endpoints); an empty
    // keep range when the bin does not fit the frontier.  When E0 and Q0 fit
    // the LDS pairs together, E0 is staged at their top (e0_top on) and
    // written out after the pass, so that the pass itself stores nothing to
    // global memory (a store in the loop would make each wait for the next
    // chunk's loads wait for the stores as well).
    uint32_t key_lo = 0, key_hi = 0, e0_top = kFront, below = 0;
    bool stage = false;
    auto find = [&]() {
        PHASE_MARK(a, 22);
        __syncthreads();
        PHASE_MARK(a, 23);
        if (tid < 64) wave_find(sm.hist, (uint32_t)a.K, 0, 1, sm.find);
        if (tid == 0) sm.cnt = 0;
        __syncthreads();
        PHASE_MARK(a, 24);
        const uint32_t tstar = sm.find[0].bin;
        const bool fits = sm.find[0].eq <= (uint32_t)a.cap;
        key_hi = tstar > 0 ? bin_cutoff(tstar - 1) : 0xFFFFFFFFu;
        key_lo = fits ? bin_cutoff(tstar) : key_hi;
        below = sm.find[0].below;
        stage = below + (fits ? sm.find[0].eq : 0u) <= (uint32_t)kFront;
        e0_top = (uint32_t)kFront - below;
    };
    // Appends are wave-aggregated per chunk: each lane builds bit masks of
    // its committed and kept elements, a wave scan of the two counts (packed
    // in one word: at most 16 per lane) gives each lane its first slots, and
    // lane 0 reserves the wave's total with one LDS atomic per category.
    static_assert(kVec * 4 <= 16 && kWaves * 64 * 16 < 65536, "packed counts");
    const int lane = lane_id();
    int32_t *oi = a.out_idx + (int64_t)r * a.K;
    float *ov = a.out_val + (int64_t)r * a.K;
    auto classify = [&](const f4 *x, const int32_t *i0, int32_t lo, int32_t hi, bool edge,
                        int32_t mv) {
        uint32_t mlt = 0, meq = 0;
#pragma unroll
        for (int m = 0; m < kVec; m++) if (m < mv) {
#pragma unroll
            for (int c = 0; c < 4; c++) {
                const uint32_t u = asc_key(fbits(x[m][c]));
                const bool in = !edge || in_window(i0[m] + c, lo, hi);
                mlt |= (in && u >= key_hi ? 1u : 0u) << (m * 4 + c);
                meq |= (in && u >= key_lo && u < key_hi ? 1u : 0u) << (m * 4 + c);
            }
        }
        const uint32_t packed = (uint32_t)__popc(mlt) | ((uint32_t)__popc(meq) << 16);
        const uint32_t incl = wave_incl_scan(packed);
        const uint32_t tot = __builtin_amdgcn_readlane(incl, 63);
        if (tot == 0) return;
        uint32_t bl = 0, be = 0;
        if (lane == 0) {
            if (tot & 0xFFFFu) bl = atomicAdd(&sm.opos, tot & 0xFFFFu);
            if (tot >> 16) be = atomicAdd(&sm.cnt, tot >> 16);
        }
        const uint32_t excl = incl - packed;
        const uint32_t pl0 = __builtin_amdgcn_readfirstlane(bl) + (excl & 0xFFFFu);
        const uint32_t pe0 = __builtin_amdgcn_readfirstlane(be) + (excl >> 16);
        // slot of the element at bit b: the first slot plus the hits below b
        auto write = [&](auto staged) {
            constexpr bool kStaged = decltype(staged)::value;
#pragma unroll
            for (int m = 0; m < kVec; m++) if (m < mv) {
#pragma unroll
                for (int c = 0; c < 4; c++) {
                    const int b = m * 4 + c;
                    const uint32_t below_b = (1u << b) - 1u;
                    const uint32_t i = (uint32_t)(i0[m] + c);
                    if ((mlt >> b) & 1u) {
                        const uint32_t pl = pl0 + (uint32_t)__popc(mlt & below_b);
                        if constexpr (kStaged) {
                            sm.ci[e0_top + pl] = i; // pl < below: inside the top
                            sm.ck[e0_top + pl] = fbits(x[m][c]);
                        } else if (pl < (uint32_t)a.K) { // never false for a consistent selection
                            oi[pl] = (int32_t)i;
                            ov[pl] = x[m][c];
                        }
                    }
                    if ((meq >> b) & 1u) {
                        const uint32_t pe = pe0 + (uint32_t)__popc(meq & below_b);
                        sm.ci[pe] = i;
                        sm.ck[pe] = ~asc_key(fbits(x[m][c]));
                    }
                }
            }
        };
        if (stage) write(std::true_type{});
        else write(std::false_type{});
    };
    const RowVecs g = row_vecs(a.scores, off, 0, (int32_t)L);
    PHASE_MARK(a, 21);
    if (have_hist) {
        find();
        stream_row<false>(a.scores, off, 0, (int32_t)L, classify);
    } else if (g.nch <= kResidentChunks) {
        resident_row(g, 0, (int32_t)L, hist, find, classify);
    } else {
        stream_row<false>(a.scores, off, 0, (int32_t)L, hist);
        find();
        stream_row<false>(a.scores, off, 0, (int32_t)L, classify);
    }
    PHASE_MARK(a, 25);
    if (stage) {
        __syncthreads();
        for (uint32_t e = (uint32_t)tid; e < below; e += kBlock) {
            oi[e] = (int32_t)sm.ci[e0_top + e];
            ov[e] = __builtin_bit_cast(float, sm.ck[e0_top + e]);
        }
    }
    clear_hist(sm);
    __syncthreads();
}

// -------------------------------------------------------- Phase 1 ----

// Row-phased view of eq:method:view: a_r = bit reversal of (r mod s).
__device__ __forceinline__ uint32_t view_phase(int r, int s_log2) {
    if (s_log2 == 0) return 0;
    const uint32_t v = (uint32_t)r & ((1u << s_log2) - 1u);
    return __builtin_bitreverse32(v) >> (32 - s_log2);
}

__device__ __forceinline__ int64_t view_size(int64_t L, uint32_t a, int s_log2) {
    const int64_t s = (int64_t)1 << s_log2;
    return ((int64_t)a < L) ? (L - a + s - 1) >> s_log2 : 0;
}

// floor(x / y) for y >= 1, exact: with x = n y + r (0 < r < y) the quotient
// is 1/y below n + 1, and since (n + 1) y <= x + y < 2^33 that gap exceeds
// half an FP64 ulp of n + 1, so the rounded quotient stays below n + 1.
__device__ __forceinline__ uint32_t udiv32(uint32_t x, uint32_t y) {
    return (uint32_t)floor((double)x / (double)y);
}

// Whether row r is sampled (Section 4.2: long enough for the floor and its
// view at least q1 samples); rows of length <= K take the direct route.
__device__ __forceinline__ bool row_sampled(const KArgs &a, int r, int64_t L) {
    return L > a.K && L >= a.l_samp_min &&
           view_size(L, view_phase(r, a.s_log2), a.s_log2) >= a.q1;
}

// Segment length of a row that the item table cuts into Pe pieces: a multiple
// of 64 elements giving exactly Pe of them (Pe - 1 pieces of 64 ceil(L / 64 Pe)
// < L / Pe + 64 elements fall short of L, as L / Pe >= kSegMin > 64 Pe).
__device__ __forceinline__ int64_t table_seg(int64_t L, int Pe) {
    return 64 * (int64_t)udiv32((uint32_t)L + 64u * (uint32_t)Pe - 1u, 64u * (uint32_t)Pe);
}

// Entry of the item table: row | segment << 14 | (segments - 1) << 20 in x
// (bit 31: no work), the length in y, the offset's low 32 bits in z, its bits
// 32..39 and the row-state slot << 8 in w.
__device__ __forceinline__ uint4 order_entry(uint32_t r, uint32_t p, uint32_t P, int32_t L,
                                             uint64_t o, uint32_t slot) {
    return make_uint4(r | (p << 14) | ((P - 1u) << 20), (uint32_t)L, (uint32_t)o,
                      ((uint32_t)(o >> 32) & 0xFFu) | (slot << 8));
}

// Sum of max(L_r, 0) over all rows of the call (every workgroup of a
// splittable call computes it to size its row's segments); len0 is this
// thread's first term, lens[threadIdx.x] (0 past the last row), loaded
// by the caller ahead of time.  Ends with a barrier.
__device__ __forceinline__ int64_t block_total_length(const KArgs a, int64_t *lsum, int32_t len0) {
    uint64_t s = (uint64_t)max(len0, 0);
    for (int t = threadIdx.x + kBlock; t < a.n_rows; t += kBlock) s += (uint64_t)max(a.lens[t], 0);
    // s < 2^53: wave sums of its bits [0,16), [16,32), [32,53) each fit 32 bits
    const uint32_t lo = wave_incl_scan((uint32_t)s & 0xFFFFu);
    const uint32_t mid = wave_incl_scan((uint32_t)(s >> 16) & 0xFFFFu);
    const uint32_t hi = wave_incl_scan((uint32_t)(s >> 32));
    if (lane_id() == 63)
        lsum[threadIdx.x >> 6] = (int64_t)lo + ((int64_t)mid << 16) + ((int64_t)hi << 32);
    __syncthreads();
    int64_t tot = 0;
#pragma unroll
    for (int w = 0; w < kWaves; w++) tot += lsum[w];
    return tot;
}

// The split plan of a row of length L (KV-split mapping, Section 4.5): when
// rows may be split, the row is cut into P0 = min(pmax, ceil(L / target))
// pieces of equal length rounded up to 64 elements, target = max(kSegMin,
// sum(L) / items), so that the call has at most about seg_items work items;
// P <= P0 <= ceil(L / kSegMin).  total = sum(L) of the call.  Every segment
// of the row computes the same plan.
__device__ __forceinline__ void segment_plan(const KArgs a, int64_t total, int64_t L, int64_t &P,
                                             int64_t &seg) {
    // (a call of more rows than items cuts only the rows longer than the
    // mean, in two: the longest rows no longer bound the call)
    const int64_t items = a.n_rows > a.seg_items ? a.n_rows
                        : a.seg_items > 2 * a.n_rows ? a.seg_items - a.n_rows
                                                     : (a.seg_items + 1) / 2;
    // Divisions in FP64 (a few instructions, where 64-bit integer division
    // takes hundreds).  target and P0 may be off by one after rounding: any
    // target >= kSegMin and any P0 in [1, ceil(L / kSegMin)] make a valid
    // plan, and every segment of the row computes the same one.  seg and P
    // are exact (udiv32).
    const double tq = ceil((double)total / (double)items);
    const uint32_t target = (uint32_t)fmax((double)kSegMin, fmin(tq, 2147483648.0));
    const uint32_t L32 = (uint32_t)L;
    const uint32_t P0 = min((uint32_t)a.pmax, (uint32_t)ceil((double)L32 / (double)target));
    const uint32_t seg32 = (udiv32(L32 + P0 - 1u, P0) + 63u) & ~63u;
    seg = seg32;
    P = udiv32(L32 + seg32 - 1u, seg32);
}

// Phase 1 in two halves.  phase1_issue loads the first kP1 view samples of
// each thread into registers; it runs before the segment's first chunk is
// issued so that waiting for the samples does not wait for the chunk.
// phase1_finish histograms them (and the rest of the view, for views larger
// than kP1 * kBlock), finds tau0 and tau1 and their FP32 endpoints
// (eq:method:sample-hist, eq:method:primary-threshold) into sm.  Every
// segment of a split row computes the same view (no cross-workgroup wait).
// sm.hist must have been cleared, before a barrier preceding phase1_finish
// when synced, else before the call.
constexpr int kP1 = 16;

__device__ __forceinline__ void phase1_issue(const KArgs a, int r, const float *row, int64_t L,
                                             float (&xs)[kP1]) {
    const uint32_t ph = view_phase(r, a.s_log2);
    const int64_t nv = view_size(L, ph, a.s_log2);
    const float *base = row + ph;
#pragma unroll
    for (int j = 0; j < kP1; j++) {
        const int64_t t = threadIdx.x + (int64_t)j * kBlock;
        xs[j] = 0.0f;
        if (t < nv) xs[j] = base[t << a.s_log2];
    }
}

// pub (segment 0 of a split row): where tau0 | tau1 << 16 | 1 << 31 is
// published for the other segments, as soon as it is known.
__device__ __forceinline__ void phase1_finish(const KArgs a, Smem &sm, int r, const float *row,
                                              int64_t L, const float (&xs)[kP1], uint32_t *pub,
                                              bool synced) {
    const int tid = threadIdx.x;
    const uint32_t ph = view_phase(r, a.s_log2);
    const int64_t nv = view_size(L, ph, a.s_log2);
    if (!synced) __syncthreads(); // the clear of sm.hist before the additions
    PHASE_MARK(a, 17);
    // bin counts, and their sums over groups of 32 bins for a two-level find
    auto add = [&](float x) {
        const uint32_t b = coarse_bin(x);
        atomicAdd(&sm.hist[b], 1u);
        atomicAdd(&sm.coarse[0][b >> 5], 1u);
    };
#pragma unroll
    for (int j = 0; j < kP1; j++) {
        const int64_t t = tid + (int64_t)j * kBlock;
        if (t < nv) add(xs[j]);
    }
    const float *base = row + ph;
    int64_t t = tid + (int64_t)kP1 * kBlock;
    for (; t + 3 * kBlock < nv; t += 4 * kBlock) {
        const float x0 = base[(t) << a.s_log2];
        const float x1 = base[(t + kBlock) << a.s_log2];
        const float x2 = base[(t + 2 * kBlock) << a.s_log2];
        const float x3 = base[(t + 3 * kBlock) << a.s_log2];
        add(x0);
        add(x1);
        add(x2);
        add(x3);
    }
    for (; t < nv; t += kBlock) add(base[t << a.s_log2]);
    __syncthreads();
    PHASE_MARK(a, 18);
    // Every wave finds both boundaries itself and stores the same values
    // into sm (each wave reads them back after its own store), so no
    // barrier follows; thread 0 publishes them.  sm.hist stays dirty: every
    // later user clears it first.
    {
        const uint32_t c = sm.coarse[0][lane_id()];
        const uint32_t incl = wave_incl_scan(c);
        const uint32_t total = __builtin_amdgcn_readlane(incl, 63);
        uint32_t t0, t1;
        wave_find_bins2(sm.hist, incl, c, total, (uint32_t)a.q0, (uint32_t)a.q1, t0, t1);
        if (tid == 0 && pub)
            __hip_atomic_store(pub, t0 | (t1 << 16) | 0x80000000u, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
        if (lane_id() == 0) {
            sm.tau0 = t0;
            sm.tau1 = t1;
            sm.cut0 = bin_cutoff(t0);
            sm.cut1 = bin_cutoff(t1);
        }
    }
    PHASE_MARK(a, 19);
}

// Shared view of a split row (Section 4.5 with the view partitioned over the
// segments instead of re-read by each): segment p takes the view positions
// a_r + k s inside its own range [beg, end), k in [k0, k1).
__device__ __forceinline__ void coop_view_range(const KArgs a, int r, int32_t beg, int32_t end,
                                                int64_t &k0, int64_t &k1) {
    const int64_t ph = view_phase(r, a.s_log2), s = (int64_t)1 << a.s_log2;
    k0 = beg > ph ? (beg - ph + s - 1) >> a.s_log2 : 0;
    k1 = end > ph ? (end - ph + s - 1) >> a.s_log2 : 0;
}

__device__ __forceinline__ void coop_view_issue(const KArgs a, int r, const float *row, int64_t k0,
                                                int64_t k1, float (&xs)[kP1]) {
    const float *base = row + view_phase(r, a.s_log2);
#pragma unroll
    for (int j = 0; j < kP1; j++) {
        const int64_t k = k0 + threadIdx.x + (int64_t)j * kBlock;
        xs[j] = 0.0f;
        if (k < k1) xs[j] = base[k << a.s_log2];
    }
}

// Histograms this segment's view samples (sm.hist clear before a preceding
// barrier), adds the non-zero bins into the row's view histogram vh, and
// arrives; the last segment to arrive loads the merged histogram, clears vh,
// finds tau0 and tau1 (eq:method:sample-hist, eq:method:primary-threshold)
// and publishes them in rs->taus, and returns true with them in sm.  The
// others return false (they poll rs->taus).  The merged histogram is that of
// the whole view, so the boundaries are the ones segment 0 alone would find.
__device__ __forceinline__ bool coop_view_finish(const KArgs a, Smem &sm, int r, const float *row,
                                                 int64_t k0, int64_t k1, const float (&xs)[kP1],
                                                 RowState *rs, uint32_t *vh, int64_t P) {
    const int tid = threadIdx.x;
#pragma unroll
    for (int j = 0; j < kP1; j++) {
        const int64_t k = k0 + tid + (int64_t)j * kBlock;
        if (k < k1) atomicAdd(&sm.hist[coarse_bin(xs[j])], 1u);
    }
    const float *base = row + view_phase(r, a.s_log2);
    for (int64_t k = k0 + tid + (int64_t)kP1 * kBlock; k < k1; k += kBlock)
        atomicAdd(&sm.hist[coarse_bin(base[k << a.s_log2])], 1u);
    __syncthreads();
    {
        const uint4 h = reinterpret_cast<const uint4 *>(sm.hist)[tid];
        uint32_t *d = vh + 4 * tid;
        if (h.x) __hip_atomic_fetch_add(d + 0, h.x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (h.y) __hip_atomic_fetch_add(d + 1, h.y, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (h.z) __hip_atomic_fetch_add(d + 2, h.z, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (h.w) __hip_atomic_fetch_add(d + 3, h.w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    // (as for the candidates: every wave's additions complete before the
    // barrier that precedes the arrival)
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (tid == 0) {
        const uint32_t old = __hip_atomic_fetch_add(&rs->varrive, 1u, __ATOMIC_RELAXED,
                                                    __HIP_MEMORY_SCOPE_AGENT);
        sm.flag = old == (uint32_t)(P - 1) ? 2u : 0u;
    }
    __syncthreads();
    if (sm.flag != 2u) return false;
    {
        uint64_t *d = reinterpret_cast<uint64_t *>(vh + 4 * tid);
        const uint64_t lo = __hip_atomic_load(d, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const uint64_t hi = __hip_atomic_load(d + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        reinterpret_cast<uint4 *>(sm.hist)[tid] =
            make_uint4((uint32_t)lo, (uint32_t)(lo >> 32), (uint32_t)hi, (uint32_t)(hi >> 32));
        // cleared for the next call once read (the values are in LDS now)
        __hip_atomic_store(d, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(d + 1, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (tid == 0) __hip_atomic_store(&rs->varrive, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    group_sums(sm.hist, sm.coarse[0]);
    __syncthreads();
    {
        const uint32_t c = sm.coarse[0][lane_id()];
        const uint32_t incl = wave_incl_scan(c);
        const uint32_t total = __builtin_amdgcn_readlane(incl, 63);
        uint32_t t0, t1;
        wave_find_bins2(sm.hist, incl, c, total, (uint32_t)a.q0, (uint32_t)a.q1, t0, t1);
        if (tid == 0)
            __hip_atomic_store(&rs->taus, t0 | (t1 << 16) | 0x80000000u, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
        if (lane_id() == 0) {
            sm.tau0 = t0;
            sm.tau1 = t1;
            sm.cut0 = bin_cutoff(t0);
            sm.cut1 = bin_cutoff(t1);
        }
    }
    return true;
}

// ---------------------------------------------------------- finish ----

// Certification and the routes after Phase 2 (Section 4.3).  For a sampled
// row, C0 = C(tau0) and C1 = C(tau1) are exact and the stored entries hold
// A(tau1) (per-wave regions if `segmented`, else [0, nstored)), complete
// unless `incomplete`.  C0 >= K certifies the proposal (Lemma
// lem:method:containment); C0 < K takes the band up to tau1
// (eq:method:rescue-band) when that suffices; what is still underfilled, or
// does not fit the frontier, runs exact coarse recovery (eq:method:exact-init).
// Every route then enters the same refinement with (E0 in the output, Q0 in
// LDS, k0).  An incomplete store is made up by re-reading the row for the
// tail the route needs.  Also counts the route and writes the trace.
__device__ __forceinline__ void finish_row(const KArgs a, Smem &sm, int r, int64_t off, int64_t L,
                                           int64_t nv, bool sampled, uint32_t C0, uint32_t C1,
                                           bool incomplete, bool segmented, uint32_t nstored,
                                           bool have_hist = false) {
    const uint32_t K = (uint32_t)a.K;
    const uint32_t cap = (uint32_t)a.cap;
    int32_t trC1 = -1, tstar = -1, nq = -1;
    uint32_t route, n_ref = 0, k_ref = K, kmin = 0;
    if (!sampled) {
        route = TOPK_ROUTE_EXACT_UNSAMPLED;
    } else if (C0 >= K && C0 <= cap) {
        route = TOPK_ROUTE_PRIMARY;
        n_ref = C0;
        kmin = sm.cut0;
    } else if (C0 < K) {
        trC1 = (int32_t)C1;
        if (C1 >= K && C1 <= cap) {
            route = TOPK_ROUTE_BAND;
            n_ref = C1;
            kmin = sm.cut1;
        } else {
            route = (C1 < K) ? TOPK_ROUTE_EXACT_UNDERFILL : TOPK_ROUTE_EXACT_OVERFLOW;
        }
    } else {
        route = TOPK_ROUTE_EXACT_OVERFLOW;
    }
    // sm.hist may already hold the row's coarse histogram (have_hist): kept
    // for the exact route, cleared for the others
    const bool exact = route >= TOPK_ROUTE_EXACT_UNSAMPLED;
    have_hist = have_hist && exact;
    if (!have_hist) clear_hist(sm);
    if (threadIdx.x == 0) sm.opos = 0;
    __syncthreads();
    PHASE_MARK(a, 8);
    // Frontier of the certified tail: A(tau0), or A(tau1) for the band, read
    // from the Phase 2 entries (FP32 bits filtered by kmin) or, when those
    // are incomplete, re-collected from the row as kappa32 keys.
    bool f_seg = segmented, f_raw = true;
    uint32_t f_n = nstored;
    // ascending-key bounds of the frontier (f_amax = 0: not known)
    uint32_t f_amin = kmin, f_amax = incomplete ? 0u : sm.amax;
    if (n_ref) {
        if (incomplete) {
            if (threadIdx.x == 0) sm.cnt = 0;
            __syncthreads();
            collect_range<false>(sm, a.scores, off, 0, (int32_t)L, kmin, 0xFFFFFFFFu, true, cap);
            __syncthreads();
            f_seg = false;
            f_raw = false;
            f_n = n_ref;
        }
        nq = (int32_t)n_ref;
    }
    // (the hint keeps this rarely taken code out of the hot path's layout;
    // measured: the decode batch runs ~1 % faster with it)
    if (__builtin_expect(exact, 0)) {
        exact_classify(a, sm, r, off, L, have_hist);
        const Find f = sm.find[0];
        tstar = (int32_t)f.bin;
        nq = (int32_t)f.eq;
        k_ref = K - f.below;
        if (f.eq <= cap) {
            n_ref = f.eq;
            f_seg = false;
            f_raw = false;
            f_n = f.eq;
            // the frontier is coarse bin tau*: ascending keys from its
            // endpoint up; the range pass measures the keys and indices
            // present (a bin of ties then needs only index digits)
            f_amin = bin_cutoff(f.bin);
            f_amax = 0u;
        } else {
            route |= TOPK_ROUTE_REREAD_FLAG;
            reread_select(a, sm, r, off, L, f.bin, k_ref);
        }
    }
    PHASE_MARK(a, 9);
    if (f_amax != 0u && f_amax < f_amin) f_amax = 0u;
    if (n_ref) {
        reset_range(sm);
        __syncthreads();
        refine(a, sm, r, f_seg, f_n, f_raw, f_amin, f_amax, n_ref, k_ref, (uint32_t)(L - 1));
    }
    PHASE_MARK(a, 13);
    if (threadIdx.x == 0) {
        atomicAdd(&a.hdr->stats[route & 7u], 1u);
        if (route & TOPK_ROUTE_REREAD_FLAG) atomicAdd(&a.hdr->stats[kStatReread], 1u);
        if (a.trace) {
            int32_t *t = a.trace + (int64_t)r * TOPK_TRACE_WORDS;
            t[0] = (int32_t)route; t[1] = (int32_t)nv;
            t[2] = sampled ? (int32_t)sm.tau0 : -1; t[3] = sampled ? (int32_t)sm.tau1 : -1;
            t[4] = sampled ? (int32_t)C0 : -1; t[5] = trC1; t[6] = tstar; t[7] = nq;
        }
    }
}

// Finish of a row certified on the primary or band route, straight from its
// candidates in registers (vi, vk: index and FP32 bits): one digit round over
// the live key range [~amax, ~cut] (fine histogram plus 32-bin group sums,
// two-level find), committed entries stored from registers straight to
// consecutive output slots of each wave, the boundary bin ranked (and stored)
// when it holds at most kSmall entries.  Slot (j, thread) holds a candidate iff j < ngroups
// (block-uniform) and j * unit + pos < lim: the merged array of a split row
// has unit = kBlock, pos = thread, lim = count; the per-wave regions of a
// single workgroup have unit = 64, pos = lane, lim = the wave's count.
// Returns false, having written nothing, when the row needs the general
// finish (other routes, unknown range, a tiny or narrow frontier, a large
// boundary bin).  Needs sm.hist and sm.coarse[0] clear.
__device__ __forceinline__ bool finish_fast(const KArgs a, Smem &sm, int r, int64_t nv,
                                            uint32_t C0, uint32_t C1, uint32_t amax,
                                            uint32_t unit, uint32_t pos, uint32_t lim,
                                            uint32_t ngroups, const uint32_t (&vi)[kPer],
                                            const uint32_t (&vk)[kPer]) {
    const int tid = threadIdx.x;
    const uint32_t lane = (uint32_t)lane_id();
    const uint32_t K = (uint32_t)a.K, cap = (uint32_t)a.cap;
    uint32_t route, kmin, n_live;
    if (C0 >= K && C0 <= cap) {
        route = TOPK_ROUTE_PRIMARY; kmin = sm.cut0; n_live = C0;
    } else if (C0 < K && C1 >= K && C1 <= cap) {
        route = TOPK_ROUTE_BAND; kmin = sm.cut1; n_live = C1;
    } else {
        return false;
    }
    if (amax == 0u || amax < kmin || n_live <= kSmall || n_live == K) return false;
    const uint32_t klo = ~amax, khi = ~kmin;
    const uint64_t span0 = ((uint64_t)(khi - klo) << 32) | 0xFFFFFFFFull;
    const int bits0 = 64 - __clzll((long long)span0);
    const Window win = key_window((uint64_t)klo << 32, ((uint64_t)khi << 32) | 0xFFFFFFFFull,
                                  bits0 > 11 ? (uint32_t)(bits0 - 11) : 0u);
    if (!win.fast || win.kspan == 0xFFFFFFFFu) return false;
    PHASE_MARK(a, 8);
    // histogram of the live keys (sm.hist and its group sums are clear);
    // tl[j]: key offset in the window, ~0 for a slot that is not live (the
    // window spans less than 2^32 - 1 keys, so ~0 is no live offset)
    // (slot groups j >= ngroups hold no entry: skipped uniformly)
    uint32_t tl[kPer];
#pragma unroll
    for (int j = 0; j < kPer; j++) {
        tl[j] = 0xFFFFFFFFu;
        if ((uint32_t)j < ngroups) {
            const uint32_t t = ~asc_key(vk[j]) - win.klo;
            const bool lv = (uint32_t)j * unit + pos < lim && t <= win.kspan;
            if (lv) {
                tl[j] = t;
                const uint32_t d = t >> win.wf;
                atomicAdd(&sm.hist[d], 1u);
                atomicAdd(&sm.coarse[0][d >> 5], 1u);
            }
        }
    }
    if (tid == 0) { sm.knext = 0u; sm.opos = 0u; }
    __syncthreads();
    PHASE_MARK(a, 9);
    // every wave locates the boundary bin itself (no second barrier)
    Find f;
    {
        const uint32_t c = sm.coarse[0][lane];
        const uint32_t incl = wave_incl_scan(c);
        const uint32_t total = __builtin_amdgcn_readlane(incl, 63);
        f = wave_find_reg(sm.hist, incl, c, total, K);
    }
    PHASE_MARK(a, 10);
    const uint32_t need = K - f.below;
    const bool take_all = f.eq == need;
    if (f.bin >= (uint32_t)kBins || (!take_all && f.eq > kSmall)) return false;
    // committed: offset below cend (bin b excluded, or included with
    // take_all); kept: offset in [cb, ce] (bin b) when not take_all
    const uint32_t cb = f.bin << win.wf;
    const uint32_t ce = min(cb + (((uint32_t)1 << win.wf) - 1u), win.kspan);
    const uint32_t cend = take_all ? ce + 1u : cb;
    const uint32_t kw = ce - cb; // keep iff tl - cb <= kw (never for ~0: ce < ~0)
    // each wave reserves its committed slots with one LDS atomic (slot order
    // is free: the outputs are a set), so no barrier is needed before placing
    uint32_t cw = 0;
#pragma unroll
    for (int j = 0; j < kPer; j++)
        if ((uint32_t)j < ngroups) cw += (uint32_t)__popcll(__ballot(tl[j] < cend));
    uint32_t cbase = 0;
    if (lane == 0 && cw) cbase = atomicAdd(&sm.opos, cw);
    cbase = __builtin_amdgcn_readfirstlane(cbase);
    PHASE_MARK(a, 11);
    const int64_t out0 = (int64_t)r * a.K;
    uint64_t *zs = reinterpret_cast<uint64_t *>(sm.hist2);
    // committed entries go straight to their output slots (slot order is
    // free: the outputs are a set)
#pragma unroll
    for (int j = 0; j < kPer; j++) {
        if ((uint32_t)j >= ngroups) continue;
        const bool commit = tl[j] < cend;
        const uint64_t mc = __ballot(commit);
        if (commit) {
            const uint32_t pos = cbase + __builtin_amdgcn_mbcnt_hi((uint32_t)(mc >> 32),
                                               __builtin_amdgcn_mbcnt_lo((uint32_t)mc, 0u));
            put_out(a, out0, pos, vi[j], vk[j]);
        }
        cbase += (uint32_t)__popcll(mc);
        const bool keep = !take_all && tl[j] - cb <= kw;
        const uint64_t mk = __ballot(keep);
        if (mk) {
            const uint32_t first = (uint32_t)__ffsll((unsigned long long)mk) - 1u;
            uint32_t kb = 0;
            if (lane == first) kb = atomicAdd(&sm.knext, (uint32_t)__popcll(mk));
            kb = __builtin_amdgcn_readlane(kb, first);
            if (keep)
                zs[kb + __builtin_amdgcn_mbcnt_hi((uint32_t)(mk >> 32),
                            __builtin_amdgcn_mbcnt_lo((uint32_t)mk, 0u))] =
                    zkey(~asc_key(vk[j]), vi[j]);
        }
    }
    PHASE_MARK(a, 12);
    PHASE_WORD(a, 30, f.eq);
    PHASE_WORD(a, 15, ngroups);
    if (!take_all) {
        __syncthreads();
        rank_small_to(zs, f.eq, need, f.below, [&](uint32_t pos, uint32_t idx, uint32_t bits) {
            put_out(a, out0, pos, idx, bits);
        });
    }
    PHASE_MARK(a, 13);
    if (tid == 0) {
        atomicAdd(&a.hdr->stats[route], 1u);
        if (a.trace) {
            int32_t *t = a.trace + (int64_t)r * TOPK_TRACE_WORDS;
            t[0] = (int32_t)route; t[1] = (int32_t)nv;
            t[2] = (int32_t)sm.tau0; t[3] = (int32_t)sm.tau1;
            t[4] = (int32_t)C0; t[5] = route == TOPK_ROUTE_BAND ? (int32_t)C1 : -1;
            t[6] = -1; t[7] = (int32_t)n_live;
        }
    }
    return true;
}

// ----------------------------------------------------------- kernel ----

// Leaves a split row's state zeroed for the next call (graph replays).
// x: also the split exact route's fields (written only in calls run from
// the item table).
__device__ __forceinline__ void reset_row_state(RowState *rs, bool x = true) {
    __hip_atomic_store(&rs->counts, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&rs->sa, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&rs->incomplete, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&rs->amax, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&rs->taus, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&rs->varrive, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (!x) return;
    __hip_atomic_store(&rs->xtau, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&rs->ocnt, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&rs->qcnt, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&rs->arrive2, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&rs->xmask, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ------------------------------------------- split exact recovery ----
//
// Exact coarse recovery (eq:method:exact-init) of a split row whose
// candidates overflowed, spread over its segments.  Every segment with an
// overflowed region has added the coarse histogram of its range, exact in
// bins 0..tau1 (its stored entries and the hits Phase 2 counted past its
// region), into the row's histogram; the finisher adds the other segments'
// stored candidates (all of their elements with c <= tau1), which makes the
// histogram the row's own in bins 0..tau1, where tau_star lies when
// C(tau1) >= K.  It publishes
// tau_star, and each segment then classifies its own range (the finisher the
// stored candidates): c < tau_star into the row's output (E0), c == tau_star
// into the candidate buffer (Q0), at slots reserved with one atomic per
// segment from its own histogram's counts.  The last to finish refines Q0.

constexpr uint64_t kXGo = 0x80000000u, kXAbandon = 0x40000000u;

// Entries of h in bins < t and in bin t, into sm.cnt0 and sm.cnt (zero
// before a preceding barrier).  Ends with a barrier.
__device__ __forceinline__ void hist_lt_eq(Smem &sm, const uint32_t *h, uint32_t t) {
    const uint32_t t4 = 4u * (uint32_t)threadIdx.x;
    const uint4 v = reinterpret_cast<const uint4 *>(h)[threadIdx.x];
    const uint32_t lt = (t4 < t ? v.x : 0u) + (t4 + 1u < t ? v.y : 0u) +
                        (t4 + 2u < t ? v.z : 0u) + (t4 + 3u < t ? v.w : 0u);
    const uint32_t eq = (t4 == t ? v.x : 0u) + (t4 + 1u == t ? v.y : 0u) +
                        (t4 + 2u == t ? v.z : 0u) + (t4 + 3u == t ? v.w : 0u);
    const uint32_t clt = wave_incl_scan(lt), ceq = wave_incl_scan(eq);
    if ((threadIdx.x & 63) == 63) {
        if (clt) atomicAdd(&sm.cnt0, clt);
        if (ceq) atomicAdd(&sm.cnt, ceq);
    }
    __syncthreads();
}

// Classify pass over row elements [beg, end): ascending keys u >= key_hi
// (c < tau_star) go to the row's output at glt + rank, key_lo <= u < key_hi
// (c == tau_star) to gc[geq + rank] as index | FP32 bits << 32; the caller
// reserved [glt, glt + n_lt) and [geq, geq + n_eq), the range's counts of the
// two.  Appends are wave-aggregated per chunk (bit masks, one wave scan, one
// LDS atomic per category); when both sets fit the LDS pairs they are staged
// there and written out after the pass, so that the loop stores nothing to
// global memory.  sm.opos and sm.cnt must be zero before a preceding
// barrier.  Ends with a barrier.
__device__ __forceinline__ void classify_range(const KArgs a, Smem &sm, int r, int64_t off,
                                               int32_t beg, int32_t end, uint32_t key_lo,
                                               uint32_t key_hi, uint32_t n_lt, uint32_t n_eq,
                                               uint32_t glt, uint32_t geq, uint64_t *gc) {
    const int tid = threadIdx.x;
    const int lane = lane_id();
    const bool stage = n_lt + n_eq <= (uint32_t)kFront;
    const uint32_t top = (uint32_t)kFront - n_lt; // staged E0 at [top, kFront)
    int32_t *oi = a.out_idx + (int64_t)r * a.K;
    float *ov = a.out_val + (int64_t)r * a.K;
    static_assert(kVec * 4 <= 16 && kWaves * 64 * 16 < 65536, "packed counts");
    stream_row<false>(a.scores, off, beg, end, [&](const f4 *x, const int32_t *i0, int32_t lo,
                                                   int32_t hi, bool edge, int32_t mv) {
        uint32_t mlt = 0, meq = 0;
#pragma unroll
        for (int m = 0; m < kVec; m++) if (m < mv) {
#pragma unroll
            for (int c = 0; c < 4; c++) {
                const uint32_t u = asc_key(fbits(x[m][c]));
                const bool in = !edge || in_window(i0[m] + c, lo, hi);
                mlt |= (in && u >= key_hi ? 1u : 0u) << (m * 4 + c);
                meq |= (in && u >= key_lo && u < key_hi ? 1u : 0u) << (m * 4 + c);
            }
        }
        const uint32_t packed = (uint32_t)__popc(mlt) | ((uint32_t)__popc(meq) << 16);
        const uint32_t incl = wave_incl_scan(packed);
        const uint32_t tot = __builtin_amdgcn_readlane(incl, 63);
        if (tot == 0) return;
        uint32_t bl = 0, be = 0;
        if (lane == 0) {
            if (tot & 0xFFFFu) bl = atomicAdd(&sm.opos, tot & 0xFFFFu);
            if (tot >> 16) be = atomicAdd(&sm.cnt, tot >> 16);
        }
        const uint32_t excl = incl - packed;
        uint32_t pl = __builtin_amdgcn_readfirstlane(bl) + (excl & 0xFFFFu);
        uint32_t pe = __builtin_amdgcn_readfirstlane(be) + (excl >> 16);
#pragma unroll
        for (int m = 0; m < kVec; m++) if (m < mv) {
#pragma unroll
            for (int c = 0; c < 4; c++) {
                const int b = m * 4 + c;
                const uint32_t i = (uint32_t)(i0[m] + c);
                const uint32_t bits = fbits(x[m][c]);
                if ((mlt >> b) & 1u) {
                    // (never false for consistent counts)
                    if (pl < n_lt && glt + pl < (uint32_t)a.K) {
                        if (stage) {
                            sm.ci[top + pl] = i;
                            sm.ck[top + pl] = bits;
                        } else {
                            oi[glt + pl] = (int32_t)i;
                            ov[glt + pl] = x[m][c];
                        }
                    }
                    pl++;
                }
                if ((meq >> b) & 1u) {
                    if (pe < n_eq && geq + pe < (uint32_t)kFront) {
                        if (stage) {
                            sm.ci[pe] = i;
                            sm.ck[pe] = bits;
                        } else {
                            __hip_atomic_store(&gc[geq + pe], (uint64_t)i | ((uint64_t)bits << 32),
                                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        }
                    }
                    pe++;
                }
            }
        }
    });
    if (stage) {
        __syncthreads();
        for (uint32_t e = (uint32_t)tid; e < n_lt && glt + e < (uint32_t)a.K; e += kBlock) {
            oi[glt + e] = (int32_t)sm.ci[top + e];
            ov[glt + e] = __builtin_bit_cast(float, sm.ck[top + e]);
        }
        for (uint32_t e = (uint32_t)tid; e < n_eq && geq + e < (uint32_t)kFront; e += kBlock)
            __hip_atomic_store(&gc[geq + e], (uint64_t)sm.ci[e] | ((uint64_t)sm.ck[e] << 32),
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
}

// Counts of the histogram h (LDS) for tau_star, the reservation of their
// slots, and the classify pass over [beg, end).  Ends with a barrier.
__device__ __forceinline__ void classify_own_range(const KArgs a, Smem &sm, int r, int64_t off,
                                                   int32_t beg, int32_t end, const uint32_t *h,
                                                   uint32_t ts, RowState *rs, uint64_t *gc) {
    if (threadIdx.x == 0) { sm.cnt0 = 0; sm.cnt = 0; sm.opos = 0; }
    __syncthreads();
    hist_lt_eq(sm, h, ts);
    const uint32_t n_lt = sm.cnt0, n_eq = sm.cnt;
    __syncthreads(); // every thread has read the counts
    if (threadIdx.x == 0) {
        sm.cnt = 0;
        sm.flag = n_lt ? __hip_atomic_fetch_add(&rs->ocnt, n_lt, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT) : 0u;
        sm.base = n_eq ? __hip_atomic_fetch_add(&rs->qcnt, n_eq, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT) : 0u;
    }
    __syncthreads();
    PHASE_MARK(a, 31);
    const uint32_t glt = sm.flag, geq = sm.base;
    const uint32_t key_hi = ts > 0 ? bin_cutoff(ts - 1u) : 0xFFFFFFFFu, key_lo = bin_cutoff(ts);
    classify_range(a, sm, r, off, beg, end, key_lo, key_hi, n_lt, n_eq, glt, geq, gc);
}

// The finisher's share: the complete segments' stored candidates, held in
// registers (slot j kBlock + tid < stored).  Ends with a barrier.
__device__ __forceinline__ void classify_stored(const KArgs a, Smem &sm, int r, RowState *rs,
                                                uint64_t *gc, const uint32_t (&vi)[kPer],
                                                const uint32_t (&vk)[kPer], uint32_t stored,
                                                uint32_t ts) {
    const int tid = threadIdx.x;
    const uint32_t w8 = (uint32_t)tid >> 6;
    const uint32_t key_hi = ts > 0 ? bin_cutoff(ts - 1u) : 0xFFFFFFFFu, key_lo = bin_cutoff(ts);
    uint32_t nl = 0, ne = 0;
#pragma unroll
    for (int j = 0; j < kPer; j++) {
        const uint32_t u = asc_key(vk[j]);
        const bool in = (uint32_t)(j * kBlock + tid) < stored;
        nl += (in && u >= key_hi) ? 1u : 0u;
        ne += (in && u >= key_lo && u < key_hi) ? 1u : 0u;
    }
    // per-thread counts of at most kPer, wave sums below 2^16
    const uint32_t own = nl | (ne << 16);
    const uint32_t incl = wave_incl_scan(own);
    if (lane_id() == 63) sm.wc[w8] = incl;
    __syncthreads();
    uint32_t wpre = 0, tot = 0;
#pragma unroll
    for (uint32_t v = 0; v < (uint32_t)kWaves; v++) {
        const uint32_t c = sm.wc[v];
        wpre += v < w8 ? c : 0u;
        tot += c;
    }
    if (tid == 0) {
        sm.flag = (tot & 0xFFFFu) ? __hip_atomic_fetch_add(&rs->ocnt, tot & 0xFFFFu, __ATOMIC_RELAXED,
                                                           __HIP_MEMORY_SCOPE_AGENT) : 0u;
        sm.base = (tot >> 16) ? __hip_atomic_fetch_add(&rs->qcnt, tot >> 16, __ATOMIC_RELAXED,
                                                       __HIP_MEMORY_SCOPE_AGENT) : 0u;
    }
    __syncthreads();
    const uint32_t first = wpre + incl - own;
    uint32_t pl = sm.flag + (first & 0xFFFFu), pe = sm.base + (first >> 16);
    int32_t *oi = a.out_idx + (int64_t)r * a.K;
    float *ov = a.out_val + (int64_t)r * a.K;
#pragma unroll
    for (int j = 0; j < kPer; j++) {
        const uint32_t u = asc_key(vk[j]);
        const bool in = (uint32_t)(j * kBlock + tid) < stored;
        if (in && u >= key_hi) {
            if (pl < (uint32_t)a.K) { // never false for consistent counts
                oi[pl] = (int32_t)vi[j];
                ov[pl] = __builtin_bit_cast(float, vk[j]);
            }
            pl++;
        } else if (in && u >= key_lo) {
            if (pe < (uint32_t)kFront)
                __hip_atomic_store(&gc[pe], (uint64_t)vi[j] | ((uint64_t)vk[j] << 32),
                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            pe++;
        }
    }
    __syncthreads();
}

// Second arrival at a split row in the exact route; xt0 is the arriving
// segment's view of the route word (0: it stopped waiting, and its segment
// bit in xmask is set first).  Returns the route word for the last arrival,
// 0 for the others.  Each wave's stores complete before the barrier that
// precedes the arrival (as for the first arrival).
__device__ __forceinline__ uint64_t arrive_again(Smem &sm, RowState *rs, int p, uint64_t xt0) {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) {
        if (!(xt0 & kXGo)) {
            __hip_atomic_fetch_or(&rs->xmask, 1ull << p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __builtin_amdgcn_s_waitcnt(0); // the bit is set before the arrival counts
        }
        const uint32_t old = __hip_atomic_fetch_add(&rs->arrive2, 1u, __ATOMIC_RELAXED,
                                                    __HIP_MEMORY_SCOPE_AGENT);
        // the finisher publishes the route word before its own arrival, so a
        // last arrival always sees it
        const uint64_t xt = __hip_atomic_load(&rs->xtau, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        sm.xword = ((xt & kXGo) && old + 1u == ((uint32_t)(xt >> 11) & 0xFFu)) ? xt : 0ull;
    }
    __syncthreads();
    return sm.xword;
}

// The last arrival of the split exact route: loads Q0 and refines it for the
// remaining K - |E0| outputs, records the row and resets its state.  Returns
// false, with nothing done, when a segment stopped waiting (its range is not
// classified): the caller then runs the whole row's exact route, which
// rewrites every output; sm.wk[2] and sm.wk[3] hold C(tau1) and C(tau0).
__device__ __forceinline__ bool split_exact_final(const KArgs a, Smem &sm, int r, int64_t L,
                                                  int64_t nv, RowState *rs, uint64_t *gc,
                                                  uint64_t xt) {
    const int tid = threadIdx.x;
    const uint32_t ts = (uint32_t)xt & 0x7FFu;
    const uint32_t eq = min((uint32_t)(xt >> 32) & 0x3FFFu, (uint32_t)kFront);
    const uint32_t below = (uint32_t)(xt >> 48) & 0x3FFFu;
    // the segment mask and the counts (|E0|, |Q0| and tau_star came with the
    // route word)
    if (tid == 0) {
        const uint64_t m = __hip_atomic_load(&rs->xmask, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const uint64_t cc = __hip_atomic_load(&rs->counts, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        sm.wk[0] = m != 0ull;
        sm.wk[2] = (uint32_t)cc;
        sm.wk[3] = (uint32_t)(cc >> 32);
    }
    __syncthreads();
    PHASE_MARK(a, 8);
    if (sm.wk[0]) return false;
    const uint32_t C1 = sm.wk[2], C0 = sm.wk[3];
    // Q0 as kappa32 keys, four loads in flight per thread
    for (uint32_t e0 = 0; e0 < eq; e0 += 4 * kBlock) {
        uint64_t q[4];
#pragma unroll
        for (int j = 0; j < 4; j++) {
            const uint32_t e = e0 + (uint32_t)(j * kBlock + tid);
            q[j] = e < eq ? __hip_atomic_load(&gc[e], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                          : 0ull;
        }
#pragma unroll
        for (int j = 0; j < 4; j++) {
            const uint32_t e = e0 + (uint32_t)(j * kBlock + tid);
            if (e < eq) {
                sm.ci[e] = (uint32_t)q[j];
                sm.ck[e] = ~asc_key((uint32_t)(q[j] >> 32));
            }
        }
    }
    clear_hist(sm);
    reset_range(sm);
    if (tid == 0) sm.opos = 0;
    __syncthreads();
    PHASE_MARK(a, 9);
    const uint32_t amin = bin_cutoff(ts);
    refine(a, sm, r, false, eq, false, amin, 0u, eq, (uint32_t)a.K - below, (uint32_t)(L - 1));
    PHASE_MARK(a, 13);
    if (tid == 0) {
        atomicAdd(&a.hdr->stats[TOPK_ROUTE_EXACT_OVERFLOW], 1u);
        if (a.trace) {
            int32_t *t = a.trace + (int64_t)r * TOPK_TRACE_WORDS;
            t[0] = TOPK_ROUTE_EXACT_OVERFLOW; t[1] = (int32_t)nv;
            t[2] = (int32_t)sm.tau0; t[3] = (int32_t)sm.tau1;
            t[4] = (int32_t)C0; t[5] = C0 < (uint32_t)a.K ? (int32_t)C1 : -1;
            t[6] = (int32_t)ts; t[7] = (int32_t)eq;
        }
        reset_row_state(rs);
    }
    return true;
}

// kOrdered: the call runs from the item table (a.order set).  Only such calls
// take the split exact route; the other instance has none of its code (with
// it, the decode batch measured 3 % slower although it never runs it).
template <bool kOrdered>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(4))) void
topk_ragged_kernel(KArgs a) {
    __shared__ Smem sm;
    const int tid = threadIdx.x;
    const int item = blockIdx.x;
#ifdef TOPK_PHASE_TIMERS
    if (a.timers && tid == 0)
        for (int k = 0; k < 32; k++) g_tmarks[k] = 0;
    TimerFlush timer_flush{a.timers};
#endif
    const int pi = item / a.n_rows;
    // Every load the prologue needs goes out at once: the row's length and
    // offset (from the item table when the call has one), the workspace
    // header, and this thread's first term of the segment plan's length sum
    // (used only when rows may be split).  (all loaded unconditionally and
    // selected afterwards: a branch here would cost a second round trip)
    constexpr bool ordered = kOrdered;
    // rows split by plan (never in an item-table call)
    const bool plan_split = !kOrdered && a.pmax > 1;
    const int ri = item - pi * a.n_rows;
    // (an item-table call never splits by plan and takes the row from its
    // entry: it loads no length or offset, and its wait holds no vector load,
    // which under load would queue behind the other workgroup's stream)
    const uint4 e = *(ordered ? a.order + item : reinterpret_cast<const uint4 *>(a.hdr));
    const int32_t len_i = ordered ? 0 : a.lens[ri];
    const int64_t off_i = ordered ? 0 : a.offs[ri];
    const int32_t len0_raw = ordered ? 0 : a.lens[min(tid, a.n_rows - 1)];
    const uint4 hw = *reinterpret_cast<const uint4 *>(a.hdr); // magic, split_rows, max_rows
    // (keeps the compiler from sinking each load to its first use, which
    // would make them several round trips instead of one)
    asm volatile("" ::"s"(e.x), "s"(e.y), "s"(e.z), "s"(e.w), "s"(len_i), "s"(off_i), "s"(hw.x),
                 "s"(hw.y), "s"(hw.z), "v"(len0_raw));
    if (ordered && (e.x >> 31)) return; // an item past the call's last segment
    // the row, its segment, the segments the item table gives it (0: none,
    // the plan decides), and its row-state block
    const int r = ordered ? (int)(e.x & 0x3FFFu) : ri;
    const int p = ordered ? (int)((e.x >> 14) & 63u) : pi;
    const int Pe = ordered ? (int)((e.x >> 20) & 63u) + 1 : 0;
    const uint32_t slot = ordered ? e.w >> 8 : (uint32_t)r;
    const int32_t len_r = ordered ? (int32_t)e.y : len_i;
    const int64_t off = ordered ? (int64_t)((((uint64_t)e.w & 0xFFu) << 32) | e.z) : off_i;
    const int64_t L = (int64_t)max(len_r, 0);
    const float *row = a.scores + off;
    PHASE_MARK(a, 0);
    PHASE_WORD(a, 6, (uint64_t)__smid());
    PHASE_WORD(a, 7, (uint64_t)p | ((uint64_t)r << 32)); // (segments filled in later)

    // Workspace check: a split plan needs per-row state for every row.
    const bool ws_bad = (hw.x != kMagic) | ((uint32_t)a.n_rows > hw.z) |
                        (plan_split & ((uint32_t)a.n_rows > hw.y));
    if (__builtin_expect(ws_bad, 0)) {
        if (p == 0) {
            write_error_row(a, r);
            if (tid == 0 && r == 0) atomicAdd(&a.hdr->stats[kStatErrors], 1u);
        }
        return;
    }
    // A row longer than TOPK_L_MAX would overflow the 32-bit byte offsets of
    // its vectors: it is not selected, and counted as an error.
    if (__builtin_expect(L > (int64_t)TOPK_L_MAX, 0)) {
        if (p == 0) {
            write_error_row(a, r);
            if (tid == 0) atomicAdd(&a.hdr->stats[kStatErrors], 1u);
        }
        return;
    }

    if (L <= a.K) {
        if (p == 0) {
            write_direct(a, r, row, L);
            if (tid == 0) {
                atomicAdd(&a.hdr->stats[TOPK_ROUTE_DIRECT], 1u);
                if (a.trace) {
                    int32_t *t = a.trace + (int64_t)r * TOPK_TRACE_WORDS;
                    t[0] = TOPK_ROUTE_DIRECT;
                    for (int w = 1; w < TOPK_TRACE_WORDS; w++) t[w] = -1;
                }
            }
        }
        return;
    }

    const uint32_t ph = view_phase(r, a.s_log2);
    const int64_t nv = view_size(L, ph, a.s_log2);
    const bool sampled = row_sampled(a, r, L);
    if (!sampled && p > 0) return; // unsampled rows run whole on segment 0

    char *rb = a.rows + (size_t)slot * kRowBlockBytes;
    RowState *rs = reinterpret_cast<RowState *>(rb);
    uint32_t *vh = reinterpret_cast<uint32_t *>(rb + kRowStateBytes);
    uint32_t *xh = reinterpret_cast<uint32_t *>(a.rows + (size_t)hw.y * kRowBlockBytes) +
                   (size_t)slot * kBins;
    // the row's merged candidates: index | FP32 bits << 32
    uint64_t *gc = reinterpret_cast<uint64_t *>(rb + kRowStateBytes + kViewHistBytes);
    uint32_t C0 = 0, C1 = 0, nstored = 0;
    bool incomplete = false, segmented = true, split = false, have_hist = false;
    // split exact route: this segment added its coarse histogram; second
    // arrivals the finisher expects (0: none)
    bool pushed = false, redo = false;
    uint32_t xexpect = 0;

    if (sampled) {
        // A row has at most ceil(L / kSegMin) segments (see below).
        if ((int64_t)p * kSegMin >= L) return;
        clear_hist(sm);
        if constexpr (kOrdered) {
            // the hits Phase 2's regions cannot keep
            uint4 *h2 = reinterpret_cast<uint4 *>(sm.hist2);
            for (int i = tid; i < kBins / 4; i += kBlock) h2[i] = make_uint4(0, 0, 0, 0);
        }
        if (tid == 0) { sm.cnt = 0; sm.cnt0 = 0; sm.incomplete = 0; sm.amax = 0; }
        // Segment 0 reads the view; its loads go out first, the segment plan
        // and the first chunk follow, and the view is histogrammed with that
        // chunk in flight.  A large view of a split row is shared instead:
        // each segment reads the part inside its own range (after the plan).
        float xs[kP1];
        const bool big_view = (nv >= kCoopView && plan_split) || (nv >= kCoopViewTable && Pe > 1);
        if (p == 0 && !big_view) phase1_issue(a, r, row, L, xs);
        // Segments: segment_plan when every row may be split, else the item
        // table's count.
        int64_t P = 1, seg = L;
        if (plan_split) {
            segment_plan(a, block_total_length(a, sm.lsum, tid < a.n_rows ? len0_raw : 0), L, P, seg);
        } else if (Pe > 1) {
            P = Pe;
            seg = table_seg(L, Pe);
        }
        if (p >= P) return;
        split = P > 1;
        const int32_t beg = (int32_t)(p * seg);
        const int32_t end = (int32_t)min(L, p * seg + seg);
        const bool coop = split && big_view;
        int64_t k0 = 0, k1 = 0;
        if (coop) {
            coop_view_range(a, r, beg, end, k0, k1);
            coop_view_issue(a, r, row, k0, k1, xs);
        } else if (p == 0 && big_view) {
            phase1_issue(a, r, row, L, xs); // not split: the whole view, after the plan
        }
        // Phase 2 over this segment: certify against cut0 and keep A(tau1).
        // The endpoints come from segment 0 (or, for a shared view, from the
        // last segment to add its part), which publishes tau0 and tau1 in one
        // agent-scope atomic word (the endpoints follow from the bins); the
        // other segments poll for it with their first chunk in flight.  The
        // wait is bounded, by a poll count and by spin_ticks of the
        // constant-rate clock: after either, the segment builds the whole
        // view itself (the same boundaries).  That bound is what guarantees
        // progress: a row's segments are normally resident together (a call
        // has fewer work items than resident workgroups), but another kernel
        // sharing the GPU can keep the publishing segment from running, and
        // with a shared view any segment may wait for one dispatched after it.
        PHASE_MARK(a, 16);
        phase2_collect<kOrdered>(sm, a.scores, off, beg, end, [&]() {
            bool have = false; // endpoints in sm
            if (coop) {
                // (orders the clear of sm.hist before the additions: only a
                // split plan's length sum has a barrier after it)
                if (!plan_split) __syncthreads();
                have = coop_view_finish(a, sm, r, row, k0, k1, xs, rs, vh, P);
            } else if (p == 0) {
                // (a split plan's length sum ended with a barrier)
                // (in an item-table call the waves that find the boundaries,
                // and below those of a finisher, issue ahead of the CU's
                // streaming waves: the edge mix 74.8 -> 73.7 us; in the
                // other instance it made the decode batch slower)
                if constexpr (kOrdered) __builtin_amdgcn_s_setprio(2);
                phase1_finish(a, sm, r, row, L, xs, split ? &rs->taus : nullptr, plan_split);
                if constexpr (kOrdered) __builtin_amdgcn_s_setprio(0);
                have = true;
            }
            if (!have) {
                if (tid == 0) {
                    uint32_t v = 0;
                    const uint64_t t_wait = wall_clock64();
                    for (int spin = 0; spin < a.spin_limit; spin++) {
                        v = __hip_atomic_load(&rs->taus, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        if ((v & 0x80000000u) || wall_clock64() - t_wait > a.spin_ticks) break;
                        __builtin_amdgcn_s_sleep(1);
                    }
                    PHASE_MARK(a, 20);
                    if (__builtin_expect((v & 0x80000000u) != 0, 1)) {
                        sm.flag = 1u;
                        sm.tau0 = v & 0xFFFFu;
                        sm.tau1 = (v >> 16) & 0x7FFFu;
                        sm.cut0 = bin_cutoff(sm.tau0);
                        sm.cut1 = bin_cutoff(sm.tau1);
                    } else {
                        sm.flag = 0u;
                        atomicAdd(&a.hdr->stats[kStatWaitFallback], 1u);
                    }
                }
                __syncthreads();
                if (__builtin_expect(sm.flag == 0u, 0)) {
                    // the whole view, on its own (sm.hist may hold this
                    // segment's part of a shared view)
                    clear_hist(sm);
                    __syncthreads();
                    phase1_issue(a, r, row, L, xs);
                    phase1_finish(a, sm, r, row, L, xs, nullptr, true);
                }
            }
            PHASE_MARK(a, 1);
        });
        // Split rows publish this segment's entries and counts
        // (eq:method:split-local), then arrive; the last arrival merges them
        // (eq:method:split-reduce) and finishes the row.  When the row has few
        // segments each wave publishes on its own, with no workgroup barrier
        // before the arrival: it reserves slots for its entries in the row's
        // merged array (the atomic's round trip overlaps its count of
        // C(tau0)), adds its two counts in one 64-bit atomic and its maximum,
        // and copies its region; a wave whose region overflowed re-counts the
        // positions it streams and marks the row incomplete.  With many
        // segments (whose per-wave atomics on the same words would queue), and
        // in a call run from the item table, the workgroup counts and
        // publishes as one, and a segment with an overflowed region publishes
        // its coarse histogram instead of entries.  Either way the workgroup
        // arrives once.
        const uint32_t w8 = (uint32_t)tid >> 6, lane = (uint32_t)lane_id();
        const bool wave_publish = split && P <= kWavePublishMaxSegs && !ordered;
        uint32_t wcnt = 0, dst = 0; // this wave's stored entries, and their first slot
        if (wave_publish) {
            const uint32_t cur_w = sm.wcnt[w8]; // this wave's own count
            if (__builtin_expect(cur_w <= (uint32_t)kWaveCap, 1)) {
                wcnt = cur_w;
                uint32_t wres = 0;
                if (lane == 0 && wcnt)
                    wres = (uint32_t)__hip_atomic_fetch_add(&rs->sa, (uint64_t)wcnt,
                                                            __ATOMIC_RELAXED,
                                                            __HIP_MEMORY_SCOPE_AGENT);
                const uint32_t beg_e = w8 * kWaveStride, end_e = beg_e + wcnt;
                uint32_t c = 0, mx = 0;
                for (uint32_t e = beg_e + lane; e < end_e; e += 64) {
                    const uint32_t u = asc_key(sm.ck[e]);
                    c += u >= sm.cut0 ? 1u : 0u;
                    mx = max(mx, u);
                }
                c = __builtin_amdgcn_readlane(wave_incl_scan(c), 63);
                mx = __builtin_amdgcn_readlane(wave_max_to63(mx), 63);
                if (lane == 0 && wcnt) {
                    __hip_atomic_fetch_add(&rs->counts, (uint64_t)wcnt | ((uint64_t)c << 32),
                                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    __hip_atomic_fetch_max(&rs->amax, mx, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT);
                }
                dst = __builtin_amdgcn_readfirstlane(wres);
            } else {
                const uint2 cc = count_range_wave(a.scores, off, beg, end, sm.cut0, sm.cut1);
                if (lane == 0) {
                    if (cc.x | cc.y)
                        __hip_atomic_fetch_add(&rs->counts, (uint64_t)cc.y | ((uint64_t)cc.x << 32),
                                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    __hip_atomic_store(&rs->incomplete, 1u, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
                }
            }
            PHASE_MARK(a, 2);
        } else {
            __syncthreads();
            C1 = sm.cnt;
            incomplete = sm.incomplete != 0;
            uint32_t wpre = 0, nst = 0, resv = 0;
            if (split) {
                // (an incomplete segment publishes a histogram instead)
#pragma unroll
                for (uint32_t v = 0; v < (uint32_t)kWaves; v++) {
                    const uint32_t cv = incomplete ? 0u : min(sm.wcnt[v], (uint32_t)kWaveCap);
                    wcnt = v == w8 ? cv : wcnt;
                    wpre += v < w8 ? cv : 0u;
                    nst += cv;
                }
                if (tid == 0 && nst)
                    resv = (uint32_t)__hip_atomic_fetch_add(&rs->sa, (uint64_t)nst,
                                                            __ATOMIC_RELAXED,
                                                            __HIP_MEMORY_SCOPE_AGENT);
            }
            // C(tau0): from the stored A(tau1) entries.  When a wave region
            // overflowed (that wave stopped early), this segment is re-read
            // for its coarse histogram, which gives C(tau0) and C(tau1) and is
            // the first pass of the exact route, should the row take it: a
            // row on one workgroup keeps it, a split row's segment adds it
            // into the row's coarse histogram xh for the finisher.
            if (__builtin_expect(incomplete, 0)) {
                __syncthreads(); // every thread has read sm.cnt
                if (tid == 0) sm.cnt = 0; // (sm.cnt0 is still zero)
                if constexpr (kOrdered) {
                    // Phase 2 went on past the overflow: its stored entries
                    // plus the hits in sm.hist2 make the coarse histogram,
                    // exact in bins 0..tau1 (enough for C(tau0), C(tau1), and
                    // for tau_star when C(tau1) >= K)
                    reinterpret_cast<uint4 *>(sm.hist)[tid] =
                        reinterpret_cast<const uint4 *>(sm.hist2)[tid];
                    __syncthreads();
                    const uint32_t w8 = (uint32_t)tid >> 6;
                    const uint32_t nw = min(sm.wcnt[w8], (uint32_t)kWaveCap);
                    for (uint32_t e = (uint32_t)lane_id(); e < nw; e += 64)
                        atomicAdd(&sm.hist[coarse_bin(__builtin_bit_cast(
                                      float, sm.ck[w8 * kWaveStride + e]))], 1u);
                    __syncthreads();
                    hist_counts(sm, sm.tau0, sm.tau1);
                } else {
                    if (!split) clear_hist(sm);
                    __syncthreads();
                    if (split) {
                        count_range(sm, a.scores, off, beg, end, sm.cut0, sm.cut1);
                    } else {
                        exact_hist(a, sm, off, beg, end);
                        hist_counts(sm, sm.tau0, sm.tau1);
                    }
                }
                if (!split) {
                    // (a histogram exact only up to tau1 serves when C(tau1) >= K)
                    have_hist = !kOrdered || sm.cnt >= (uint32_t)a.K;
                } else if (kOrdered) {
                    const uint4 h = reinterpret_cast<const uint4 *>(sm.hist)[tid];
                    uint32_t *d = xh + 4 * tid;
                    if (h.x) __hip_atomic_fetch_add(d + 0, h.x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    if (h.y) __hip_atomic_fetch_add(d + 1, h.y, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    if (h.z) __hip_atomic_fetch_add(d + 2, h.z, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    if (h.w) __hip_atomic_fetch_add(d + 3, h.w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    pushed = true; // (and sm.hist is kept for the classify pass)
                }
                C0 = sm.cnt0;
                C1 = sm.cnt;
            } else {
                C0 = count_tail(sm, sm.cut0);
            }
            PHASE_MARK(a, 2);
            if (split) {
                if (tid == 0) {
                    sm.base = resv;
                    if (C1 | C0)
                        __hip_atomic_fetch_add(&rs->counts, (uint64_t)C1 | ((uint64_t)C0 << 32),
                                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    if (incomplete)
                        __hip_atomic_fetch_add(&rs->incomplete, 1u, __ATOMIC_RELAXED,
                                               __HIP_MEMORY_SCOPE_AGENT);
                    else if (nst)
                        __hip_atomic_fetch_max(&rs->amax, sm.amax, __ATOMIC_RELAXED,
                                               __HIP_MEMORY_SCOPE_AGENT);
                }
                __syncthreads();
                dst = sm.base + wpre;
            }
        }
        PHASE_WORD(a, 7, (uint64_t)p | ((uint64_t)P << 16) | ((uint64_t)r << 32));

        if (split) {
            // each wave copies its own region, consecutive slots
            for (uint32_t e = lane; e < wcnt; e += 64) {
                const uint32_t d = dst + e;
                const uint32_t t = w8 * kWaveStride + e;
                if (d < (uint32_t)kFront)
                    __hip_atomic_store(&gc[d], ((uint64_t)sm.ck[t] << 32) | sm.ci[t],
                                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            // (the histogram is cleared for the finisher's use while the
            // copies complete)
            if (!pushed) clear_hist(sm);
            // Every value another workgroup reads (entries, counts, the
            // arrival counter) is an agent-scope atomic access, which the
            // hardware keeps coherent across the XCDs' L2 caches without a
            // writeback or invalidate of the whole L2.  Each wave waits until
            // its own accesses have completed; after the barrier all of them
            // are visible device-wide, before the arrival is made.
            __builtin_amdgcn_s_waitcnt(0);
            __syncthreads();
            if (tid == 0) {
                const uint64_t old = __hip_atomic_fetch_add(&rs->sa, 1ull << 32, __ATOMIC_RELAXED,
                                                            __HIP_MEMORY_SCOPE_AGENT);
                sm.flag = ((uint32_t)(old >> 32) == (uint32_t)(P - 1)) ? 2u : 0u;
                sm.base = (uint32_t)old; // every segment has reserved by now
            }
            __syncthreads();
            PHASE_MARK(a, 3);
            if (sm.flag != 2u) {
                if (__builtin_expect(!pushed, 1)) return;
                // Split exact route: wait for the finisher's route word
                // (bounded as the boundary wait; after it the last arrival
                // classifies this range), classify this range, arrive again.
                if (tid == 0) {
                    uint64_t v = 0;
                    const uint64_t t_wait = wall_clock64();
                    for (int spin = 0; spin < a.spin_limit; spin++) {
                        v = __hip_atomic_load(&rs->xtau, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        if ((v & kXGo) || wall_clock64() - t_wait > a.spin_ticks) break;
                        __builtin_amdgcn_s_sleep(1);
                    }
                    sm.xword = v;
                    if (!(v & kXGo)) atomicAdd(&a.hdr->stats[kStatWaitFallback], 1u);
                }
                __syncthreads();
                PHASE_MARK(a, 29);
                const uint64_t xv = sm.xword;
                if ((xv & (kXGo | kXAbandon)) == kXGo)
                    classify_own_range(a, sm, r, off, beg, end, sm.hist,
                                              (uint32_t)xv & 0x7FFu, rs, gc);
                PHASE_MARK(a, 27);
                const uint64_t xt = arrive_again(sm, rs, p, xv);
                PHASE_MARK(a, 28);
                if (!xt) return;
                if (xt & kXAbandon) {
                    if (tid == 0) reset_row_state(rs);
                    return;
                }
                if (split_exact_final(a, sm, r, L, nv, rs, gc, xt)) {
                    PHASE_MARK(a, 5);
                    return;
                }
                redo = true;
            }

            if (!redo) {
            if constexpr (kOrdered) __builtin_amdgcn_s_setprio(2); // (see the boundaries)
            // Finisher (its sm.cut0, cut1, tau0, tau1 are the row's endpoints).
            // The counts and the slot groups that hold candidates are loaded
            // in one round trip (slots past the stored count in the last
            // group hold stale words, ignored), all as agent-scope atomics;
            // each wave loads the counts itself, so no barrier follows.
            const uint32_t stored = sm.base;
            const uint32_t ngroups = (min(stored, (uint32_t)kFront) + kBlock - 1) / kBlock;
            uint32_t c1 = 0, c0 = 0, inc = 0, amx = 0;
            if (lane == 0) {
                const uint64_t cc = __hip_atomic_load(&rs->counts, __ATOMIC_RELAXED,
                                                      __HIP_MEMORY_SCOPE_AGENT);
                c1 = (uint32_t)cc;
                c0 = (uint32_t)(cc >> 32);
                inc = __hip_atomic_load(&rs->incomplete, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                amx = __hip_atomic_load(&rs->amax, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            uint32_t vi[kPer], vk[kPer];
#pragma unroll
            for (int j = 0; j < kPer; j++) {
                uint64_t v = 0;
                if ((uint32_t)j < ngroups)
                    v = __hip_atomic_load(&gc[j * kBlock + tid], __ATOMIC_RELAXED,
                                          __HIP_MEMORY_SCOPE_AGENT);
                vi[j] = (uint32_t)v;
                vk[j] = (uint32_t)(v >> 32);
            }
            C1 = __builtin_amdgcn_readfirstlane(c1);
            C0 = __builtin_amdgcn_readfirstlane(c0);
            amx = __builtin_amdgcn_readfirstlane(amx);
            incomplete = __builtin_amdgcn_readfirstlane(inc) != 0 || stored > (uint32_t)kFront;
            if (tid == 0) sm.amax = amx; // for the general finish (barriers follow)
            nstored = incomplete ? 0u : stored;
            segmented = false;
            PHASE_MARK(a, 4);
            if (!incomplete &&
                finish_fast(a, sm, r, nv, C0, C1, amx, kBlock, (uint32_t)tid, nstored,
                            ngroups, vi, vk)) {
                PHASE_MARK(a, 5);
                if (tid == 0) reset_row_state(rs, false); // (no segment took the exact route)
                return;
            }
            // general finish: the merged frontier into LDS
            __syncthreads();
#pragma unroll
            for (int j = 0; j < kPer; j++) {
                const uint32_t t = (uint32_t)(j * kBlock + tid);
                if (t < nstored) {
                    sm.ci[t] = vi[j];
                    sm.ck[t] = vk[j];
                }
            }
            // segments that added a coarse histogram (block publishing only)
            const uint32_t nx =
                kOrdered && !wave_publish ? __builtin_amdgcn_readfirstlane(inc) : 0u;
            if (__builtin_expect(nx != 0, 0)) {
                // The overflowed segments' merged coarse histogram, cleared
                // for the next call once read (this segment's own, if it
                // added one, is kept in sm.ck for its classify pass).  Every
                // other segment stored all of its elements with c <= tau1;
                // with them added the histogram is the row's own in bins
                // 0..tau1, which holds tau_star whenever C(tau1) >= K (an
                // overflowing row).
                uint64_t *d = reinterpret_cast<uint64_t *>(xh + 4 * tid);
                const uint64_t lo = __hip_atomic_load(d, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                const uint64_t hi = __hip_atomic_load(d + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                if (pushed)
                    reinterpret_cast<uint4 *>(sm.ck)[tid] = reinterpret_cast<const uint4 *>(sm.hist)[tid];
                reinterpret_cast<uint4 *>(sm.hist)[tid] =
                    make_uint4((uint32_t)lo, (uint32_t)(lo >> 32), (uint32_t)hi, (uint32_t)(hi >> 32));
                __hip_atomic_store(d, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(d + 1, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                const uint32_t cap = (uint32_t)a.cap, K = (uint32_t)a.K;
                have_hist = stored <= (uint32_t)kFront && (C0 > cap || (C0 < K && C1 > cap));
                if (have_hist) {
                    __syncthreads();
#pragma unroll
                    for (int j = 0; j < kPer; j++)
                        if ((uint32_t)(j * kBlock + tid) < stored)
                            atomicAdd(&sm.hist[coarse_bin(__builtin_bit_cast(float, vk[j]))], 1u);
                }
                __syncthreads();
                bool dist = false;
                if (have_hist) {
                    if (tid < 64) wave_find(sm.hist, K, 0, 1, sm.find);
                    __syncthreads();
                    dist = sm.find[0].eq <= cap;
                }
                // every segment that added a histogram waits for the route
                // word; this workgroup arrives once more as well
                xexpect = nx + (pushed ? 0u : 1u);
                if (dist) {
                    const Find f = sm.find[0];
                    if (tid == 0)
                        __hip_atomic_store(&rs->xtau,
                                           kXGo | ((uint64_t)xexpect << 11) | f.bin |
                                               ((uint64_t)f.eq << 32) | ((uint64_t)f.below << 48),
                                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    PHASE_MARK(a, 4);
                    classify_stored(a, sm, r, rs, gc, vi, vk, stored, f.bin);
                    PHASE_MARK(a, 26);
                    if (pushed) classify_own_range(a, sm, r, off, beg, end, sm.ck, f.bin, rs, gc);
                    PHASE_MARK(a, 27);
                    const uint64_t xt = arrive_again(sm, rs, p, kXGo);
                    PHASE_MARK(a, 28);
                    if (!xt) return;
                    if (split_exact_final(a, sm, r, L, nv, rs, gc, xt)) {
                        PHASE_MARK(a, 5);
                        return;
                    }
                    redo = true;
                } else if (tid == 0) {
                    // any other route runs here, on this workgroup
                    __hip_atomic_store(&rs->xtau, kXGo | kXAbandon | ((uint64_t)xexpect << 11),
                                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                }
            }
            __syncthreads();
            } // !redo
            if (__builtin_expect(redo, 0)) {
                // A segment of the split exact route stopped waiting: this
                // last arrival runs the row's exact route on its own, which
                // rewrites every output (the others are done with the row).
                C1 = sm.wk[2];
                C0 = sm.wk[3];
                incomplete = true;
                nstored = 0;
                segmented = false;
                have_hist = false;
                xexpect = 0;
                __syncthreads();
            }
        }
    }

    if (sampled && !split && !incomplete) {
        // A single workgroup's candidates, each wave's region into its own
        // lanes' registers.
        const uint32_t w8 = (uint32_t)tid >> 6, lane = (uint32_t)lane_id();
        const uint32_t cnt = min(sm.wcnt[w8], (uint32_t)kWaveCap);
        uint32_t cmax = 0;
#pragma unroll
        for (uint32_t v = 0; v < (uint32_t)kWaves; v++) cmax = max(cmax, min(sm.wcnt[v], (uint32_t)kWaveCap));
        uint32_t vi[kPer], vk[kPer];
#pragma unroll
        for (int j = 0; j < kPer; j++) {
            const uint32_t e = (uint32_t)j * 64u + lane;
            vi[j] = 0u;
            vk[j] = 0u;
            if (e < cnt) {
                vi[j] = sm.ci[w8 * kWaveStride + e];
                vk[j] = sm.ck[w8 * kWaveStride + e];
            }
        }
        clear_hist(sm);
        __syncthreads();
        if (finish_fast(a, sm, r, nv, C0, C1, sm.amax, 64u, lane, cnt, (cmax + 63u) / 64u, vi,
                        vk)) {
            PHASE_MARK(a, 5);
            return;
        }
        __syncthreads();
    }
    finish_row(a, sm, r, off, L, nv, sampled, C0, C1, incomplete, segmented, nstored,
                      have_hist);
    PHASE_MARK(a, 5);

    // the row state is reset once every segment is done with it
    if (split) {
        if (xexpect) {
            if (arrive_again(sm, rs, p, kXGo) && tid == 0) reset_row_state(rs);
        } else if (tid == 0) {
            reset_row_state(rs, kOrdered && redo);
        }
    }
}

// Length class of a row for the longest-first order: 8 classes per octave
// of the length (rows shorter than 8 elements: the length itself), so the
// class never decreases with the length; at most 247.
__device__ __forceinline__ uint32_t length_class(int32_t L) {
    if (L < 8) return L <= 0 ? 0u : (uint32_t)L;
    const uint32_t e = 31u - (uint32_t)__clz(L);
    return e * 8u + (((uint32_t)L >> (e - 3u)) & 7u);
}

// Pre-pass of a call with more rows than resident workgroups: a counting
// sort of the rows by length class, longest first (any order within a
// class), then the work items in that order into order[0, n + extra).
// One workgroup; n <= kOrderMaxRows, extra <= kOrderExtra.  Thread t takes
// rows [R t, R (t + 1)), and a run of equal classes among them takes one LDS
// atomic: rows of similar length would otherwise all add into one counter at
// once.  R = 1 when the rows fit the workgroup (each row's rank costs its
// thread a dependent LDS atomic: a call of 1024 rows of random lengths spent
// 3.5 us ranking on one wave), else kOrderPer, which places each wave's 1024
// rows of a class as one block (smaller blocks made the chunked-prefill block
// 2 % slower: see the order's measurements).
//
// Splitting (KV-split mapping, Section 4.5, for calls too large to split
// every row): a sampled row among the kOrderBlock longest gets
// P = min(kMaxSplit, L / kSegMin, ceil(L / S)) segments, S = max(kSegMin,
// sum(L) / slots), the mean work of a resident workgroup, so that no row
// outlasts the call on one workgroup.  Going down the order, rows keep their
// segments while the extra items stay within `extra` and the split rows
// within the workspace's per-row state (slot k for the k-th split row);
// every later row runs whole.  A row's segments are consecutive items, and
// items past the last are marked empty.
template <int R>
__global__ __launch_bounds__(kOrderBlock) void row_order_kernel(KArgs a, uint4 *order,
                                                                int32_t extra, int32_t slots) {
    static_assert(R == 1 || R == kOrderPer, "rows per thread");
    constexpr uint32_t kNone = 256; // class of a position past the last row
    constexpr int kW = kOrderBlock / 64;
    __shared__ uint32_t cnt[256];
    __shared__ uint32_t rinfo[kOrderBlock]; // by rank: extra segments, then the plan
    __shared__ uint32_t rrow[kOrderBlock];  // by rank: the row and its length
    __shared__ int32_t rlen[kOrderBlock];
    __shared__ uint32_t wtot[kW];
    __shared__ int64_t lsum[kW];
    __shared__ uint32_t ecap_s;
    const int n = a.n_rows;
    const int tid = threadIdx.x;
    const int w = tid >> 6;
    const int i0 = tid * R;
    if (tid < 256) cnt[tid] = 0;
    if (tid == 0) ecap_s = 0;
    rlen[tid] = 0;
    const uint32_t max_split = a.hdr->split_rows;
    int32_t Ls[kOrderPer];
    int64_t Os[kOrderPer]; // loaded with the lengths: one round trip to memory
    // (16-byte loads where the arrays allow and a thread takes kOrderPer
    // rows: its rows are contiguous, so the lanes of one load are 64 bytes
    // apart)
    const bool vec = R == kOrderPer && ((reinterpret_cast<uintptr_t>(a.lens) |
                       reinterpret_cast<uintptr_t>(a.offs)) & 15u) == 0 && i0 + kOrderPer <= n;
    if (vec) {
        const int4 *l4 = reinterpret_cast<const int4 *>(a.lens + i0);
        const longlong2 *o2 = reinterpret_cast<const longlong2 *>(a.offs + i0);
#pragma unroll
        for (int q = 0; q < kOrderPer / 4; q++) {
            const int4 v = l4[q];
            Ls[4 * q] = v.x; Ls[4 * q + 1] = v.y; Ls[4 * q + 2] = v.z; Ls[4 * q + 3] = v.w;
        }
#pragma unroll
        for (int q = 0; q < kOrderPer / 2; q++) {
            const longlong2 v = o2[q];
            Os[2 * q] = v.x; Os[2 * q + 1] = v.y;
        }
    } else {
#pragma unroll
        for (int j = 0; j < kOrderPer; j++) {
            Ls[j] = j < R && i0 + j < n ? a.lens[i0 + j] : 0;
            Os[j] = j < R && i0 + j < n ? a.offs[i0 + j] : 0;
        }
    }
    uint32_t cls[kOrderPer], run[kOrderPer]; // run[j]: rows of j's run from j on
#pragma unroll
    for (int j = 0; j < kOrderPer; j++)
        cls[j] = j < R && i0 + j < n ? length_class(Ls[j]) : kNone;
    run[kOrderPer - 1] = 1;
#pragma unroll
    for (int j = kOrderPer - 2; j >= 0; j--) run[j] = cls[j] == cls[j + 1] ? run[j + 1] + 1 : 1;
    // the call's total length (at most 2^14 rows of < 2^31: wave sums of the
    // bits [0,16), [16,32) and [32,36) of each thread's sum fit 32 bits)
    uint64_t ls = 0;
#pragma unroll
    for (int j = 0; j < kOrderPer; j++) ls += cls[j] != kNone ? (uint64_t)max(Ls[j], 0) : 0u;
    {
        const uint32_t lo = wave_incl_scan((uint32_t)ls & 0xFFFFu);
        const uint32_t mid = wave_incl_scan((uint32_t)(ls >> 16) & 0xFFFFu);
        const uint32_t hi = wave_incl_scan((uint32_t)(ls >> 32));
        if (lane_id() == 63) lsum[w] = (int64_t)lo + ((int64_t)mid << 16) + ((int64_t)hi << 32);
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kOrderPer; j++)
        if (cls[j] != kNone && (j == 0 || cls[j] != cls[j - 1])) atomicAdd(&cnt[cls[j]], run[j]);
    __syncthreads();
    if (tid < 64) {
        // start of class c = rows in classes above c; lane l holds classes
        // 255 - 4l .. 252 - 4l, longest first
        uint32_t c4[4], t = 0;
#pragma unroll
        for (int k = 0; k < 4; k++) { c4[k] = cnt[255 - 4 * tid - k]; t += c4[k]; }
        uint32_t acc = wave_incl_scan(t) - t;
#pragma unroll
        for (int k = 0; k < 4; k++) { cnt[255 - 4 * tid - k] = acc; acc += c4[k]; }
    }
    int64_t total = 0;
#pragma unroll
    for (int q = 0; q < kW; q++) total += lsum[q];
    const uint32_t S = (uint32_t)fmax((double)kSegMin,
                                      fmin(ceil((double)total / (double)slots), 2147483648.0));
    const float rS = __builtin_amdgcn_rcpf((float)S);
    __syncthreads();
    // ranks; the desired segments of the kOrderBlock longest rows
    uint32_t rk[kOrderPer];
    uint32_t pos = 0;
#pragma unroll
    for (int j = 0; j < kOrderPer; j++) {
        rk[j] = 0xFFFFFFFFu;
        if (cls[j] == kNone) continue;
        if (j == 0 || cls[j] != cls[j - 1]) pos = atomicAdd(&cnt[cls[j]], run[j]);
        else pos++;
        rk[j] = pos;
        if (pos < (uint32_t)kOrderBlock) {
            rrow[pos] = (uint32_t)(i0 + j);
            rlen[pos] = Ls[j];
        }
    }
    __syncthreads();
    {
        // thread tid: the segments of rank tid
        const int32_t L = rlen[tid];
        uint32_t P = 1;
        if (L >= 2 * kSegMin && L <= (int32_t)TOPK_L_MAX && row_sampled(a, (int)rrow[tid], L)) {
            // ceil(L / S) from a single-precision quotient (off by at most
            // one: L / S < 2^18) and one exact integer correction
            uint32_t q = (uint32_t)ceilf((float)L * rS);
            if ((uint64_t)q * S < (uint64_t)L) q++;
            else if (q > 1u && (uint64_t)(q - 1u) * S >= (uint64_t)L) q--;
            P = min(min((uint32_t)kMaxSplit, (uint32_t)L / (uint32_t)kSegMin), q);
        }
        rinfo[tid] = P - 1u;
    }
    {
        // rank tid: extra segments E and split rows Ns up to and including it
        // (sums of at most 63 x 1024 and 1024, packed in one word)
        const uint32_t x = rinfo[tid];
        const uint32_t winc = wave_incl_scan(x | (x ? 1u << 16 : 0u));
        if (lane_id() == 63) wtot[w] = winc;
        __syncthreads();
        uint32_t inc = winc;
#pragma unroll
        for (int q = 0; q < kW; q++) inc += q < w ? wtot[q] : 0u;
        const uint32_t E = inc & 0xFFFFu, Ns = inc >> 16;
        const bool kept = E <= (uint32_t)extra && Ns <= max_split;
        const uint32_t em = wave_max_to63(kept ? E : 0u);
        if (lane_id() == 63 && em) atomicMax(&ecap_s, em);
        __syncthreads();
        const uint32_t ecap = ecap_s;
        // items of the ranks before this one beyond their first, segments,
        // slot (a kept rank's prefix never exceeds ecap)
        const uint32_t ex = min(E - x, ecap);
        const uint32_t xk = kept ? x : 0u;
        rinfo[tid] = ex | (xk << 11) | ((xk ? Ns - 1u : 0u) << 17);
    }
    __syncthreads();
    const uint32_t ecap = ecap_s;
#pragma unroll
    for (int j = 0; j < kOrderPer; j++) {
        if (rk[j] == 0xFFFFFFFFu) continue;
        const uint32_t k = rk[j];
        uint32_t base = k + ecap, P = 1, slot = 0;
        if (k < (uint32_t)kOrderBlock) {
            const uint32_t inf = rinfo[k];
            base = k + (inf & 0x7FFu);
            P = ((inf >> 11) & 63u) + 1u;
            slot = inf >> 17;
        }
        for (uint32_t q = 0; q < P; q++)
            order[base + q] = order_entry((uint32_t)(i0 + j), q, P, Ls[j], (uint64_t)Os[j], slot);
    }
    for (uint32_t i = ecap + (uint32_t)tid; i < (uint32_t)extra; i += kOrderBlock)
        order[n + i] = make_uint4(0x80000000u, 0u, 0u, 0u);
}

// Workspace set-up: header and zeroed per-row state (the candidate arrays
// need no initialisation: only entries below the published count are read).
__global__ void ws_init_kernel(WsHeader *hdr, char *rows, uint32_t split_rows, uint32_t max_rows,
                               uint32_t cap) {
    for (uint32_t r = blockIdx.x; r < split_rows; r += gridDim.x) {
        uint32_t *w = reinterpret_cast<uint32_t *>(rows + (size_t)r * kRowBlockBytes);
        for (uint32_t i = threadIdx.x; i < (kRowStateBytes + kViewHistBytes) / 4; i += blockDim.x)
            w[i] = 0;
        uint32_t *x = reinterpret_cast<uint32_t *>(rows + (size_t)split_rows * kRowBlockBytes +
                                                   (size_t)r * kViewHistBytes);
        for (uint32_t i = threadIdx.x; i < kBins; i += blockDim.x) x[i] = 0;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        hdr->split_rows = split_rows;
        hdr->max_rows = max_rows;
        hdr->cap = cap;
        for (int s = 0; s < 16; s++) hdr->stats[s] = 0;
        hdr->magic = kMagic;
    }
}

__global__ void stats_reset_kernel(WsHeader *hdr) {
    if (threadIdx.x < 16) hdr->stats[threadIdx.x] = 0;
}

__global__ void debug_coarse_kernel(const float *x, int64_t n, uint16_t *out) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) out[i] = (uint16_t)coarse_bin(x[i]);
}

__global__ void debug_cutoff_kernel(uint32_t *out) {
    const int t = blockIdx.x * blockDim.x + threadIdx.x;
    if (t < kBins) out[t] = bin_cutoff((uint32_t)t);
}

// ------------------------------------------------------------- host ----

// Read-only ceiling of a call: the same work items as topk_ragged_kernel
// (the same item table or split plan; every other row is read by one
// workgroup) stream every valid score once with the same
// loads (two chunks of 16-byte non-temporal loads in flight per thread) and
// keep only the largest ascending key, which one atomic per workgroup adds
// into out_max[r] (atomics on one address queue: one per wave made the
// long-split batch's ceiling 1.5 times slower than the selector itself).  It
// measures what reading the call's rows costs in this launch geometry, with
// none of the selection.
__global__ __launch_bounds__(kBlock) void read_ceiling_kernel(KArgs a, uint32_t *out_max) {
    __shared__ int64_t lsum[kWaves];
    __shared__ uint32_t wmax[kWaves];
    const int tid = threadIdx.x;
    const int pi = blockIdx.x / a.n_rows;
    const bool ordered = a.order != nullptr;
    const uint4 e = ordered ? a.order[blockIdx.x] : make_uint4(0u, 0u, 0u, 0u);
    if (ordered && (e.x >> 31)) return;
    const int r = ordered ? (int)(e.x & 0x3FFFu) : (int)blockIdx.x - pi * a.n_rows;
    const int p = ordered ? (int)((e.x >> 14) & 63u) : pi;
    const int Pe = ordered ? (int)((e.x >> 20) & 63u) + 1 : 0;
    const int32_t len_r = a.lens[r];
    const int64_t off = a.offs[r];
    const int32_t len0 = a.lens[min(tid, a.n_rows - 1)];
    const int64_t L = (int64_t)max(len_r, 0);
    const bool sampled = row_sampled(a, r, L);
    if (!sampled && p > 0) return;
    int64_t P = 1, seg = L;
    if (sampled && a.pmax > 1) {
        if ((int64_t)p * kSegMin >= L) return;
        segment_plan(a, block_total_length(a, lsum, tid < a.n_rows ? len0 : 0), L, P, seg);
    } else if (sampled && Pe > 1) {
        P = Pe;
        seg = table_seg(L, Pe);
    }
    if (p >= P) return;
    const int32_t beg = (int32_t)(p * seg);
    const int32_t end = (int32_t)min(L, p * seg + seg);
    uint32_t mx = 0;
    stream_row<true>(a.scores, off, beg, end, [&](const f4 *x, const int32_t *i0, int32_t lo,
                                                   int32_t hi, bool, int32_t mv) {
#pragma unroll
        for (int m = 0; m < kVec; m++) if (m < mv) {
#pragma unroll
            for (int c = 0; c < 4; c++) {
                const uint32_t u = asc_key(fbits(x[m][c]));
                mx = in_window(i0[m] + c, lo, hi) ? max(mx, u) : mx;
            }
        }
    });
    mx = wave_max_to63(mx);
    if (lane_id() == 63) wmax[tid >> 6] = mx;
    __syncthreads();
    if (tid == 0) {
        uint32_t m = 0;
#pragma unroll
        for (int w = 0; w < kWaves; w++) m = max(m, wmax[w]);
        atomicMax(&out_max[r], m);
    }
}

struct DeviceInfo {
    int cus = 0;
    int clock_khz = 0; // rate of the constant-rate clock (wall_clock64)
    bool ok = false;
};

int device_info(DeviceInfo *di) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return TOPK_ELAUNCH;
    static thread_local int cached_dev = -1;
    static thread_local DeviceInfo cached;
    if (dev != cached_dev) {
        hipDeviceProp_t prop;
        if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return TOPK_ELAUNCH;
        cached.cus = prop.multiProcessorCount;
        int khz = 0;
        if (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess ||
            khz <= 0)
            khz = 100000; // 100 MHz, the rate on gfx9 parts
        cached.clock_khz = khz;
        cached.ok = (prop.gcnArchName[0] == 'g' && prop.gcnArchName[3] == '9' &&
                     prop.gcnArchName[4] == '5' && prop.gcnArchName[5] == '0');
        cached_dev = dev;
    }
    *di = cached;
    return cached.ok ? TOPK_OK : TOPK_EUNSUPPORTED;
}

uint32_t split_rows_for(int32_t max_rows, int cus) {
    const int64_t lim = 4ll * cus;
    return (uint32_t)((max_rows < lim) ? max_rows : lim);
}

// Work-item target of a split call: 1.5 items per compute unit, below the
// two workgroups per compute unit that can be resident (LDS bound), so that
// every item of a call starts at once.
int32_t plan_items(int cus) {
#ifdef TOPK_PHASE_TIMERS
    if (const char *e = getenv("TOPK_SEG_ITEMS")) return atoi(e);
#endif
    return (3 * cus) / 2;
}

// Most segments per row: a power of two in [1, kMaxSplit] with n_rows x pmax
// at most twice the item target (the grid; workgroups beyond a row's actual
// segment count exit at once), and at least 2 while the call has at most
// 2 x CUs rows; above that no row is split.
int32_t plan_pmax(int32_t n_rows, int cus) {
    const int64_t lim = 2ll * plan_items(cus);
    int32_t p = 1;
    while (p < kMaxSplit && (int64_t)(p * 2) * n_rows <= lim) p *= 2;
    // while the call's rows fit the resident workgroups at once, long rows
    // may still be halved (with more rows, halving cost the edge-case batch
    // more in its rows' exact recoveries than it saved elsewhere)
    if (p == 1 && (int64_t)n_rows <= 2ll * cus) p = 2;
    return p;
}

// Items beyond one per row that the order pre-pass may add (segments of the
// longest rows), and the resident workgroups whose mean work sets the
// segment length.
int32_t plan_extra(int cus) { return 2 * cus < kOrderExtra ? 2 * cus : kOrderExtra; }
int32_t plan_slots(int cus) { return 2 * cus; }

size_t ws_bytes(uint32_t split_rows) {
    return kHeaderBytes + kOrderBytes + (size_t)split_rows * (kRowBlockBytes + kViewHistBytes);
}

topk_ragged_policy default_policy() {
    topk_ragged_policy p;
    p.s_log2 = 7;
    p.rho_num = 3;
    p.rho_den = 2;
    p.rho1_num = 7;
    p.rho1_den = 4;
    p.l_samp_min = -4;
    p.cap = kCap;
    return p;
}

// The constants recalibrated for other K (Section 4.5: the coarse target, its
// sample rank and the candidate budget depend on K, the correctness argument
// does not), measured on synthetic decode rows.  Below K = 2048 the view
// stays at s = 128 and the margins widen as K shrinks, so that the sample
// ranks keep an underfilled proposal no likelier than in the evaluated
// configuration (sample ranks 8 and 10 at least); from K = 2560 the budget is
// tight, so s = 16 sharpens the estimate under margins of 5/4 and 11/8; from
// K = 4352 even those would overflow the frontier too often (C(tau0) above the
// capacity on about 1 row in 100), so every row takes the exact route.  Below
// K = 2048 rows shorter than 8192 take the exact route as well: there the
// candidates are a large share of a short row, span a wide key range, and
// the exact route measured faster.
topk_ragged_policy policy_for_k(int32_t K) {
    topk_ragged_policy p = default_policy();
    if (K < 2048) p.l_samp_min = 8192;
    if (K >= 4352) {
        p.l_samp_min = 0x7FFFFFFF;
    } else if (K >= 2560) {
        p.s_log2 = 4;
        p.rho_num = 5; p.rho_den = 4;
        p.rho1_num = 11; p.rho1_den = 8;
    } else if (K >= 2048) {
        // the evaluated configuration
    } else if (K >= 768) {
        p.rho_num = 2; p.rho_den = 1;
        p.rho1_num = 5; p.rho1_den = 2;
    } else if (K >= 384) {
        p.rho_num = 3; p.rho_den = 1;
        p.rho1_num = 4; p.rho1_den = 1;
    } else {
        // sample ranks 8 and 10 at s = 128
        p.rho_num = 8 << 7; p.rho_den = K;
        p.rho1_num = 10 << 7; p.rho1_den = K;
    }
    return p;
}

// Boundary-word polls before a segment builds the view itself; 0 = kSpinLimit
// (tests lower it to exercise that path).
int32_t g_spin_limit = 0;

int32_t sample_rank(int32_t K, int32_t num, int32_t den, int32_t s_log2) {
    const int64_t d = (int64_t)den << s_log2;
    return (int32_t)(((int64_t)num * K + d - 1) / d);
}

} // namespace

extern "C" {

int topk_ragged_default_policy(topk_ragged_policy *out) {
    if (!out) return TOPK_EINVAL;
    *out = default_policy();
    return TOPK_OK;
}

int topk_ragged_policy_for_k(int32_t K, topk_ragged_policy *out) {
    if (!out || K < 1 || K > TOPK_K_MAX) return TOPK_EINVAL;
    *out = policy_for_k(K);
    return TOPK_OK;
}

size_t topk_ragged_workspace_size(int32_t max_rows, int32_t K) {
    if (max_rows < 0 || K < 1 || K > TOPK_K_MAX) return 0;
    DeviceInfo di;
    if (device_info(&di) != TOPK_OK) return 0;
    return ws_bytes(split_rows_for(max_rows, di.cus));
}

int topk_ragged_workspace_init(void *workspace, size_t bytes, int32_t max_rows, int32_t K,
                               void *stream) {
    if (!workspace || max_rows < 0 || K < 1 || K > TOPK_K_MAX) return TOPK_EINVAL;
    if (reinterpret_cast<uintptr_t>(workspace) % kWorkspaceAlign) return TOPK_EINVAL;
    DeviceInfo di;
    const int st = device_info(&di);
    if (st != TOPK_OK) return st;
    const uint32_t sr = split_rows_for(max_rows, di.cus);
    if (bytes < ws_bytes(sr)) return TOPK_EWORKSPACE;
    WsHeader *hdr = static_cast<WsHeader *>(workspace);
    char *rows = static_cast<char *>(workspace) + kHeaderBytes + kOrderBytes;
    const int blocks = sr ? (int)(sr < 1024 ? sr : 1024) : 1;
    hipLaunchKernelGGL(ws_init_kernel, dim3(blocks), dim3(64), 0, (hipStream_t)stream, hdr, rows,
                       sr, (uint32_t)max_rows, (uint32_t)kCap);
    return hipGetLastError() == hipSuccess ? TOPK_OK : TOPK_ELAUNCH;
}

#ifdef TOPK_PHASE_TIMERS
static uint64_t *g_timers = nullptr;
// Debug builds only: device buffer of 8 x (grid size) words for the next calls
// (NULL disables).
extern "C" int topk_ragged_debug_set_timers(uint64_t *buf) {
    g_timers = buf;
    return TOPK_OK;
}
#endif

} // extern "C"

namespace {

// One call: the order pre-pass when the plan runs each row on one workgroup,
// then the main kernel.  split_cap: calls of more rows than this are not
// split (pmax = 1), so that they need no per-row state.
int launch_call(const float *scores, const int64_t *row_offsets, const int32_t *row_lengths,
                int32_t n_rows, int32_t K, int32_t *out_idx, float *out_val, void *workspace,
                const topk_ragged_policy *policy, int32_t *row_trace, void *stream,
                int32_t split_cap) {
    if (n_rows < 0 || K < 1 || K > TOPK_K_MAX) return TOPK_EINVAL;
    if (n_rows == 0) return TOPK_OK;
    if (!scores || !row_offsets || !row_lengths || !out_idx || !out_val || !workspace)
        return TOPK_EINVAL;
    if (reinterpret_cast<uintptr_t>(workspace) % kWorkspaceAlign) return TOPK_EINVAL;
    const topk_ragged_policy pol = policy ? *policy : policy_for_k(K);
    if (pol.s_log2 < 0 || pol.s_log2 > 12 || pol.rho_num < 1 || pol.rho_den < 1 ||
        pol.rho1_num < 1 || pol.rho1_den < 1 || pol.cap < 1 || pol.cap > kCap)
        return TOPK_EINVAL;
    DeviceInfo di;
    const int st = device_info(&di);
    if (st != TOPK_OK) return st;
    const int32_t pmax = n_rows > split_cap ? 1 : plan_pmax(n_rows, di.cus);
    if ((int64_t)n_rows * pmax > 0x7FFFFFFFll) return TOPK_EINVAL;
    KArgs a;
    a.scores = scores;
    a.offs = row_offsets;
    a.lens = row_lengths;
    a.out_idx = out_idx;
    a.out_val = out_val;
    a.trace = row_trace;
    a.hdr = static_cast<WsHeader *>(workspace);
    a.rows = static_cast<char *>(workspace) + kHeaderBytes + kOrderBytes;
    a.order = nullptr;
    a.n_rows = n_rows;
    a.K = K;
    a.pmax = pmax;
    a.seg_items = plan_items(di.cus);
    a.s_log2 = pol.s_log2;
    a.q0 = sample_rank(K, pol.rho_num, pol.rho_den, pol.s_log2);
    a.q1 = sample_rank(K, pol.rho1_num, pol.rho1_den, pol.s_log2);
    if (a.q1 < a.q0) a.q1 = a.q0;
    const int64_t floor_k = -(int64_t)pol.l_samp_min * K;
#ifdef TOPK_PHASE_TIMERS
    a.timers = g_timers;
#endif
    a.l_samp_min = pol.l_samp_min >= 0 ? pol.l_samp_min
                                       : (int32_t)(floor_k < 0x7FFFFFFF ? floor_k : 0x7FFFFFFF);
    a.cap = pol.cap;
    a.spin_limit = g_spin_limit > 0 ? g_spin_limit : kSpinLimit;
    a.spin_ticks = (uint32_t)((int64_t)kSpinMicros * di.clock_khz / 1000);
    int64_t grid = (int64_t)n_rows * pmax;
    if (pmax == 1 && n_rows <= kOrderMaxRows) {
        // more rows than resident workgroups: longest rows first, so that
        // the last to start is short, the longest of them in segments
        const int32_t extra = plan_extra(di.cus);
        uint4 *order = reinterpret_cast<uint4 *>(static_cast<char *>(workspace) + kHeaderBytes);
        if (n_rows <= kOrderBlock)
            hipLaunchKernelGGL(row_order_kernel<1>, dim3(1), dim3(kOrderBlock), 0,
                               (hipStream_t)stream, a, order, extra, plan_slots(di.cus));
        else
            hipLaunchKernelGGL(row_order_kernel<kOrderPer>, dim3(1), dim3(kOrderBlock), 0,
                               (hipStream_t)stream, a, order, extra, plan_slots(di.cus));
        if (hipGetLastError() != hipSuccess) return TOPK_ELAUNCH;
        a.order = order;
        grid += extra;
    }
    if (a.order)
        hipLaunchKernelGGL(topk_ragged_kernel<true>, dim3((unsigned)grid), dim3(kBlock), 0,
                           (hipStream_t)stream, a);
    else
        hipLaunchKernelGGL(topk_ragged_kernel<false>, dim3((unsigned)grid), dim3(kBlock), 0,
                           (hipStream_t)stream, a);
    return hipGetLastError() == hipSuccess ? TOPK_OK : TOPK_ELAUNCH;
}

} // namespace

extern "C" {

int topk_ragged_ex(const float *scores, const int64_t *row_offsets, const int32_t *row_lengths,
                   int32_t n_rows, int32_t K, int32_t *out_idx, float *out_val, void *workspace,
                   const topk_ragged_policy *policy, int32_t *row_trace, void *stream) {
    return launch_call(scores, row_offsets, row_lengths, n_rows, K, out_idx, out_val, workspace,
                       policy, row_trace, stream, INT32_MAX);
}

int topk_ragged(const float *scores, const int64_t *row_offsets, const int32_t *row_lengths,
                int32_t n_rows, int32_t K, int32_t *out_idx, float *out_val, void *workspace,
                void *stream) {
    return topk_ragged_ex(scores, row_offsets, row_lengths, n_rows, K, out_idx, out_val,
                          workspace, nullptr, nullptr, stream);
}

} // extern "C"

// ------------------------------------------- allocation-free variant ----
//
// The workspace of topk_ragged_noalloc: a file-scope device array (one copy
// per GPU, held until the process ends) laid out like a workspace for
// TOPK_NOALLOC_MAX_ROWS rows with per-row state for TOPK_NOALLOC_SPLIT_ROWS
// split rows.  Host code never passes the array's name to a kernel (on the
// host it is only a stand-in for the symbol): its device address is looked up
// once per device with hipGetSymbolAddress and kept in g_scratch_ptr.
constexpr size_t kScratchBytes = kHeaderBytes + kOrderBytes +
                                 (size_t)TOPK_NOALLOC_SPLIT_ROWS * (kRowBlockBytes + kViewHistBytes);
static_assert(TOPK_NOALLOC_MAX_ROWS <= kOrderMaxRows, "the order region covers every row");
static __device__ __align__(256) char scratch[kScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];

// The current device's scratch address; on the first call on a device the
// address is looked up and the header and per-row state are initialised by a
// kernel enqueued on `stream` (ahead of the call that follows on it).
int scratch_for_current_device(void **out, hipStream_t stream) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return TOPK_ELAUNCH;
    if (dev < 0 || dev >= kMaxDevices) return TOPK_EUNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr)
            return TOPK_ELAUNCH;
        WsHeader *hdr = static_cast<WsHeader *>(ptr);
        char *rows = static_cast<char *>(ptr) + kHeaderBytes + kOrderBytes;
        hipLaunchKernelGGL(ws_init_kernel, dim3(TOPK_NOALLOC_SPLIT_ROWS), dim3(64), 0, stream, hdr,
                           rows, (uint32_t)TOPK_NOALLOC_SPLIT_ROWS,
                           (uint32_t)TOPK_NOALLOC_MAX_ROWS, (uint32_t)kCap);
        if (hipGetLastError() != hipSuccess) return TOPK_ELAUNCH;
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return TOPK_OK;
}

} // namespace

extern "C" {

int topk_ragged_noalloc(const float *scores, const int64_t *row_offsets,
                        const int32_t *row_lengths, int32_t n_rows, int32_t K, int32_t *out_idx,
                        float *out_val, void *stream) {
    if (n_rows < 0 || K < 1 || K > TOPK_K_MAX) return TOPK_EINVAL;
    if (n_rows > TOPK_NOALLOC_MAX_ROWS) return TOPK_EWORKSPACE;
    if (n_rows == 0) return TOPK_OK;
    if (!scores || !row_offsets || !row_lengths || !out_idx || !out_val) return TOPK_EINVAL;
    DeviceInfo di;
    const int st = device_info(&di);
    if (st != TOPK_OK) return st;
    void *ws = nullptr;
    const int sst = scratch_for_current_device(&ws, (hipStream_t)stream);
    if (sst != TOPK_OK) return sst;
    return launch_call(scores, row_offsets, row_lengths, n_rows, K, out_idx, out_val, ws, nullptr,
                       nullptr, stream, TOPK_NOALLOC_SPLIT_ROWS);
}

int topk_ragged_read_stats(void *workspace, topk_ragged_stats *out, void *stream) {
    if (!workspace || !out) return TOPK_EINVAL;
    if (reinterpret_cast<uintptr_t>(workspace) % kWorkspaceAlign) return TOPK_EINVAL;
    WsHeader *hdr = static_cast<WsHeader *>(workspace);
    uint32_t st[16];
    hipStream_t s = (hipStream_t)stream;
    if (hipMemcpyAsync(st, hdr->stats, sizeof st, hipMemcpyDeviceToHost, s) != hipSuccess)
        return TOPK_ELAUNCH;
    if (hipStreamSynchronize(s) != hipSuccess) return TOPK_ELAUNCH;
    for (int i = 0; i < 6; i++) out->route[i] = st[i];
    out->reread = st[kStatReread];
    out->wait_fallback = st[kStatWaitFallback];
    out->errors = st[kStatErrors];
    hipLaunchKernelGGL(stats_reset_kernel, dim3(1), dim3(64), 0, s, hdr);
    return hipGetLastError() == hipSuccess ? TOPK_OK : TOPK_ELAUNCH;
}

int topk_ragged_debug_set_spin_limit(int32_t polls) {
    if (polls < 0) return TOPK_EINVAL;
    g_spin_limit = polls;
    return TOPK_OK;
}

int topk_ragged_debug_coarse(const float *x, int64_t n, uint16_t *out_c, void *stream) {
    if (n < 0 || (n > 0 && (!x || !out_c))) return TOPK_EINVAL;
    if (n == 0) return TOPK_OK;
    const int64_t blocks = (n + 255) / 256;
    if (blocks > 0x7FFFFFFFll) return TOPK_EINVAL;
    hipLaunchKernelGGL(debug_coarse_kernel, dim3((unsigned)blocks), dim3(256), 0,
                       (hipStream_t)stream, x, n, out_c);
    return hipGetLastError() == hipSuccess ? TOPK_OK : TOPK_ELAUNCH;
}

int topk_ragged_debug_read_ceiling(const float *scores, const int64_t *row_offsets,
                                   const int32_t *row_lengths, int32_t n_rows, int32_t K,
                                   uint32_t *out_max, void *workspace, void *stream) {
    if (n_rows < 0 || K < 1 || K > TOPK_K_MAX) return TOPK_EINVAL;
    if (n_rows == 0) return TOPK_OK;
    if (!scores || !row_offsets || !row_lengths || !out_max || !workspace) return TOPK_EINVAL;
    if (reinterpret_cast<uintptr_t>(workspace) % kWorkspaceAlign) return TOPK_EINVAL;
    DeviceInfo di;
    const int st = device_info(&di);
    if (st != TOPK_OK) return st;
    const int32_t pmax = plan_pmax(n_rows, di.cus);
    if ((int64_t)n_rows * pmax > 0x7FFFFFFFll) return TOPK_EINVAL;
    const topk_ragged_policy pol = policy_for_k(K);
    KArgs a = {};
    a.scores = scores;
    a.offs = row_offsets;
    a.lens = row_lengths;
    a.n_rows = n_rows;
    a.K = K;
    a.pmax = pmax;
    a.seg_items = plan_items(di.cus);
    a.s_log2 = pol.s_log2;
    a.q0 = sample_rank(K, pol.rho_num, pol.rho_den, pol.s_log2);
    a.q1 = sample_rank(K, pol.rho1_num, pol.rho1_den, pol.s_log2);
    if (a.q1 < a.q0) a.q1 = a.q0;
    const int64_t floor_k = -(int64_t)pol.l_samp_min * K;
    a.l_samp_min = pol.l_samp_min >= 0 ? pol.l_samp_min
                                       : (int32_t)(floor_k < 0x7FFFFFFF ? floor_k : 0x7FFFFFFF);
    a.hdr = static_cast<WsHeader *>(workspace);
    int64_t grid = (int64_t)n_rows * pmax;
    if (pmax == 1 && n_rows <= kOrderMaxRows) {
        // the selector's item table (its pre-pass is not part of the timing
        // it is compared with either)
        const int32_t extra = plan_extra(di.cus);
        uint4 *order = reinterpret_cast<uint4 *>(static_cast<char *>(workspace) + kHeaderBytes);
        if (n_rows <= kOrderBlock)
            hipLaunchKernelGGL(row_order_kernel<1>, dim3(1), dim3(kOrderBlock), 0,
                               (hipStream_t)stream, a, order, extra, plan_slots(di.cus));
        else
            hipLaunchKernelGGL(row_order_kernel<kOrderPer>, dim3(1), dim3(kOrderBlock), 0,
                               (hipStream_t)stream, a, order, extra, plan_slots(di.cus));
        if (hipGetLastError() != hipSuccess) return TOPK_ELAUNCH;
        a.order = order;
        grid += extra;
    }
    hipLaunchKernelGGL(read_ceiling_kernel, dim3((unsigned)grid), dim3(kBlock), 0,
                       (hipStream_t)stream, a, out_max);
    return hipGetLastError() == hipSuccess ? TOPK_OK : TOPK_ELAUNCH;
}

int topk_ragged_debug_cutoffs(uint32_t *out_cut, void *stream) {
    if (!out_cut) return TOPK_EINVAL;
    hipLaunchKernelGGL(debug_cutoff_kernel, dim3(kBins / 256), dim3(256), 0, (hipStream_t)stream,
                       out_cut);
    return hipGetLastError() == hipSuccess ? TOPK_OK : TOPK_ELAUNCH;
}

const char *topk_ragged_status_str(int status) {
    switch (status) {
    case TOPK_OK: return "ok";
    case TOPK_EINVAL: return "invalid argument";
    case TOPK_EUNSUPPORTED: return "unsupported device (gfx950 required)";
    case TOPK_ELAUNCH: return "HIP launch or runtime error";
    case TOPK_EWORKSPACE: return "workspace too small";
    default: return "unknown status";
    }
}

} // extern "C"
