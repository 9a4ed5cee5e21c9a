// Exact Top-K over ragged FP32 rows for gfx950 (wave64): kernels and C-ABI.
//
// One kernel launch per call.  Work item = (row r, segment p); blockIdx.x =
// p * n_rows + r, so every row's first segment is dispatched before any
// second segment.  Each item is one 512-thread workgroup.
//
//   L <= K            segment 0 writes the direct layout (Section 2.1).
//   not sampled       segment 0 runs exact coarse recovery alone
//                     (eq:method:exact-init): coarse histogram pass, classify
//                     pass, refinement.
//   sampled, 1 seg    Phase 1 (view histogram, eq:method:sample-hist and
//                     eq:method:primary-threshold) -> Phase 2 (complete-row
//                     certify + compact, eq:method:candidate-set) -> band or
//                     exact recovery when underfilled -> Phase 3 refinement.
//   sampled, P segs   segment 0 runs Phase 1 and publishes the endpoints;
//                     every segment certifies and compacts its contiguous
//                     part of the row (eq:method:split-local); the last
//                     segment to arrive merges the candidate ranges
//                     (eq:method:split-reduce) and finishes the row.
//
// Keys: asc = order-preserving uint32 of the FP32 bits; the descending key
// kappa32 = ~asc (Section 4.3) is what the frontier stores and what the
// radix digits are taken from.  Ties at rank K are resolved by three more
// radix digits over the row index, so the result is the K smallest composite
// keys (kappa32, index): the lowest index wins among equal values.

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <climits>
#include <type_traits>

#include "../../include/topk_ragged.h"

namespace {

constexpr int kBlock = 512;                 // threads per workgroup (8 waves)
constexpr int kBins = 2048;                 // 11-bit digits and coarse bins
constexpr int kWaves = kBlock / 64;
constexpr int kCap = TOPK_FRONTIER_CAP;     // largest policy frontier (pairs)
constexpr int kFront = 7168;                // LDS frontier storage (pairs)
constexpr int kWaveCap = kFront / kWaves - 1; // Phase 2 storage per wave (+1 spill slot)
constexpr int kWaveStride = kFront / kWaves;
static_assert(kCap <= kFront, "policy capacity must fit the storage");
constexpr int kVec = 8;                     // 16-byte loads per thread per chunk
static_assert(kVec * 4 <= 64, "per-thread element masks are 64-bit");
static_assert(kFront % kBlock == 0 && kFront % kWaves == 0, "frontier layout");
constexpr int kChunkVecs = kBlock * kVec;   // 16-byte vectors per chunk
constexpr int kMaxSplit = 64;               // most segments per row
constexpr int kSegMin = 8192;               // shortest segment, elements
constexpr uint32_t kMagic = 0x544F504Bu;    // workspace header tag
constexpr int kSpinLimit = 1 << 15;         // polls before recomputing the view
constexpr size_t kHeaderBytes = 1024;
constexpr size_t kRowStateBytes = 256;
constexpr size_t kRowBlockBytes = kRowStateBytes + 2 * kFront * sizeof(uint32_t);

typedef float f4 __attribute__((ext_vector_type(4)));

// Per-row state of a split row.  Row r of a split call owns the workspace
// block at kHeaderBytes + r * kRowBlockBytes: this state, padded to 256
// bytes, then kFront candidate indices and kFront candidate FP32 bit patterns
// (the segments' A(tau1) entries, concatenated).
struct RowState {
    uint32_t flag;       // 1 once cut0/cut1/taus are published by segment 0
    uint32_t cut0;       // ascending-key endpoint of tau0
    uint32_t cut1;       // ascending-key endpoint of tau1
    uint32_t taus;       // tau0 | tau1 << 16
    uint32_t arrive;     // segments done with Phase 2
    uint32_t count1;     // C(tau1) of the row (exact)
    uint32_t count0;     // C(tau0) of the row (exact)
    uint32_t stored;     // entries reserved in the candidate buffer
    uint32_t incomplete; // a segment could not keep all of its A(tau1)
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
    int32_t n_rows;
    int32_t K;
    int32_t pmax;
    int32_t s_log2;
    int32_t q0, q1;
    int32_t l_samp_min;
    int32_t cap;
#ifdef TOPK_PHASE_TIMERS
    uint64_t *timers; // 16 words per workgroup, see PHASE_MARK
#endif
};

// Optional phase timers (built only with -DTOPK_PHASE_TIMERS): thread 0 of
// each workgroup stamps the constant-rate clock at fixed points of the row
// pipeline: 0 start, 1 endpoints known, 2 Phase 2 done, 3 arrived, 4 finisher
// has the merged frontier, 5 row done; word 6 = hardware id, 7 = role;
// 8 finish entered, 9 frontier ready, 10..12 after refinement rounds 0..2,
// 13 refinement done, 14 live entries entering refinement, 15 rounds run.
#ifdef TOPK_PHASE_TIMERS
#define PHASE_MARK(a, k)                                                                 \
    do {                                                                                 \
        if ((a).timers && threadIdx.x == 0)                                              \
            (a).timers[(size_t)blockIdx.x * 16 + (k)] = wall_clock64();                   \
    } while (0)
#define PHASE_WORD(a, k, v)                                                              \
    do {                                                                                 \
        if ((a).timers && threadIdx.x == 0) (a).timers[(size_t)blockIdx.x * 16 + (k)] = (v); \
    } while (0)
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

// Wave64 OR / AND of a value; the result is valid in lane 63.
__device__ __forceinline__ uint32_t wave_or_to63(uint32_t v) {
    v |= __builtin_amdgcn_update_dpp(0u, v, 0x111, 0xf, 0xf, false);
    v |= __builtin_amdgcn_update_dpp(0u, v, 0x112, 0xf, 0xf, false);
    v |= __builtin_amdgcn_update_dpp(0u, v, 0x114, 0xf, 0xf, false);
    v |= __builtin_amdgcn_update_dpp(0u, v, 0x118, 0xf, 0xf, false);
    v |= __builtin_amdgcn_update_dpp(0u, v, 0x142, 0xa, 0xf, false);
    v |= __builtin_amdgcn_update_dpp(0u, v, 0x143, 0xc, 0xf, false);
    return v;
}

__device__ __forceinline__ uint32_t wave_and_to63(uint32_t v) {
    v &= __builtin_amdgcn_update_dpp(~0u, v, 0x111, 0xf, 0xf, false);
    v &= __builtin_amdgcn_update_dpp(~0u, v, 0x112, 0xf, 0xf, false);
    v &= __builtin_amdgcn_update_dpp(~0u, v, 0x114, 0xf, 0xf, false);
    v &= __builtin_amdgcn_update_dpp(~0u, v, 0x118, 0xf, 0xf, false);
    v &= __builtin_amdgcn_update_dpp(~0u, v, 0x142, 0xa, 0xf, false);
    v &= __builtin_amdgcn_update_dpp(~0u, v, 0x143, 0xc, 0xf, false);
    return v;
}

// Wave-aggregated append: every lane of the wave must call it.  Returns the
// slot of this lane's item (meaningful only where pred is true).
__device__ __forceinline__ uint32_t wave_append(bool pred, uint32_t *ctr) {
    const uint64_t m = __ballot(pred);
    if (m == 0) return 0;
    const uint32_t pre = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                                   __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
    uint32_t base = 0;
    if (lane_id() == 0) base = atomicAdd(ctr, (uint32_t)__popcll(m));
    return __builtin_amdgcn_readfirstlane(base) + pre;
}

// Wave-aggregated append for a ballot mask already computed by the caller:
// one LDS atomic per wave.  Every lane of the wave must call it.
__device__ __forceinline__ uint32_t wave_append_bits(uint64_t m, uint32_t *ctr) {
    const uint32_t pre = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                                   __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
    uint32_t base = 0;
    if (lane_id() == 0) base = atomicAdd(ctr, (uint32_t)__popcll(m));
    return __builtin_amdgcn_readfirstlane(base) + pre;
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

// ------------------------------------------------- shared state ----

struct alignas(16) Smem {
    uint32_t hist[kBins];
    uint32_t hist2[kBins]; // refinement alternates between hist and hist2
    uint32_t ci[kFront]; // frontier indices (row-relative)
    uint32_t ck[kFront]; // frontier keys: FP32 bits after Phase 2, kappa32 after compaction
    uint32_t wcnt[kWaves]; // Phase 2 hits per wave (exact, may exceed kWaveCap)
    uint32_t red[2][4];    // refinement: OR (lo, hi) and AND (lo, hi) of live keys
    Find find[2];
    uint32_t cnt;       // C(tau1), or the append counter of the current pass
    uint32_t cnt0;      // C(tau0)
    uint32_t incomplete;
    uint32_t opos;      // outputs written for the current row
    uint32_t next;      // compaction counter in refinement
    uint32_t cut0, cut1, tau0, tau1;
    uint32_t flag;
    uint32_t base;
};

__device__ __forceinline__ void clear_hist(Smem &sm) {
    uint4 *h4 = reinterpret_cast<uint4 *>(sm.hist);
    for (int i = threadIdx.x; i < kBins / 4; i += kBlock) h4[i] = make_uint4(0, 0, 0, 0);
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

// Double-buffered chunks: while one chunk (kVec 16-byte loads per thread) is
// consumed, the next one is in flight.  Loads are unconditional -- lanes and
// chunks past the end re-read the last vector of the range (one cache line per
// wave), masked by the window test -- so the in-order load counter lets each
// consume wait for its own chunk only.  prologue() runs once, by every thread:
// before the first issue when it loads from memory itself (its loads would
// otherwise queue behind the chunk), else with the first chunk in flight.
template <bool kNT, class F, class Pro = NoPrologue>
__device__ __forceinline__ void stream_row(const float *scores, int64_t off, int32_t beg,
                                           int32_t end, F &&fn, Pro &&prologue = Pro(),
                                           bool prologue_first = false) {
    if (beg >= end) {
        prologue();
        return;
    }
    const uintptr_t sp = reinterpret_cast<uintptr_t>(scores);
    const int64_t sh = (int64_t)((sp & 15) >> 2);
    const int64_t v0 = (off + beg + sh) >> 2;
    const int32_t nvec = (int32_t)(((off + end + sh + 3) >> 2) - v0);
    const char *vbase = reinterpret_cast<const char *>(sp & ~(uintptr_t)15) + v0 * 16;
    const int32_t ibase = (int32_t)(v0 * 4 - sh - off); // row index of vbase's first element
    const int32_t nch = (nvec + kChunkVecs - 1) / kChunkVecs;
    const int tid = threadIdx.x;
    f4 xa[kVec], xb[kVec];
    auto issue = [&](f4 *dst, int32_t c) {
        const int32_t cb = c * kChunkVecs;
#pragma unroll
        for (int m = 0; m < kVec; m++) {
            const int32_t vi = min(cb + m * kBlock + tid, nvec - 1);
            dst[m] = load4<kNT>(reinterpret_cast<const f4 *>(vbase + (uint32_t)vi * 16u));
        }
    };
    auto consume = [&](const f4 *src, int32_t c) {
        if (c >= nch) return;
        const int32_t cb = c * kChunkVecs;
        // vectors of this chunk per thread (block-uniform)
        const int32_t mv = min(kVec, (nvec - cb + kBlock - 1) / kBlock);
        int32_t i0[kVec];
#pragma unroll
        for (int m = 0; m < kVec; m++) i0[m] = ibase + (cb + m * kBlock + tid) * 4;
        // interior chunks need no per-element window test
        const bool edge = ibase + cb * 4 < beg || ibase + (cb + mv * kBlock) * 4 > end;
        fn(src, i0, beg, end, edge, mv);
    };
    if (prologue_first) prologue();
    issue(xa, 0);
    if (!prologue_first) prologue();
    for (int32_t c = 0; c < nch; c += 2) {
        issue(xb, c + 1);
        consume(xa, c);
        issue(xa, c + 2);
        consume(xb, c + 1);
    }
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
// bits) in the private region of its wave: sm.ci/ck[w * kWaveCap ..), in
// element order within the wave.  Each element costs one compare; a
// wave-wide ballot places the hits with no atomics.  C(tau1) and C(tau0) are
// counted exactly even where a wave region overflows (sm.incomplete is then
// set).  The endpoints are read from sm after prologue() has run.
template <class Pro>
__device__ __forceinline__ void phase2_collect(Smem &sm, const float *scores, int64_t off,
                                               int32_t beg, int32_t end, bool prologue_first,
                                               Pro &&prologue) {
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
#pragma unroll
                for (int m = 0; m < kVec; m++) if (m < mv) {
#pragma unroll
                    for (int c = 0; c < 4; c++) {
                        const uint32_t b = fbits(x[m][c]);
                        const bool h1 = kPos ? (int32_t)b >= t1 : asc_key(b) >= cut1;
                        bool hit = h1;
                        if constexpr (kEdge) hit = h1 && in_window(i0[m] + c, lo, hi);
                        const uint64_t m1 = __ballot(hit);
                        if (m1) {
                            // slot kWaveCap of the region absorbs hits past its
                            // capacity (the count stays exact)
                            const uint32_t q = min(cur + __builtin_amdgcn_mbcnt_hi(
                                                             (uint32_t)(m1 >> 32),
                                                             __builtin_amdgcn_mbcnt_lo((uint32_t)m1, 0u)),
                                                   (uint32_t)kWaveCap);
                            if (hit) { wi[q] = (uint32_t)(i0[m] + c); wk[q] = b; }
                            cur += (uint32_t)__popcll(m1);
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
        prologue, prologue_first);
    if ((threadIdx.x & 63) == 0) {
        sm.wcnt[w] = cur;
        atomicAdd(&sm.cnt, cur);
        if (cur > (uint32_t)kWaveCap) sm.incomplete = 1u;
    }
}

// C(tau0) from the stored entries of Phase 2 (all of A(tau1) when complete).
// Ends with a barrier.
__device__ __forceinline__ uint32_t count_tail(Smem &sm, bool segmented, uint32_t n,
                                               uint32_t kmin) {
    uint32_t c = 0;
    for (uint32_t t = threadIdx.x; t < (uint32_t)kFront; t += kBlock) {
        bool v;
        if (segmented) {
            const uint32_t w = t / kWaveStride;
            v = (t - w * kWaveStride) < min(sm.wcnt[w], (uint32_t)kWaveCap);
        } else {
            v = t < n;
        }
        c += (v && asc_key(sm.ck[t]) >= kmin) ? 1u : 0u;
    }
    c = wave_incl_scan(c);
    if ((threadIdx.x & 63) == 63 && c) atomicAdd(&sm.cnt0, c);
    __syncthreads();
    return sm.cnt0;
}

// C(tau0) of row elements [beg, end) by re-reading them (overflow fallback).
// sm.cnt0 must be zero on entry.  Ends with a barrier.
__device__ __forceinline__ uint32_t count_range(Smem &sm, const float *scores, int64_t off,
                                                int32_t beg, int32_t end, uint32_t kmin) {
    uint32_t c = 0;
    stream_row<false>(scores, off, beg, end, [&](const f4 *x, const int32_t *i0, int32_t lo,
                                                 int32_t hi, bool, int32_t mv) {
#pragma unroll
        for (int m = 0; m < kVec; m++) if (m < mv) {
#pragma unroll
            for (int cc = 0; cc < 4; cc++)
                c += (in_window(i0[m] + cc, lo, hi) && asc_key(fbits(x[m][cc])) >= kmin) ? 1u : 0u;
        }
    });
    c = wave_incl_scan(c);
    if ((threadIdx.x & 63) == 63 && c) atomicAdd(&sm.cnt0, c);
    __syncthreads();
    return sm.cnt0;
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
// written) is read once into registers, kPer entries per thread, from either
// the per-wave regions of Phase 2 (`segmented`) or [0, n) of sm.ci/ck, as
// FP32 bits filtered by ascending key >= kmin (`raw`) or as kappa32 keys.
// The entries are ordered by the composite key z = (kappa32 << 32) | index
// (ties broken toward the lowest index).  Each round histograms an 11-bit
// digit of z over the live entries, finds b = min{b : H(b) >= k}
// (eq:method:digit-boundary), commits the groups before b
// (eq:method:committed-group), keeps group b (eq:method:refine-recurrence)
// and stops once the kept group exactly fills the quota.  The paper's digits
// are fixed 11/11/10-bit fields of kappa32; here each round takes the 11 bits
// just below the highest bit position at which the live keys still differ
// (all live keys agree above it), which selects the same set in fewer rounds
// and spreads the histogram over more bins.  Entries never move: each thread
// keeps a live mask.  Entry and exit with all threads converged and sm.hist
// cleared.
constexpr int kPer = kFront / kBlock;

__device__ __forceinline__ uint64_t zkey(uint32_t kappa, uint32_t idx) {
    return ((uint64_t)kappa << 32) | idx;
}

// Block-wide OR and AND of the live composite keys into sm.red[par][0..3]
// (written by one lane per wave; the caller's next barrier publishes them).
__device__ __forceinline__ void reduce_live(Smem &sm, int par, const uint32_t *ri,
                                            const uint32_t *rk, uint32_t live) {
    uint32_t olo = 0, ohi = 0, alo = ~0u, ahi = ~0u;
#pragma unroll
    for (int j = 0; j < kPer; j++) {
        if (live & (1u << j)) {
            olo |= ri[j]; ohi |= rk[j];
            alo &= ri[j]; ahi &= rk[j];
        }
    }
    olo = wave_or_to63(olo);
    ohi = wave_or_to63(ohi);
    alo = wave_and_to63(alo);
    ahi = wave_and_to63(ahi);
    if (lane_id() == 63) {
        atomicOr(&sm.red[par][0], olo);
        atomicOr(&sm.red[par][1], ohi);
        atomicAnd(&sm.red[par][2], alo);
        atomicAnd(&sm.red[par][3], ahi);
    }
}

// Lowest bit of the 11-bit digit window: just below the highest differing bit.
__device__ __forceinline__ uint32_t window_shift(const Smem &sm, int par) {
    const uint64_t o = ((uint64_t)sm.red[par][1] << 32) | sm.red[par][0];
    const uint64_t n = ((uint64_t)sm.red[par][3] << 32) | sm.red[par][2];
    const uint64_t diff = o ^ n;
    const int h = diff ? 63 - __clzll((long long)diff) : 0;
    return h >= 10 ? (uint32_t)(h - 10) : 0u;
}

__device__ __forceinline__ void reset_red(Smem &sm, int par) {
    if (threadIdx.x < 4) sm.red[par][threadIdx.x] = threadIdx.x < 2 ? 0u : ~0u;
}

__device__ __forceinline__ void refine(const KArgs a, Smem &sm, int r, bool segmented, uint32_t n,
                                       bool raw, uint32_t kmin, uint32_t n_live, uint32_t k,
                                       int64_t L) {
    (void)L;
    const int tid = threadIdx.x;
    uint32_t ri[kPer], rk[kPer];
    uint32_t live = 0;
#pragma unroll
    for (int j = 0; j < kPer; j++) {
        const uint32_t t = (uint32_t)(j * kBlock + tid);
        bool v;
        if (segmented) {
            const uint32_t w = t / kWaveStride;
            v = (t - w * kWaveStride) < min(sm.wcnt[w], (uint32_t)kWaveCap);
        } else {
            v = t < n;
        }
        ri[j] = v ? sm.ci[t] : 0u;
        const uint32_t word = v ? sm.ck[t] : 0u;
        if (raw) {
            rk[j] = ~asc_key(word);
            v = v && asc_key(word) >= kmin;
        } else {
            rk[j] = word;
        }
        live |= (v ? 1u : 0u) << j;
    }
    PHASE_WORD(a, 14, n_live);
    int rounds_run = 0;
    uint32_t done = 0; // committed entries (written out after the last round)
    if (k > 0 && n_live > k) {
        // sm.red[0] and sm.red[1] were reset by the caller before its barrier
        reduce_live(sm, 0, ri, rk, live);
        __syncthreads();
    }
    // Round t histograms into H[t & 1], finds into sm.find[t & 1] and
    // reduces its survivors into sm.red[(t + 1) & 1]; each buffer of the
    // other parity is reset while this round histograms (its last readers
    // are behind this round's first barrier... of the previous round).
    while (k > 0 && n_live > k) {
        const int par = rounds_run & 1;
        const uint32_t shift = window_shift(sm, par);
        uint32_t *H = par ? sm.hist2 : sm.hist;
        uint32_t *Hn = par ? sm.hist : sm.hist2;
        {
            uint4 *h4 = reinterpret_cast<uint4 *>(Hn);
            for (int i = tid; i < kBins / 4; i += kBlock) h4[i] = make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int j = 0; j < kPer; j++)
            if (live & (1u << j))
                atomicAdd(&H[(uint32_t)(zkey(rk[j], ri[j]) >> shift) & 0x7FFu], 1u);
        __syncthreads();
        if (tid < 64) wave_find(H, k, 0, 1, &sm.find[par]);
        reset_red(sm, par ^ 1);
        __syncthreads();
        const Find f = sm.find[par];
        const uint32_t need = k - f.below;                   // > 0 and <= f.eq
        const bool take_all = (f.eq == need);
        uint32_t keep = 0;
#pragma unroll
        for (int j = 0; j < kPer; j++) {
            const bool lv = (live >> j) & 1u;
            const uint32_t d = (uint32_t)(zkey(rk[j], ri[j]) >> shift) & 0x7FFu;
            done |= ((lv && (d < f.bin || (take_all && d == f.bin))) ? 1u : 0u) << j;
            keep |= ((lv && !take_all && d == f.bin) ? 1u : 0u) << j;
        }
        live = keep;
        n_live = take_all ? 0u : f.eq;
        k = take_all ? 0u : need;
        if (rounds_run < 3) PHASE_MARK(a, 10 + rounds_run);
        rounds_run++;
        if (k > 0 && n_live > k) {
            reduce_live(sm, par ^ 1, ri, rk, live);
            __syncthreads();
        }
    }
    // both histogram buffers back to zero for the next user of sm.hist
    __syncthreads();
    clear_hist(sm);
    {
        uint4 *h4 = reinterpret_cast<uint4 *>(sm.hist2);
        for (int i = tid; i < kBins / 4; i += kBlock) h4[i] = make_uint4(0, 0, 0, 0);
    }
    PHASE_WORD(a, 15, (uint64_t)rounds_run);
    if (k > 0) done |= live; // every live entry is in: n_live == k
    // Output: one LDS atomic per wave places this thread's committed entries
    // (no global store inside the rounds, so no barrier waits on one).
    const uint32_t mine = (uint32_t)__popc(done);
    const uint32_t incl = wave_incl_scan(mine);
    const uint32_t total = __builtin_amdgcn_readlane(incl, 63);
    uint32_t base = 0;
    if (total) {
        if (lane_id() == 63) base = atomicAdd(&sm.opos, total);
        base = __builtin_amdgcn_readlane(base, 63);
    }
    uint32_t op = base + incl - mine;
#pragma unroll
    for (int j = 0; j < kPer; j++)
        if (done & (1u << j)) emit(a, r, op++, ri[j], rk[j]);
    __syncthreads();
}

// ------------------------------------------------------ exact routes ----

__device__ __forceinline__ uint64_t composite(uint32_t key, uint32_t idx) {
    return ((uint64_t)key << 32) | idx;
}

// Resolves an exact boundary bin that exceeds the frontier capacity without
// materialising it: each round re-reads the row and histograms the next digit
// of the composite key (kappa32, index) among boundary-bin elements that
// match the digits fixed so far, until the k-th smallest key T is known; a
// last pass commits every boundary-bin element with key <= T.
__device__ __forceinline__ void reread_select(const KArgs a, Smem &sm, int r, int64_t off, int64_t L,
                              uint32_t tstar, uint32_t k) {
    const int tid = threadIdx.x;
    const float *scores = a.scores;
    uint64_t prefix = 0; // chosen digits so far, left-aligned in the 64-bit key
    int shift_done = 64; // bits of the composite key fixed = 64 - shift_done
    uint64_t T = ~0ull; // select composite <= T
    for (int j = 0; j < 6; j++) {
        const int w = (j % 3 == 2) ? 10 : 11;
        const int shift = shift_done - w;
        clear_hist(sm);
        __syncthreads();
        const uint64_t hi_mask = (shift_done >= 64) ? 0ull : (~0ull << shift_done);
        stream_row<false>(scores, off, 0, (int32_t)L, [&](const f4 *x, const int32_t *i0, int32_t lo,
                                                 int32_t hi, bool, int32_t mv) {
#pragma unroll
            for (int m = 0; m < kVec; m++) if (m < mv) {
#pragma unroll
                for (int c = 0; c < 4; c++) {
                    const int32_t i = i0[m] + c;
                    if (!in_window(i, lo, hi)) continue;
                    if (coarse_bin(x[m][c]) != tstar) continue;
                    const uint64_t z = composite(~asc_key(fbits(x[m][c])),
                                                 (uint32_t)i);
                    if ((z & hi_mask) != prefix) continue;
                    atomicAdd(&sm.hist[(uint32_t)(z >> shift) & ((1u << w) - 1u)], 1u);
                }
            }
        });
        __syncthreads();
        if (tid < 64) wave_find(sm.hist, k, 0, 1, sm.find);
        __syncthreads();
        const Find f = sm.find[0];
        prefix |= (uint64_t)f.bin << shift;
        shift_done = shift;
        const uint32_t need = k - f.below;
        __syncthreads();
        if (f.eq == need || j == 5) {
            T = prefix | ((shift == 0) ? 0ull : ((1ull << shift) - 1ull));
            break;
        }
        k = need;
    }
    // Output pass: every boundary-bin element with composite key <= T.
    stream_row<false>(scores, off, 0, (int32_t)L, [&](const f4 *x, const int32_t *i0, int32_t lo,
                                             int32_t hi, bool, int32_t mv) {
#pragma unroll
        for (int m = 0; m < kVec; m++) if (m < mv) {
#pragma unroll
            for (int c = 0; c < 4; c++) {
                const int32_t i = i0[m] + c;
                if (!in_window(i, lo, hi)) continue;
                if (coarse_bin(x[m][c]) != tstar) continue;
                const uint32_t key = ~asc_key(fbits(x[m][c]));
                if (composite(key, (uint32_t)i) > T) continue;
                const uint32_t op = atomicAdd(&sm.opos, 1u);
                emit(a, r, op, (uint32_t)i, key);
            }
        }
    });
    __syncthreads();
}

// Exact coarse recovery (eq:method:exact-init) over the whole row by this
// workgroup: a coarse histogram pass finds tau_star = min{b : C(b) >= K}; a
// classify pass commits c < tau_star to the output (E0) and keeps
// c == tau_star as the frontier Q0 when it fits the capacity.  Returns
// (tau_star, |E0|, |Q0|) in sm.find[0]; ends with a barrier, sm.hist cleared.
__device__ __forceinline__ void exact_classify(const KArgs a, Smem &sm, int r, int64_t off, int64_t L) {
    const int tid = threadIdx.x;
    const float *scores = a.scores;
    stream_row<false>(scores, off, 0, (int32_t)L, [&](const f4 *x, const int32_t *i0, int32_t lo,
                                                      int32_t hi, bool, int32_t mv) {
#pragma unroll
        for (int m = 0; m < kVec; m++) if (m < mv) {
#pragma unroll
            for (int c = 0; c < 4; c++)
                if (in_window(i0[m] + c, lo, hi)) atomicAdd(&sm.hist[coarse_bin(x[m][c])], 1u);
        }
    });
    __syncthreads();
    if (tid < 64) wave_find(sm.hist, (uint32_t)a.K, 0, 1, sm.find);
    if (tid == 0) sm.cnt = 0;
    __syncthreads();
    const uint32_t tstar = sm.find[0].bin;
    const bool fits = sm.find[0].eq <= (uint32_t)a.cap;
    stream_row<false>(scores, off, 0, (int32_t)L, [&](const f4 *x, const int32_t *i0, int32_t lo,
                                                      int32_t hi, bool, int32_t mv) {
#pragma unroll
        for (int m = 0; m < kVec; m++) if (m < mv) {
#pragma unroll
            for (int c = 0; c < 4; c++) {
                const int32_t i = i0[m] + c;
                if (!in_window(i, lo, hi)) continue;
                const uint32_t cb = coarse_bin(x[m][c]);
                if (cb > tstar) continue;
                const uint32_t key = ~asc_key(fbits(x[m][c]));
                if (cb < tstar) {
                    const uint32_t op = atomicAdd(&sm.opos, 1u);
                    emit(a, r, op, (uint32_t)i, key);
                } else if (fits) {
                    const uint32_t q = atomicAdd(&sm.cnt, 1u);
                    sm.ci[q] = (uint32_t)i;
                    sm.ck[q] = key;
                }
            }
        }
    });
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

// Sample histogram over the view and the two boundaries (eq:method:sample-hist,
// eq:method:primary-threshold); leaves tau0/tau1 and their endpoints in sm.
// Ends with a barrier; the histogram is cleared again on exit.
__device__ __forceinline__ void phase1(const KArgs a, Smem &sm, int r, const float *row, int64_t L) {
    const int tid = threadIdx.x;
    const uint32_t ph = view_phase(r, a.s_log2);
    const int64_t nv = view_size(L, ph, a.s_log2);
    clear_hist(sm);
    __syncthreads();
    const float *base = row + ph;
    int64_t t = tid;
    for (; t + 3 * kBlock < nv; t += 4 * kBlock) {
        const float x0 = base[(t) << a.s_log2];
        const float x1 = base[(t + kBlock) << a.s_log2];
        const float x2 = base[(t + 2 * kBlock) << a.s_log2];
        const float x3 = base[(t + 3 * kBlock) << a.s_log2];
        atomicAdd(&sm.hist[coarse_bin(x0)], 1u);
        atomicAdd(&sm.hist[coarse_bin(x1)], 1u);
        atomicAdd(&sm.hist[coarse_bin(x2)], 1u);
        atomicAdd(&sm.hist[coarse_bin(x3)], 1u);
    }
    for (; t < nv; t += kBlock) atomicAdd(&sm.hist[coarse_bin(base[t << a.s_log2])], 1u);
    __syncthreads();
    if (tid < 64) {
        wave_find(sm.hist, (uint32_t)a.q0, (uint32_t)a.q1, 2, sm.find);
        if (tid == 0) {
            sm.tau0 = sm.find[0].bin;
            sm.tau1 = sm.find[1].bin;
            sm.cut0 = bin_cutoff(sm.tau0);
            sm.cut1 = bin_cutoff(sm.tau1);
        }
    }
    __syncthreads();
    clear_hist(sm);
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
                                           bool incomplete, bool segmented, uint32_t nstored) {
    const uint32_t K = (uint32_t)a.K;
    const uint32_t cap = (uint32_t)a.cap;
    int32_t trC1 = -1, tstar = -1, nq = -1;
    uint32_t route, n_ref = 0, k_ref = K, kmin = 0;
    clear_hist(sm);
    if (threadIdx.x == 0) sm.opos = 0;
    __syncthreads();
    PHASE_MARK(a, 8);
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
    // Frontier of the certified tail: A(tau0), or A(tau1) for the band, read
    // from the Phase 2 entries (FP32 bits filtered by kmin) or, when those
    // are incomplete, re-collected from the row as kappa32 keys.
    bool f_seg = segmented, f_raw = true;
    uint32_t f_n = nstored;
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
    if (route >= TOPK_ROUTE_EXACT_UNSAMPLED) {
        exact_classify(a, sm, r, off, L);
        const Find f = sm.find[0];
        tstar = (int32_t)f.bin;
        nq = (int32_t)f.eq;
        k_ref = K - f.below;
        if (f.eq <= cap) {
            n_ref = f.eq;
            f_seg = false;
            f_raw = false;
            f_n = f.eq;
        } else {
            route |= TOPK_ROUTE_REREAD_FLAG;
            reread_select(a, sm, r, off, L, f.bin, k_ref);
        }
    }
    PHASE_MARK(a, 9);
    if (n_ref) {
        reset_red(sm, 0);
        reset_red(sm, 1);
        __syncthreads();
        refine(a, sm, r, f_seg, f_n, f_raw, kmin, n_ref, k_ref, L);
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

// ----------------------------------------------------------- kernel ----

__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(4))) void
topk_ragged_kernel(KArgs a) {
    __shared__ Smem sm;
    const int tid = threadIdx.x;
    const int item = blockIdx.x;
    const int p = item / a.n_rows;
    const int r = item - p * a.n_rows;

    const int64_t L = (int64_t)max(a.lens[r], 0);
    const int64_t off = a.offs[r];
    const float *row = a.scores + off;
    PHASE_MARK(a, 0);
    PHASE_WORD(a, 6, (uint64_t)__smid());

    // Workspace check: a split plan needs per-row state for every row.
    const WsHeader *hdr = a.hdr;
    if (hdr->magic != kMagic || (uint32_t)a.n_rows > hdr->max_rows ||
        (a.pmax > 1 && (uint32_t)a.n_rows > hdr->split_rows)) {
        if (p == 0) {
            write_error_row(a, r);
            if (tid == 0 && r == 0) atomicAdd(&a.hdr->stats[kStatErrors], 1u);
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
    const bool sampled = L >= a.l_samp_min && nv >= a.q1;

    // Segments of a sampled row: P0 = min(pmax, ceil(L / kSegMin)) pieces of
    // equal length rounded up to 64 elements.  Unsampled rows run whole on
    // segment 0.
    int64_t P = 1, seg = L;
    if (sampled) {
        const int64_t P0 = min((int64_t)a.pmax, (L + kSegMin - 1) / kSegMin);
        seg = (((L + P0 - 1) / P0) + 63) & ~(int64_t)63;
        P = (L + seg - 1) / seg;
    }
    if (p >= P) return;
    const bool split = P > 1;
    RowState *rs = reinterpret_cast<RowState *>(a.rows + (size_t)r * kRowBlockBytes);
    uint32_t *gi = reinterpret_cast<uint32_t *>(a.rows + (size_t)r * kRowBlockBytes +
                                                kRowStateBytes);
    uint32_t *gk = gi + kFront;
    uint32_t C0 = 0, C1 = 0, nstored = 0;
    bool incomplete = false, segmented = true;

    if (sampled) {
        // Phase 1 runs while the first chunk of this segment is loading:
        // segment 0 (or the only segment) builds the view; other segments
        // wait for its published endpoints and rebuild the same view
        // themselves if it does not arrive within the spin limit.
        if (tid == 0) { sm.cnt = 0; sm.cnt0 = 0; sm.incomplete = 0; }
        const int32_t beg = (int32_t)(p * seg);
        const int32_t end = (int32_t)min(L, p * seg + seg);
        auto endpoints = [&]() {
            bool own_view = !split || p == 0;
            if (!own_view) {
                if (tid == 0) {
                    // Relaxed polls (an acquire per poll would invalidate this
                    // XCD's L2 every time); one acquire once the flag is set.
                    uint32_t f = 0;
                    for (int spin = 0; spin < kSpinLimit; spin++) {
                        f = __hip_atomic_load(&rs->flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        if (f) break;
                        __builtin_amdgcn_s_sleep(2);
                    }
                    sm.flag = f;
                    if (f) {
                        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
                        sm.cut0 = __hip_atomic_load(&rs->cut0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        sm.cut1 = __hip_atomic_load(&rs->cut1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        const uint32_t taus =
                            __hip_atomic_load(&rs->taus, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        sm.tau0 = taus & 0xFFFFu;
                        sm.tau1 = taus >> 16;
                    } else {
                        atomicAdd(&a.hdr->stats[kStatWaitFallback], 1u);
                    }
                }
                __syncthreads();
                own_view = sm.flag == 0;
            }
            if (own_view) phase1(a, sm, r, row, L);
            if (split && p == 0 && tid == 0) {
                __hip_atomic_store(&rs->cut0, sm.cut0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(&rs->cut1, sm.cut1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(&rs->taus, sm.tau0 | (sm.tau1 << 16), __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(&rs->flag, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
            }
            PHASE_MARK(a, 1);
        };
        // Phase 2 over this segment: certify against cut0 and keep A(tau1).
        phase2_collect(sm, a.scores, off, beg, end, /*prologue_first=*/!split || p == 0,
                       endpoints);
        __syncthreads();
        C1 = sm.cnt;
        incomplete = sm.incomplete != 0;
        // C(tau0): from the stored A(tau1) entries, or by re-reading this
        // segment when a wave region overflowed.
        C0 = incomplete ? count_range(sm, a.scores, off, beg, end, sm.cut0)
                        : count_tail(sm, true, 0, sm.cut0);
        PHASE_MARK(a, 2);
        PHASE_WORD(a, 7, (uint64_t)p | ((uint64_t)P << 16) | ((uint64_t)r << 32));

        if (split) {
            // Publish this segment's entries and counts (eq:method:split-local),
            // then arrive; the last arrival merges them (eq:method:split-reduce)
            // and finishes the row.
            uint32_t pre[kWaves + 1];
            pre[0] = 0;
#pragma unroll
            for (int w = 0; w < kWaves; w++) pre[w + 1] = pre[w] + min(sm.wcnt[w], (uint32_t)kWaveCap);
            if (tid == 0) {
                sm.base = pre[kWaves] ? __hip_atomic_fetch_add(&rs->stored, pre[kWaves],
                                                               __ATOMIC_RELAXED,
                                                               __HIP_MEMORY_SCOPE_AGENT)
                                      : 0u;
                if (C1) __hip_atomic_fetch_add(&rs->count1, C1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                if (C0) __hip_atomic_fetch_add(&rs->count0, C0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                if (incomplete)
                    __hip_atomic_store(&rs->incomplete, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            __syncthreads();
            const uint32_t base = sm.base;
            for (uint32_t t = tid; t < (uint32_t)kFront; t += kBlock) {
                const uint32_t w = t / kWaveStride, j = t - w * kWaveStride;
                if (j < pre[w + 1] - pre[w]) {
                    const uint32_t d = base + pre[w] + j;
                    if (d < (uint32_t)kFront) { gi[d] = sm.ci[t]; gk[d] = sm.ck[t]; }
                }
            }
            // Every wave waits for its own stores to reach L2; after the
            // barrier one thread writes the L2 back for the other XCDs
            // (agent-scope release) and arrives.
            __builtin_amdgcn_s_waitcnt(0);
            __syncthreads();
            if (tid == 0) {
                __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
                const uint32_t old = __hip_atomic_fetch_add(&rs->arrive, 1u, __ATOMIC_RELAXED,
                                                            __HIP_MEMORY_SCOPE_AGENT);
                const bool last = old == (uint32_t)(P - 1);
                if (last) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
                sm.flag = last ? 2u : 0u;
            }
            __syncthreads();
            PHASE_MARK(a, 3);
            if (sm.flag != 2u) return;

            // Finisher.  Segment 0 published the endpoints before arriving.
            if (tid == 0) {
                sm.cnt = __hip_atomic_load(&rs->count1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                sm.cnt0 = __hip_atomic_load(&rs->count0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                sm.base = __hip_atomic_load(&rs->stored, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                sm.incomplete = __hip_atomic_load(&rs->incomplete, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                sm.cut0 = __hip_atomic_load(&rs->cut0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                sm.cut1 = __hip_atomic_load(&rs->cut1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                const uint32_t taus =
                    __hip_atomic_load(&rs->taus, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                sm.tau0 = taus & 0xFFFFu;
                sm.tau1 = taus >> 16;
            }
            __syncthreads();
            C1 = sm.cnt;
            C0 = sm.cnt0;
            const uint32_t stored = sm.base;
            incomplete = sm.incomplete != 0 || stored > (uint32_t)kFront;
            nstored = min(stored, (uint32_t)kFront);
            segmented = false;
            for (uint32_t t = tid; t < nstored; t += kBlock) {
                sm.ci[t] = gi[t];
                sm.ck[t] = gk[t];
            }
            __syncthreads();
            PHASE_MARK(a, 4);
        }
    }

    finish_row(a, sm, r, off, L, nv, sampled, C0, C1, incomplete, segmented, nstored);
    PHASE_MARK(a, 5);

    if (split && tid == 0) {
        // Leave the row state zeroed for the next call (graph replays).
        __hip_atomic_store(&rs->count1, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&rs->count0, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&rs->stored, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&rs->incomplete, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&rs->arrive, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&rs->flag, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// Workspace set-up: header and zeroed per-row state (the candidate arrays
// need no initialisation: only entries below the published count are read).
__global__ void ws_init_kernel(WsHeader *hdr, char *rows, uint32_t split_rows, uint32_t max_rows,
                               uint32_t cap) {
    for (uint32_t r = blockIdx.x; r < split_rows; r += gridDim.x) {
        uint32_t *w = reinterpret_cast<uint32_t *>(rows + (size_t)r * kRowBlockBytes);
        if (threadIdx.x < kRowStateBytes / 4) w[threadIdx.x] = 0;
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

struct DeviceInfo {
    int cus = 0;
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

// Segments per row: enough work items for about 8 workgroups per compute
// unit, as a power of two in [1, kMaxSplit]; rows are split only when the
// call has at most 4 x CUs rows.
int32_t plan_pmax(int32_t n_rows, int cus) {
    const int64_t target = 8ll * cus;
    int32_t p = 1;
    while (p < kMaxSplit && (int64_t)(p * 2) * n_rows <= target) p *= 2;
    return p;
}

size_t ws_bytes(uint32_t split_rows) {
    return kHeaderBytes + (size_t)split_rows * kRowBlockBytes;
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

size_t topk_ragged_workspace_size(int32_t max_rows, int32_t K) {
    if (max_rows < 0 || K < 1 || K > TOPK_K_MAX) return 0;
    DeviceInfo di;
    if (device_info(&di) != TOPK_OK) return 0;
    return ws_bytes(split_rows_for(max_rows, di.cus));
}

int topk_ragged_workspace_init(void *workspace, size_t bytes, int32_t max_rows, int32_t K,
                               void *stream) {
    if (!workspace || max_rows < 0 || K < 1 || K > TOPK_K_MAX) return TOPK_EINVAL;
    DeviceInfo di;
    const int st = device_info(&di);
    if (st != TOPK_OK) return st;
    const uint32_t sr = split_rows_for(max_rows, di.cus);
    if (bytes < ws_bytes(sr)) return TOPK_EWORKSPACE;
    WsHeader *hdr = static_cast<WsHeader *>(workspace);
    char *rows = static_cast<char *>(workspace) + kHeaderBytes;
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

int topk_ragged_ex(const float *scores, const int64_t *row_offsets, const int32_t *row_lengths,
                   int32_t n_rows, int32_t K, int32_t *out_idx, float *out_val, void *workspace,
                   const topk_ragged_policy *policy, int32_t *row_trace, void *stream) {
    if (n_rows < 0 || K < 1 || K > TOPK_K_MAX) return TOPK_EINVAL;
    if (n_rows == 0) return TOPK_OK;
    if (!scores || !row_offsets || !row_lengths || !out_idx || !out_val || !workspace)
        return TOPK_EINVAL;
    const topk_ragged_policy pol = policy ? *policy : default_policy();
    if (pol.s_log2 < 0 || pol.s_log2 > 12 || pol.rho_num < 1 || pol.rho_den < 1 ||
        pol.rho1_num < 1 || pol.rho1_den < 1 || pol.cap < 1 || pol.cap > kCap)
        return TOPK_EINVAL;
    DeviceInfo di;
    const int st = device_info(&di);
    if (st != TOPK_OK) return st;
    const int32_t pmax = plan_pmax(n_rows, di.cus);
    if ((int64_t)n_rows * pmax > 0x7FFFFFFFll) return TOPK_EINVAL;
    KArgs a;
    a.scores = scores;
    a.offs = row_offsets;
    a.lens = row_lengths;
    a.out_idx = out_idx;
    a.out_val = out_val;
    a.trace = row_trace;
    a.hdr = static_cast<WsHeader *>(workspace);
    a.rows = static_cast<char *>(workspace) + kHeaderBytes;
    a.n_rows = n_rows;
    a.K = K;
    a.pmax = pmax;
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
    hipLaunchKernelGGL(topk_ragged_kernel, dim3((unsigned)(n_rows * pmax)), dim3(kBlock), 0,
                       (hipStream_t)stream, a);
    return hipGetLastError() == hipSuccess ? TOPK_OK : TOPK_ELAUNCH;
}

int topk_ragged(const float *scores, const int64_t *row_offsets, const int32_t *row_lengths,
                int32_t n_rows, int32_t K, int32_t *out_idx, float *out_val, void *workspace,
                void *stream) {
    return topk_ragged_ex(scores, row_offsets, row_lengths, n_rows, K, out_idx, out_val,
                          workspace, nullptr, nullptr, stream);
}

int topk_ragged_read_stats(void *workspace, topk_ragged_stats *out, void *stream) {
    if (!workspace || !out) return TOPK_EINVAL;
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

int topk_ragged_debug_coarse(const float *x, int64_t n, uint16_t *out_c, void *stream) {
    if (n < 0 || (n > 0 && (!x || !out_c))) return TOPK_EINVAL;
    if (n == 0) return TOPK_OK;
    const int64_t blocks = (n + 255) / 256;
    if (blocks > 0x7FFFFFFFll) return TOPK_EINVAL;
    hipLaunchKernelGGL(debug_coarse_kernel, dim3((unsigned)blocks), dim3(256), 0,
                       (hipStream_t)stream, x, n, out_c);
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
