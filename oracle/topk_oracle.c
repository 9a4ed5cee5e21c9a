/*
 * CPU oracle for exact Top-K selection over ragged FP32 score rows.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  The GPU library never
 * links, includes or calls anything here, and nothing here is shared with it.
 *
 * Two independent computations live in this file:
 *
 *   oracle_topk_ragged   the plain definition of the operator (Section 2.1,
 *                        "Operator contract"; exactness criterion of the
 *                        evaluation section, eq:eval:exactness): every row is
 *                        fully sorted on a unique composite key and the first
 *                        min(K, L) entries are kept.  Slow and obviously right.
 *
 *   oracle_route_model   the sample-guided pipeline of Section 4 written out in
 *                        the paper's order and notation: the row-phased view
 *                        (eq:method:view), the sample histogram and its prefix
 *                        (eq:method:sample-hist), the primary and nested
 *                        boundaries (eq:method:primary-threshold), the admitted
 *                        tail and its count (eq:method:candidate-set), the band
 *                        extension (eq:method:rescue-band), exact coarse
 *                        recovery (eq:method:exact-init) and the three-digit
 *                        radix refinement (eq:method:refine-prefix ..
 *                        eq:method:refine-recurrence).  It reports per row the
 *                        route taken and the integer quantities that decide it,
 *                        and also returns the selected indices, which must equal
 *                        the plain definition's.
 *
 * Readings where the paper is silent (fixed by the operator contract used here):
 *   - order is that of the order-preserving uint32 transform of the FP32 bits,
 *     so -0.0 sorts below +0.0 and subnormals are ordered numerically;
 *   - ties at rank K are broken toward the lowest index;
 *   - rows with L <= K return 0..L-1 in order, then -1 (value -inf);
 *   - a negative length is treated as 0;
 *   - the phase permutation pi_s is bit reversal of (r mod s) over log2(s) bits;
 *   - FP16 projection is IEEE round-to-nearest-even with overflow to infinity.
 *
 * Built with plain gcc (C11) and OpenMP over rows only.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* ---------------------------------------------------------------- keys --- */

static uint32_t bits_of(float x) {
    uint32_t b;
    memcpy(&b, &x, sizeof b);
    return b;
}

/* Order-preserving (ascending) uint32 key of an FP32 bit pattern: negative
 * patterns are complemented, non-negative ones get the sign bit set.  A larger
 * number gets a larger key; -0.0 gets 0x7FFFFFFF and +0.0 gets 0x80000000. */
uint32_t oracle_asc32(uint32_t b) {
    if (b & 0x80000000u)
        return ~b;
    return b | 0x80000000u;
}

/* Descending sortable key kappa32 (Section 4.3): larger value, smaller key. */
uint32_t oracle_desc32(uint32_t b) { return 0xFFFFFFFFu - oracle_asc32(b); }

/* IEEE binary16 round-to-nearest-even projection of an FP32 value, written from
 * the format's definition (Section 4.2 uses "round-to-nearest FP16").  NaN is
 * outside the operator's domain and is mapped to the canonical quiet NaN. */
uint16_t oracle_fp16_rn(float xf) {
    uint32_t b = bits_of(xf);
    uint16_t sign = (uint16_t)((b >> 16) & 0x8000u);
    double a = fabs((double)xf); /* exact: every float is a double */
    if (isnan(a))
        return (uint16_t)(sign | 0x7E00u);
    if (isinf(a))
        return (uint16_t)(sign | 0x7C00u);
    if (a == 0.0)
        return sign;
    /* binade exponent E with 2^E <= a < 2^(E+1); binary16 normals have
     * E in [-14, 15]; below that the quantum stays at 2^-24 (subnormals). */
    int e2;
    (void)frexp(a, &e2); /* a = f * 2^e2, f in [0.5, 1) */
    int E = e2 - 1;
    if (E < -14)
        E = -14;
    double quantum = ldexp(1.0, E - 10); /* spacing of binary16 in this binade */
    double n = nearbyint(a / quantum);   /* a/quantum is exact; ties to even */
    if (n >= 2048.0) {                   /* rounded up into the next binade */
        n = 1024.0;
        E += 1;
    }
    if (E > 15)
        return (uint16_t)(sign | 0x7C00u); /* overflow to infinity */
    if (n < 1024.0)                        /* only possible when E == -14 */
        return (uint16_t)(sign | (uint16_t)n);
    return (uint16_t)(sign | (uint16_t)((E + 15) << 10) | (uint16_t)(n - 1024.0));
}

/* Ascending 16-bit key of a binary16 pattern, same construction as asc32. */
static uint32_t asc16(uint16_t h) {
    if (h & 0x8000u)
        return (uint32_t)(~h) & 0xFFFFu;
    return (uint32_t)h | 0x8000u;
}

/* Coarse map c(x) = floor(kappa16(fp16_rn(x)) / 2^5) in [0, 2^11)
 * (eq:method:coarse-map); kappa16 is the descending 16-bit key. */
uint32_t oracle_coarse(float x) {
    uint32_t kappa16 = 0xFFFFu - asc16(oracle_fp16_rn(x));
    return kappa16 >> 5;
}

/* Smallest ascending FP32 key u (over non-NaN patterns) whose value has coarse
 * bin <= tau: the inclusive FP32 endpoint of bin tau (Section 4.3).  Found by
 * bisection on the monotone predicate c(value(u)) <= tau; returns 0xFFFFFFFF
 * when no non-NaN value qualifies. */
static float value_of_asc(uint32_t u) {
    uint32_t b = (u & 0x80000000u) ? (u & 0x7FFFFFFFu) : ~u;
    float x;
    memcpy(&x, &b, sizeof x);
    return x;
}

uint32_t oracle_cutoff(uint32_t tau) {
    const uint32_t lo_key = 0x007FFFFFu; /* asc32(-inf) */
    const uint32_t hi_key = 0xFF800000u; /* asc32(+inf) */
    if (oracle_coarse(value_of_asc(hi_key)) > tau)
        return 0xFFFFFFFFu;
    uint32_t lo = lo_key, hi = hi_key; /* invariant: c(hi) <= tau */
    if (oracle_coarse(value_of_asc(lo)) <= tau)
        return lo;
    while (hi - lo > 1) { /* invariant: c(lo) > tau */
        uint32_t mid = lo + (hi - lo) / 2;
        if (oracle_coarse(value_of_asc(mid)) <= tau)
            hi = mid;
        else
            lo = mid;
    }
    return hi;
}

/* Phase schedule a_r = pi_s(r mod s) (eq:method:view), with pi_s read as bit
 * reversal over log2(s) bits; s must be a power of two. */
int32_t oracle_phase(int32_t r, int32_t s) {
    int bitsn = 0;
    while ((1 << bitsn) < s)
        bitsn++;
    uint32_t v = (uint32_t)(r % s), out = 0;
    for (int i = 0; i < bitsn; i++)
        if (v & (1u << i))
            out |= 1u << (bitsn - 1 - i);
    return (int32_t)out;
}

/* ------------------------------------------------- plain definition ------ */

/* Composite key: descending value first, then ascending index.  Unique. */
static uint64_t composite(uint32_t bits, uint32_t idx) {
    return ((uint64_t)oracle_desc32(bits) << 32) | (uint64_t)idx;
}

static int cmp_u64(const void *a, const void *b) {
    uint64_t x = *(const uint64_t *)a, y = *(const uint64_t *)b;
    return (x > y) - (x < y);
}

static const float NEG_INF_VAL = -INFINITY;

static void write_direct(const float *x, int64_t L, int32_t K, int32_t *oi, float *ov) {
    for (int32_t j = 0; j < K; j++) {
        if (j < L) {
            oi[j] = j;
            ov[j] = x[j];
        } else {
            oi[j] = -1;
            ov[j] = NEG_INF_VAL;
        }
    }
}

/* Exact Top-K of every row (Section 2.1).  Row r is
 * scores[row_offsets[r] .. row_offsets[r] + row_lengths[r]).  Outputs are
 * [n_rows x K]; for L > K the K entries come in ascending composite-key order
 * (largest value first, lowest index first among equal values); for L <= K
 * they are 0..L-1 followed by -1 / -inf.  Returns 0, or -1 on bad arguments.
 * n_threads <= 0 uses the OpenMP default. */
int oracle_topk_ragged(const float *scores, const int64_t *row_offsets,
                       const int32_t *row_lengths, int32_t n_rows, int32_t K,
                       int32_t *out_idx, float *out_val, int n_threads) {
    if (n_rows < 0 || K < 1)
        return -1;
    if (n_rows == 0)
        return 0;
    if (!scores || !row_offsets || !row_lengths || !out_idx || !out_val)
        return -1;
#ifdef _OPENMP
    if (n_threads > 0)
        omp_set_num_threads(n_threads);
#else
    (void)n_threads;
#endif
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : bad)
    for (int32_t r = 0; r < n_rows; r++) {
        int64_t L = row_lengths[r] > 0 ? row_lengths[r] : 0;
        const float *x = scores + row_offsets[r];
        int32_t *oi = out_idx + (int64_t)r * K;
        float *ov = out_val + (int64_t)r * K;
        if (L <= K) {
            write_direct(x, L, K, oi, ov);
            continue;
        }
        uint64_t *z = (uint64_t *)malloc((size_t)L * sizeof(uint64_t));
        if (!z) {
            bad |= 1;
            continue;
        }
        for (int64_t i = 0; i < L; i++)
            z[i] = composite(bits_of(x[i]), (uint32_t)i);
        qsort(z, (size_t)L, sizeof(uint64_t), cmp_u64);
        for (int32_t j = 0; j < K; j++) {
            uint32_t i = (uint32_t)(z[j] & 0xFFFFFFFFu);
            oi[j] = (int32_t)i;
            ov[j] = x[i];
        }
        free(z);
    }
    return bad ? -2 : 0;
}

/* ------------------------------------------------------- route model ----- */

/* Policy of the sampled pipeline.  rho = rho_num / rho_den is the retention
 * margin (K~ = rho K), rho1 the nested secondary target (K~1 = rho1 K, raised
 * to K~ when below it); s is the view stride; rows with L < l_samp_min or a
 * view smaller than q1 take the exact route; cap is the frontier capacity: a
 * candidate set larger than cap
 * is not materialised (sampled rows then take exact coarse recovery; an exact
 * boundary bin larger than cap is resolved by re-reading the row). */
typedef struct {
    int32_t s;
    int32_t rho_num, rho_den;
    int32_t rho1_num, rho1_den;
    int32_t l_samp_min;
    int32_t cap;
} oracle_policy;

enum {
    ROUTE_DIRECT = 0,
    ROUTE_PRIMARY = 1,
    ROUTE_BAND = 2,
    ROUTE_EXACT_UNSAMPLED = 3,
    ROUTE_EXACT_UNDERFILL = 4,
    ROUTE_EXACT_OVERFLOW = 5,
    ROUTE_REREAD_FLAG = 16
};

enum { TRACE_WORDS = 8 };

static int64_t ceil_div64(int64_t a, int64_t b) { return (a + b - 1) / b; }

/* Sample rank q = ceil(K~ / s) for K~ = (num/den) K, in integers. */
int32_t oracle_sample_rank(int32_t K, int32_t num, int32_t den, int32_t s) {
    return (int32_t)ceil_div64((int64_t)num * K, (int64_t)den * s);
}

/* First bin b with inclusive prefix H(b) >= q; 2048 when none does. */
static int32_t first_reaching(const int64_t *h, int32_t nbins, int64_t q) {
    int64_t H = 0;
    for (int32_t b = 0; b < nbins; b++) {
        H += h[b];
        if (H >= q)
            return b;
    }
    return nbins;
}

static int cmp_u32(const void *a, const void *b) {
    uint32_t x = *(const uint32_t *)a, y = *(const uint32_t *)b;
    return (x > y) - (x < y);
}

/* Radix refinement over an initial state (E0, Q0, k0) following
 * eq:method:refine-prefix .. eq:method:refine-recurrence with D = 3 digits of
 * widths 11, 11, 10 of kappa32, then the final equal-key fill from Q_D
 * (lowest indices first).  Appends the selected indices to sel[*nsel..]. */
static void refine(const float *x, uint32_t *Q, int64_t nQ, int64_t k,
                   int32_t *sel, int64_t *nsel) {
    static const int width[3] = {11, 11, 10};
    static const int shift[3] = {21, 10, 0};
    int64_t *h = (int64_t *)calloc(2048, sizeof(int64_t));
    for (int j = 0; j < 3 && k > 0; j++) {
        uint32_t mask = (1u << width[j]) - 1u;
        memset(h, 0, 2048 * sizeof(int64_t));
        for (int64_t t = 0; t < nQ; t++)
            h[(oracle_desc32(bits_of(x[Q[t]])) >> shift[j]) & mask]++;
        int32_t bj = first_reaching(h, 1 << width[j], k);
        int64_t nnext = 0, committed = 0;
        for (int64_t t = 0; t < nQ; t++) {
            uint32_t d = (oracle_desc32(bits_of(x[Q[t]])) >> shift[j]) & mask;
            if ((int32_t)d < bj) {
                sel[(*nsel)++] = (int32_t)Q[t];
                committed++;
            } else if ((int32_t)d == bj) {
                Q[nnext++] = Q[t];
            }
        }
        nQ = nnext;
        k -= committed;
    }
    /* Q_D holds equal FP32 keys; take the k lowest indices. */
    qsort(Q, (size_t)nQ, sizeof(uint32_t), cmp_u32);
    for (int64_t t = 0; t < k; t++)
        sel[(*nsel)++] = (int32_t)Q[t];
    free(h);
}

/* Route model of the sampled pipeline for every row.  row_ids (may be NULL)
 * gives the row number that selects each row's view phase, so a subset of a
 * larger call can be modelled; NULL means row r uses phase a_r of r.
 * Writes the selection to
 * out_idx / out_val (any order within a row for L > K; direct layout for
 * L <= K) and, when trace != NULL, 8 int32 per row:
 *   [0] route (ROUTE_*; ROUTE_REREAD_FLAG or-ed in when an exact boundary bin
 *       exceeds cap), [1] view size |V| (-1 for L <= K), [2] tau0, [3] tau1
 *   (-1 when not sampled), [4] C(tau0), [5] C(tau1) (-1 when not evaluated),
 *   [6] tau_star (-1 unless exact recovery ran), [7] |Q0| entering refinement
 *   (-1 for L <= K). */
int oracle_route_model(const float *scores, const int64_t *row_offsets,
                       const int32_t *row_lengths, const int32_t *row_ids, int32_t n_rows,
                       int32_t K, const oracle_policy *pol, int32_t *out_idx, float *out_val,
                       int32_t *trace, int n_threads) {
    if (n_rows < 0 || K < 1 || !pol || pol->s < 1 || (pol->s & (pol->s - 1)))
        return -1;
    if (n_rows == 0)
        return 0;
#ifdef _OPENMP
    if (n_threads > 0)
        omp_set_num_threads(n_threads);
#else
    (void)n_threads;
#endif
    const int32_t s = pol->s;
    const int32_t q0 = oracle_sample_rank(K, pol->rho_num, pol->rho_den, s);
    /* The nested target is never below the primary one (Section 4.3: tau1 is
     * the looser, nested boundary, K~1 >= K~).  A policy that sets it lower
     * gets K~1 = K~, so a sampled row's view holds both ranks and tau1 = tau0. */
    int32_t q1 = oracle_sample_rank(K, pol->rho1_num, pol->rho1_den, s);
    if (q1 < q0)
        q1 = q0;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : bad)
    for (int32_t r = 0; r < n_rows; r++) {
        int64_t L = row_lengths[r] > 0 ? row_lengths[r] : 0;
        const float *x = scores + row_offsets[r];
        int32_t *oi = out_idx + (int64_t)r * K;
        float *ov = out_val + (int64_t)r * K;
        int32_t tr[TRACE_WORDS] = {ROUTE_DIRECT, -1, -1, -1, -1, -1, -1, -1};
        if (L <= K) {
            write_direct(x, L, K, oi, ov);
            if (trace)
                memcpy(trace + (int64_t)r * TRACE_WORDS, tr, sizeof tr);
            continue;
        }
        int64_t *h = (int64_t *)calloc(2048, sizeof(int64_t));
        uint32_t *c = (uint32_t *)malloc((size_t)L * sizeof(uint32_t));
        uint32_t *Q = (uint32_t *)malloc((size_t)L * sizeof(uint32_t));
        int32_t *sel = (int32_t *)malloc((size_t)K * sizeof(int32_t));
        if (!h || !c || !Q || !sel) {
            bad |= 1;
            free(h), free(c), free(Q), free(sel);
            continue;
        }
        for (int64_t i = 0; i < L; i++)
            c[i] = oracle_coarse(x[i]);

        /* Phase 1: row-phased view and its coarse histogram. */
        int32_t a = oracle_phase(row_ids ? row_ids[r] : r, s);
        int64_t nv = (a < L) ? ceil_div64(L - a, s) : 0;
        tr[1] = (int32_t)nv;
        int route;
        int64_t nQ = 0, k0 = K, nsel = 0;
        if (L >= pol->l_samp_min && nv >= q1) {
            for (int64_t i = a; i < L; i += s)
                h[c[i]]++;
            int32_t tau0 = first_reaching(h, 2048, q0);
            int32_t tau1 = first_reaching(h, 2048, q1);
            tr[2] = tau0;
            tr[3] = tau1;
            /* Phase 2: complete-row count of the admitted tail A(tau0). */
            int64_t C0 = 0;
            for (int64_t i = 0; i < L; i++)
                C0 += (c[i] <= (uint32_t)tau0);
            tr[4] = (int32_t)C0;
            int32_t tau = -1;
            if (C0 >= K) {
                route = (C0 <= pol->cap) ? ROUTE_PRIMARY : ROUTE_EXACT_OVERFLOW;
                tau = tau0;
            } else {
                /* Band extension: A(tau1) = A(tau0) + {tau0 < c <= tau1}. */
                int64_t C1 = C0;
                for (int64_t i = 0; i < L; i++)
                    C1 += (c[i] > (uint32_t)tau0 && c[i] <= (uint32_t)tau1);
                tr[5] = (int32_t)C1;
                if (C1 >= K) {
                    route = (C1 <= pol->cap) ? ROUTE_BAND : ROUTE_EXACT_OVERFLOW;
                    tau = tau1;
                } else {
                    route = ROUTE_EXACT_UNDERFILL;
                }
            }
            if (route == ROUTE_PRIMARY || route == ROUTE_BAND) {
                /* Sampled initialisation: E0 empty, Q0 = A(tau), k0 = K. */
                for (int64_t i = 0; i < L; i++)
                    if (c[i] <= (uint32_t)tau)
                        Q[nQ++] = (uint32_t)i;
            }
        } else {
            route = ROUTE_EXACT_UNSAMPLED;
        }
        if (route != ROUTE_PRIMARY && route != ROUTE_BAND) {
            /* Exact coarse recovery over all L values. */
            memset(h, 0, 2048 * sizeof(int64_t));
            for (int64_t i = 0; i < L; i++)
                h[c[i]]++;
            int32_t tstar = first_reaching(h, 2048, K);
            tr[6] = tstar;
            for (int64_t i = 0; i < L; i++) {
                if (c[i] < (uint32_t)tstar)
                    sel[nsel++] = (int32_t)i; /* E0: committed */
                else if (c[i] == (uint32_t)tstar)
                    Q[nQ++] = (uint32_t)i; /* Q0: boundary bin */
            }
            k0 = K - nsel;
            if (nQ > pol->cap)
                route |= ROUTE_REREAD_FLAG;
        }
        tr[0] = route;
        tr[7] = (int32_t)nQ;
        refine(x, Q, nQ, k0, sel, &nsel);
        for (int32_t j = 0; j < K; j++) {
            oi[j] = sel[j];
            ov[j] = x[sel[j]];
        }
        if (nsel != K)
            bad |= 2;
        if (trace)
            memcpy(trace + (int64_t)r * TRACE_WORDS, tr, sizeof tr);
        free(h), free(c), free(Q), free(sel);
    }
    return bad ? -2 : 0;
}

/* Vector helpers for tests: apply the scalar maps to arrays. */
void oracle_coarse_many(const float *x, int64_t n, uint32_t *out) {
    for (int64_t i = 0; i < n; i++)
        out[i] = oracle_coarse(x[i]);
}

void oracle_fp16_many(const float *x, int64_t n, uint16_t *out) {
    for (int64_t i = 0; i < n; i++)
        out[i] = oracle_fp16_rn(x[i]);
}

void oracle_asc32_many(const uint32_t *b, int64_t n, uint32_t *out) {
    for (int64_t i = 0; i < n; i++)
        out[i] = oracle_asc32(b[i]);
}

void oracle_cutoff_all(uint32_t *out2048) {
    for (uint32_t t = 0; t < 2048; t++)
        out2048[t] = oracle_cutoff(t);
}
