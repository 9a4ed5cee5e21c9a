/*
 * topk_ragged -- exact Top-K over ragged FP32 score rows on AMD MI355X (gfx950).
 *
 * Implements the sample-guided exact selection of "Sample-Guided Exact Top-K
 * Selection for Long-Context Sparse Attention" (arXiv 2609.08450):
 *   Phase 1  a fixed-stride, row-phased view proposes a coarse boundary
 *            (Section 4.2, eq:method:view .. eq:method:primary-threshold);
 *   Phase 2  one complete-row pass certifies it and compacts the admitted
 *            candidates (Section 4.3, eq:method:candidate-set, Lemma
 *            lem:method:containment), with a nested secondary boundary and
 *            exact coarse recovery for underfilled proposals
 *            (eq:method:rescue-band, eq:method:exact-init);
 *   Phase 3  exact radix refinement over the surviving frontier
 *            (Section 4.4, eq:method:refine-prefix .. refine-recurrence),
 * behind a ragged-row dispatcher: rows with L <= K are written directly,
 * short rows run on one workgroup, long rows are split across several
 * workgroups whose admitted candidates are merged by the last one to finish
 * (Section 4.5, eq:method:split-local, eq:method:split-reduce); a call with
 * more rows than resident workgroups runs its rows longest first and splits
 * only the longest, and a split row whose candidates overflow takes the exact
 * coarse recovery across its segments.
 *
 * Semantics (Section 2.1 operator contract, with the choices the paper leaves
 * open fixed as follows):
 *   - order is that of the order-preserving uint32 transform of the FP32 bits:
 *     -inf < ... < -0.0 < +0.0 < ... < +inf, subnormals ordered; no NaN input;
 *   - ties at rank K go to the lowest index;
 *   - row r with L_r = max(0, row_lengths[r]) <= K returns indices 0..L_r-1 in
 *     order, then -1 with value -inf;
 *   - for L_r > K the K returned (index, value) pairs are in no particular
 *     order.
 *
 * All entry points are host functions returning a status code synchronously.
 * Device pointers are caller-owned; the library never allocates, never
 * synchronises (except topk_ragged_read_stats) and enqueues only on `stream`,
 * so topk_ragged can be captured in a HIP graph.  `stream` is a hipStream_t
 * passed as void* (NULL = the default stream).
 */
#ifndef TOPK_RAGGED_H
#define TOPK_RAGGED_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
#define TOPK_OK 0
#define TOPK_EINVAL (-1)       /* bad scalar argument or null pointer */
#define TOPK_EUNSUPPORTED (-2) /* current device is not gfx950 */
#define TOPK_ELAUNCH (-3)      /* a HIP call failed (see hipGetLastError) */
#define TOPK_EWORKSPACE (-4)   /* workspace too small for the plan */

/* Largest supported K.  Results are exact for every K up to this value; the
 * sampled pipeline needs its candidates (about K~ = 1.5 K at K = 2048) to fit
 * the on-chip frontier of TOPK_FRONTIER_CAP entries, so the per-K policy
 * (topk_ragged_policy_for_k) sends every row of a larger K to the exact
 * route. */
#define TOPK_K_MAX 16384
/* Longest row, in elements: the kernels address a row's 16-byte vectors with
 * 32-bit byte offsets from the 128-byte line that holds its first element. */
#define TOPK_L_MAX 0x3FFFFFDF
/* Frontier capacity of one workgroup, in (index, key) pairs. */
#define TOPK_FRONTIER_CAP 6144
/* Words per row written by topk_ragged_ex when row_trace is not NULL. */
#define TOPK_TRACE_WORDS 8

/* Route codes (trace word 0, and the stats counters). */
#define TOPK_ROUTE_DIRECT 0          /* L <= K */
#define TOPK_ROUTE_PRIMARY 1         /* C(tau0) >= K, certified proposal */
#define TOPK_ROUTE_BAND 2            /* C(tau0) < K <= C(tau1), band extension */
#define TOPK_ROUTE_EXACT_UNSAMPLED 3 /* view unusable or row below sampling floor */
#define TOPK_ROUTE_EXACT_UNDERFILL 4 /* C(tau1) < K: exact coarse recovery */
#define TOPK_ROUTE_EXACT_OVERFLOW 5  /* admitted tail larger than the frontier */
#define TOPK_ROUTE_REREAD_FLAG 16    /* or-ed in: exact boundary bin larger than
                                        the frontier, resolved by re-reading */

/* Policy of the sampled pipeline (Section 4.2 constants).  The defaults are
 * s = 128, K~ = 1.5 K, K~1 = 1.75 K (the configuration the paper evaluates),
 * sampling floor 4 K elements, frontier capacity TOPK_FRONTIER_CAP. */
typedef struct topk_ragged_policy {
    int32_t s_log2;     /* view stride s = 2^s_log2, 0 <= s_log2 <= 12 */
    int32_t rho_num;    /* K~  = ceil(rho_num  K / rho_den)  (as sample rank) */
    int32_t rho_den;
    int32_t rho1_num;   /* K~1 = ceil(rho1_num K / rho1_den) (nested target;
                           raised to K~ when below it) */
    int32_t rho1_den;
    int32_t l_samp_min; /* rows shorter than this take the exact route; a
                           negative value -m means m * K */
    int32_t cap;        /* frontier capacity, 1 <= cap <= TOPK_FRONTIER_CAP */
} topk_ragged_policy;

/* Route counters accumulated in the workspace (one increment per row), and
 * error/diagnostic counts.  The routes are the outcomes of certification
 * (Section 4.3: primary proposal, band of eq:method:rescue-band, exact coarse
 * recovery of eq:method:exact-init); their fractions over the rows of a call
 * are the primary-underfill and residual exact-recovery rates that the
 * paper's ablations report (Section 6.4, "Retention margin" and "Conditional
 * rescue"). */
typedef struct topk_ragged_stats {
    uint64_t route[6];     /* indexed by TOPK_ROUTE_* (flag stripped) */
    uint64_t reread;       /* rows that took the re-read fallback */
    uint64_t wait_fallback;/* split segments that stopped waiting: for the
                              boundaries (they recompute the view locally),
                              or for tau_star of the split exact route (the
                              last segment then runs the row's exact route) */
    uint64_t errors;       /* rejected on the device: one per call with a bad
                              workspace, one per row longer than TOPK_L_MAX */
} topk_ragged_stats;

/* Fills *out with the evaluated configuration above (the policy for K
 * around 2048).  Returns TOPK_OK. */
int topk_ragged_default_policy(topk_ragged_policy *out);

/* Fills *out with the policy used for this K when none is given.  Section 4.5
 * leaves the coarse target, its sample rank and the candidate budget to be
 * recalibrated per K; measured on synthetic decode rows:
 *   K < 384:           sample ranks 8 and 10 (K~ = 1024, K~1 = 1280);
 *   384 <= K < 768:    K~ = 3 K,   K~1 = 4 K;
 *   768 <= K < 2048:   K~ = 2 K,   K~1 = 5/2 K;
 *   2048 <= K < 2560:  the evaluated configuration;
 *   2560 <= K < 4352:  s = 16, K~ = 5/4 K, K~1 = 11/8 K;
 *   4352 <= K:         every row takes the exact route (l_samp_min = INT32_MAX);
 * s = 128 unless stated; the sampling floor is 4 K from K = 2048 and 8192
 * elements below (shorter rows measured faster on the exact route).  Returns TOPK_OK, or
 * TOPK_EINVAL for a null pointer or K outside [1, TOPK_K_MAX]. */
int topk_ragged_policy_for_k(int32_t K, topk_ragged_policy *out);

/* Bytes of workspace needed for calls with n_rows <= max_rows and this K on
 * the current device.  The serving path needs a workspace bounded
 * independently of the batch's contents (Section 2.1, "Deployment
 * requirements"), and the plan that sizes it is fixed before capture from the
 * row capacity and the device (Section 5.5, "Shape-stable dispatch"): the
 * size depends only on (max_rows, K, device), never on row lengths.  Per-row
 * state (about 72 KB) is kept only for rows split across workgroups, and at
 * most min(max_rows, 4 x (compute units)) rows of a call are split.  Pure host
 * computation; returns 0 for invalid arguments (max_rows < 0, K outside
 * [1, TOPK_K_MAX]). */
size_t topk_ragged_workspace_size(int32_t max_rows, int32_t K);

/* One-time initialisation of a workspace of `bytes` bytes (enqueued on
 * `stream` with kernels only, no memset nodes): writes the header (tag,
 * capacities) and zeroes every counter and per-row state.  The paper's
 * dispatch restores its persistent counters on the device so that replays
 * need no host work (Section 5.5, "Shape-stable dispatch"); here every call's
 * kernels return the state they used to zero, so this runs once, before the
 * first topk_ragged call on that workspace, and graph replays need no
 * re-initialisation.  workspace: device memory owned by the caller, 256-byte
 * aligned (as hipMalloc returns), at least topk_ragged_workspace_size(max_rows,
 * K) bytes.  Returns TOPK_EINVAL for a null or misaligned workspace or
 * invalid max_rows / K, TOPK_EWORKSPACE for a size below that, TOPK_ELAUNCH if
 * the launch fails. */
int topk_ragged_workspace_init(void *workspace, size_t bytes, int32_t max_rows, int32_t K,
                               void *stream);

/* Exact Top-K of every row.
 *   scores       device, FP32; row r is scores[row_offsets[r] ..
 *                row_offsets[r] + row_lengths[r]).  Rows may be packed
 *                back-to-back or padded to a pitch (row_offsets[r] = r*pitch);
 *                any 4-byte alignment is accepted.  Must be free of NaN.
 *   row_offsets  device, int64 [n_rows], element offsets (>= 0).
 *   row_lengths  device, int32 [n_rows], valid lengths (negative = 0), at
 *                most TOPK_L_MAX; a longer row is not selected: its outputs
 *                are -1 / -inf and the stats count an error.
 *   n_rows       >= 0; 0 is a no-op.
 *   K            1 <= K <= TOPK_K_MAX.
 *   out_idx      device, int32 [n_rows x K], row-relative indices.
 *   out_val      device, FP32 [n_rows x K], bit-exact copies of the scores.
 *   workspace    device, 256-byte aligned (as hipMalloc returns), initialised
 *                by topk_ragged_workspace_init with max_rows >= n_rows; not
 *                shared by concurrent calls (calls with separate workspaces
 *                may run concurrently, e.g. on different streams).
 * Row lengths and offsets stay on the device; the launch geometry depends
 * only on (n_rows, K, device).  A call of more than 2 x CUs and at most
 * 16384 rows enqueues a one-workgroup pre-pass before the main kernel: it
 * writes the work items into the workspace, rows longest first, the longest
 * of them cut into segments (at most 2 x CUs more items; row offsets below
 * 2^40 elements).  If the workspace is invalid for n_rows the kernel writes
 * -1 / -inf to every output and counts an error in the stats.
 * Returns TOPK_OK or an error code; nothing is enqueued on an argument
 * error. */
int topk_ragged(const float *scores, const int64_t *row_offsets, const int32_t *row_lengths,
                int32_t n_rows, int32_t K, int32_t *out_idx, float *out_val, void *workspace,
                void *stream);

/* topk_ragged with an explicit policy (NULL = topk_ragged_policy_for_k(K),
 * which is also what topk_ragged uses) and an optional per-row trace (device,
 * int32 [n_rows x TOPK_TRACE_WORDS], caller-owned, NULL = none) of the
 * integers that decide the row's route, in the paper's notation:
 *   [0] route (TOPK_ROUTE_*, TOPK_ROUTE_REREAD_FLAG or-ed in);
 *   [1] view size |V| (eq:method:view; -1 if L <= K);
 *   [2] tau0, [3] tau1: the primary and nested coarse boundaries of
 *       eq:method:primary-threshold (-1 if not sampled);
 *   [4] C(tau0): the admitted count of eq:method:candidate-set (Section 4.3);
 *   [5] C(tau1), evaluated only when C(tau0) < K (the band of
 *       eq:method:rescue-band; -1 otherwise);
 *   [6] tau_star: the exact coarse boundary of eq:method:exact-init (-1
 *       unless exact coarse recovery ran);
 *   [7] |Q0|: the frontier entering refinement (Section 4.4; -1 if L <= K).
 * Same errors as topk_ragged, plus TOPK_EINVAL for a policy out of range. */
int topk_ragged_ex(const float *scores, const int64_t *row_offsets, const int32_t *row_lengths,
                   int32_t n_rows, int32_t K, int32_t *out_idx, float *out_val, void *workspace,
                   const topk_ragged_policy *policy, int32_t *row_trace, void *stream);

/* Limits of topk_ragged_noalloc: most rows per call, and most rows with
 * per-row state: a call of at most that many rows may split any row, a larger
 * one splits at most that many of its longest rows. */
#define TOPK_NOALLOC_MAX_ROWS 16384
#define TOPK_NOALLOC_SPLIT_ROWS 64

/* topk_ragged without a workspace argument, for callers that cannot allocate
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).  The library keeps the workspace in a device array of about
 * 5.0 MB per GPU (header, work-item region, per-row state for
 * TOPK_NOALLOC_SPLIT_ROWS split rows), held until the process ends; this call
 * allocates nothing and calls no allocating routine.  The first call on a
 * device looks up the array's address and enqueues its one-time
 * initialisation on `stream` ahead of the call.  Arguments, outputs and
 * results are those of topk_ragged with the per-K policy: the same (index,
 * value) sets; a call of more than TOPK_NOALLOC_SPLIT_ROWS rows splits at most
 * that many rows.  Every call on one GPU uses that GPU's array: calls that overlap on
 * one GPU (concurrent streams or threads) race and must not be made; the
 * kernels leave the array's state zeroed for the next call.  Returns
 * TOPK_EWORKSPACE for n_rows > TOPK_NOALLOC_MAX_ROWS, otherwise as
 * topk_ragged. */
int topk_ragged_noalloc(const float *scores, const int64_t *row_offsets,
                        const int32_t *row_lengths, int32_t n_rows, int32_t K, int32_t *out_idx,
                        float *out_val, void *stream);

/* Copies the workspace's accumulated route counters (see topk_ragged_stats:
 * the per-route row counts behind the recovery rates of Section 6.4) to *out
 * (host memory owned by the caller) and resets them.  Synchronises `stream`:
 * for diagnostics outside timed or captured regions.  Returns TOPK_EINVAL for
 * a null or misaligned workspace or a null out, TOPK_ELAUNCH if a HIP call
 * fails. */
int topk_ragged_read_stats(void *workspace, topk_ragged_stats *out, void *stream);

/* Building-block probes for tests (device pointers):
 * coarse bins c(x) of n values (eq:method:coarse-map) into uint16 out_c, and
 * the inclusive ascending-key endpoint of each of the 2048 coarse bins into
 * out_cut (0xFFFFFFFF when no value falls in bins <= tau). */
int topk_ragged_debug_coarse(const float *x, int64_t n, uint16_t *out_c, void *stream);
int topk_ragged_debug_cutoffs(uint32_t *out_cut, void *stream);

/* Read-only ceiling of a call, for measurement: the work items topk_ragged
 * would launch for these rows and this K (the same split plan, per-K policy,
 * one workgroup for every row it does not split) stream every valid score
 * once with the same 16-byte loads and keep only the row's largest score.
 * Algorithmic bytes are the operator's own (one read of every valid score,
 * R_eq = 1 of Section 2.1, "Why long rows are expensive"), so the time of
 * this call bounds what the selector can reach in that geometry.  out_max: device, uint32
 * [n_rows], caller-owned, zeroed by the caller; receives the order-preserving
 * key of each row's largest score (0 for an empty row).  workspace: an
 * initialised workspace for at least n_rows rows (as for topk_ragged), whose
 * item-table region receives the work items of a call with more rows than
 * resident workgroups; no other part of it is written.  Same argument errors
 * as topk_ragged. */
int topk_ragged_debug_read_ceiling(const float *scores, const int64_t *row_offsets,
                                   const int32_t *row_lengths, int32_t n_rows, int32_t K,
                                   uint32_t *out_max, void *workspace, void *stream);

/* For tests of the split-row wait (Section 4.5 mapping): the number of polls a
 * segment makes for segment 0's published boundaries before it builds the
 * view itself (counted in topk_ragged_stats.wait_fallback), for the calls
 * launched after it; 0 restores the default.  Results do not depend on it.
 * Process-wide, not synchronised with concurrent calls.  Returns TOPK_OK, or
 * TOPK_EINVAL for a negative count. */
int topk_ragged_debug_set_spin_limit(int32_t polls);

/* Human-readable text for a status code. */
const char *topk_ragged_status_str(int status);

#ifdef __cplusplus
}
#endif

#endif /* TOPK_RAGGED_H */
