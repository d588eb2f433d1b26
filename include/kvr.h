/*
 * kvr.h — C ABI of the MI355X (gfx950) calibration-replay library.
 *
 * The library evaluates the GPU-opportunity cost of keeping a suspended
 * request's KV cache under every candidate retention policy, over a
 * calibration sample of approval waits, and selects the cheapest policy per
 * load level.  This is the calibration replay of "Adaptive KV Retention for
 * LLM Agents at Human-Approval Timescales" (Section 3.4: replay held-out
 * waits under both host branches, total the cost, freeze the cheaper branch),
 * widened to a grid of candidate timers, loads and bootstrap resamples.
 *
 * Cost definition (Section 3.1 Eq. 1, Section 3.3 Eq. 3, Appendix D):
 *   a request of T tokens suspends for w seconds.  It stays in HBM for
 *   min(w, t1) seconds at alpha_1 = T*a1 GPU-s/s (beta_1 = 0).  If w > t1 it
 *   is offloaded to host DRAM at t1 and a one-shot host timer t2 is armed;
 *   the deadline, measured from suspension, is e = t1 + t2 rounded once to
 *   binary64.  On the host it pays alpha_2(lambda) = T*a2(lambda) GPU-s/s
 *   until min(w, e), with
 *       a2(lambda) = max(0, lambda - lambda_crit) * b3 / C2,
 *       lambda_crit = C2 / W_ref            (Little's law saturation),
 *   then pays beta_2 = T*b2 at resume if w <= e (restore from host), or
 *   beta_3 = T*b3 if the copy was discarded at e (recompute); the copy made
 *   at offload is free unless kvr_prices.offload_per_token charges it (see
 *   there).  t2 = +inf is host-retain.  The cost of a policy (t1_a, t2_k, lambda_l) is the mean of
 *   the per-request cost over the sample, in GPU-s per request (the unit of
 *   Table 6).
 *
 * Conventions shared by every entry point:
 *   - Return value: KVR_OK (0) or a negative KVR_E_* code.  No exception
 *     crosses the ABI.  Errors detected on the host launch nothing and leave
 *     every output untouched.
 *   - "device" pointers are HIP device allocations owned by the caller
 *     (e.g. torch tensors); "host" pointers are ordinary host memory that the
 *     call reads before it returns and does not keep.
 *   - All device work is enqueued on hip_stream (a hipStream_t; NULL is the
 *     null stream) and is asynchronous: inputs must stay unchanged and
 *     outputs must not be read until the stream has been synchronised.
 *   - Workspace: calls that take (d_ws, ws_bytes) size it in two phases.
 *     With d_ws == NULL they write the required byte count into *ws_bytes,
 *     launch nothing and return KVR_OK; with d_ws != NULL, *ws_bytes must be
 *     at least that count (else KVR_E_WORKSPACE).  d_ws must be 256-byte
 *     aligned.  Apart from the optional profiling events of
 *     kvr_set_profile_events, the library keeps no state between calls;
 *     calls on distinct workspaces may run concurrently from different
 *     threads.
 *   - Device-detected domain errors (a wait that is NaN, infinite or
 *     negative; a context size below 1; a bootstrap index outside [0, n))
 *     cannot be reported by the return value of an asynchronous call.  The
 *     kernels record them in a status word at the start of the workspace and
 *     replace the offending value by a safe one; kvr_workspace_status() reads
 *     the word after synchronising the stream.  Outputs of such a call are
 *     meaningless.
 *   - Sizes: 1 <= n <= 2^31 - 1 samples; 1 <= n_t1, n_t2, n_lam;
 *     n_t1 * n_t2 <= 2^24 policies; n_lam <= 4096; n_resamples * m <= 2^40;
 *     n_resamples * n_lam <= 2^31 - 1; and every launch of the brute-force
 *     plan fits 2^31 - 1 workgroups (about n_resamples * n_t1 * n_t2 / 64
 *     for the grid kernel).  Beyond these: KVR_E_SIZE.
 */
#ifndef KVR_H
#define KVR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    KVR_OK = 0,
    KVR_E_NULL = -1,       /* a required pointer is NULL                          */
    KVR_E_SIZE = -2,       /* a count is out of range, or a product overflows     */
    KVR_E_GRID = -3,       /* timer/load grid invalid (see kvr_policy_grid)       */
    KVR_E_PRICE = -4,      /* a price, C2 or W_ref not finite and > 0 (offload >= 0) */
    KVR_E_WORKSPACE = -5,  /* workspace too small or not 256-byte aligned         */
    KVR_E_DOMAIN = -6,     /* device-detected bad sample or index (status word)   */
    KVR_E_HIP = -7,        /* a HIP runtime call failed                           */
    KVR_E_METHOD = -8      /* unknown method, or an option the method lacks       */
};

enum { KVR_BRUTE = 0, KVR_SORTED = 1 };   /* kvr_cost_grid methods            */
enum { KVR_RETAIN = 0, KVR_EXPIRE = 1 };  /* branch codes of kvr_select_policy */

/* Price vector per token (Appendix B) plus the host-tier constants of
 * Section 3.3.  The first five fields must be finite and > 0;
 * offload_per_token must be finite and >= 0 (anything else is KVR_E_PRICE).
 *
 * offload_per_token is an optional charge for the device-to-host copy made
 * when a context leaves HBM at t1: each request with w > t1 pays
 * T * offload_per_token once.  The paper leaves that copy uncharged (Section
 * 3.2: transfer time overlaps GPU execution; Eq. 1 prices resumes only), so
 * 0, what kvr_prices_from_platform writes, is the paper's model.  The grid
 * entry points (kvr_cost_grid, kvr_bootstrap, kvr_bootstrap_factored) add
 * it; kvr_eq3_timer and kvr_crossover_statistic do not depend on it (it is
 * paid before the host timer starts, and t* compares HBM holding with
 * recompute); the finite-capacity replay entry points (kvr_capacity_replay,
 * kvr_controller_select) model Table 6 without it and return KVR_E_METHOD
 * when it is not 0. */
typedef struct {
    double a1_per_token;       /* alpha_1 / T: GPU-s per second of HBM residency */
    double b2_per_token;       /* beta_2 / T: GPU-s to restore from host at resume */
    double b3_per_token;       /* beta_3 / T: GPU-s to recompute at resume       */
    double host_slots_c2;      /* C2: suspended contexts that fit in host DRAM   */
    double w_ref_s;            /* W_ref: reference residence time, seconds       */
    double offload_per_token;  /* GPU-s per token for the copy at offload; 0 = uncharged */
} kvr_prices;

/* Candidate policies and loads; all three arrays are HOST pointers.
 *   t1[n_t1]:  GPU-tier timers, seconds; finite, >= 0, strictly ascending.
 *              {0} means offload at suspension (Section 3.4).
 *   t2[n_t2]:  host timers, seconds; > 0, strictly ascending, not NaN; only
 *              the last may be +INFINITY (host-retain).
 *   lam[n_lam]: offered loads, suspended requests per second; finite, >= 0,
 *              any order.
 * Policies are indexed by the flat index f = a * n_t2 + k. */
typedef struct {
    const double *t1;  int32_t n_t1;
    const double *t2;  int32_t n_t2;
    const double *lam; int32_t n_lam;
} kvr_policy_grid;

/*
 * Appendix B price vector per token from platform constants (host only):
 *   a1 = n_gpu * kv_bytes_per_token / hbm_usable_bytes   (share of usable HBM)
 *   b2 = n_gpu * kv_bytes_per_token / host_link_bytes_per_s (restore time)
 *   b3 = n_gpu / prefill_tokens_per_s                     (re-prefill time)
 * host_slots_c2 and w_ref_s are copied through and offload_per_token is set to
 * 0 (the copy at offload uncharged; a caller who charges it sets the field,
 * e.g. to b2 for a link with the same bandwidth both ways).  Every argument
 * must be finite and > 0 (else KVR_E_PRICE); out must not be NULL
 * (KVR_E_NULL).
 */
int kvr_prices_from_platform(double kv_bytes_per_token, double hbm_usable_bytes,
                             double host_link_bytes_per_s, double prefill_tokens_per_s,
                             double n_gpu, double host_slots_c2, double w_ref_s,
                             kvr_prices *out);

/*
 * Cost grid of one calibration sample (the replay of Section 3.4 over every
 * candidate policy and load).
 *   d_wait_s[n]     device, float64: suspension (approval) waits, seconds.
 *   d_ctx_tokens[n] device, int32: context tokens per request (T >= 1).
 *   p, g            host: prices and policy grid (validated on the host).
 *   method          KVR_BRUTE: the load-dependent holding term of every
 *                   (sample, policy, load) evaluated, one fp64 FMA each; the
 *                   load-independent terms are summed once per (sample, t1)
 *                   (HBM residency, offload) and, for the recompute branch,
 *                   counted once per (sample, deadline) through deadline bins;
 *                   KVR_SORTED: stable radix sort of the waits, prefix sums
 *                   of T and T*w, closed form per policy.
 *   d_cost          device, float64 [n_lam][n_t1][n_t2]: mean GPU-s per
 *                   request (written in full).
 *   d_perm          device, int32 [n] or NULL: KVR_SORTED only, the stable
 *                   ascending order of the waits (-0.0 equals +0.0; equal
 *                   waits keep input order).  Non-NULL with KVR_BRUTE is
 *                   KVR_E_METHOD.
 *   d_ws, ws_bytes  workspace (two-phase sizing, see above).
 */
int kvr_cost_grid(const double *d_wait_s, const int32_t *d_ctx_tokens, int64_t n,
                  const kvr_prices *p, const kvr_policy_grid *g, int32_t method,
                  double *d_cost, int32_t *d_perm,
                  void *d_ws, size_t *ws_bytes, void *hip_stream);

/*
 * Policy selection (Section 3.4: freeze the cheaper branch), per load.
 *   d_cost          device, float64 [batch][n_lam][n_t1][n_t2].
 *   last_t2_is_inf  1 if the last host timer is +inf (host-retain), else 0.
 *   d_best          device, int32 [batch][n_lam]: flat index f = a*n_t2 + k
 *                   of the smallest cost; exact ties go to the larger f.
 *   d_best_cost     device, float64 [batch][n_lam].
 *   d_branch        device, int32 [batch][n_lam] or NULL: KVR_RETAIN if the
 *                   chosen timer is the infinite one, else KVR_EXPIRE.
 * No workspace; costs are expected to be finite (NaN costs give an
 * unspecified index).
 */
int kvr_select_policy(const double *d_cost, int64_t batch, int32_t n_lam, int32_t n_t1,
                      int32_t n_t2, int32_t last_t2_is_inf,
                      int32_t *d_best, double *d_best_cost, int32_t *d_branch,
                      void *hip_stream);

/*
 * Bootstrap calibration: the brute-force grid (as KVR_BRUTE of kvr_cost_grid:
 * every (draw, policy, load) holding term evaluated, the load-independent
 * terms summed per (draw, t1) and binned per (draw, deadline)) over every
 * resample, with the selection fused per resample.
 *   d_wait_s[n], d_ctx_tokens[n]  device: the base sample (as kvr_cost_grid).
 *   d_idx           device, int32 [n_resamples][m]: with-replacement draws,
 *                   each in [0, n).  The caller draws them (seeded).
 *   d_best          device, int32 [n_resamples][n_lam]: selected flat index.
 *   d_best_cost     device, float64 [n_resamples][n_lam].
 *   d_cost          device, float64 [n_resamples][n_lam][n_t1][n_t2] or
 *                   NULL: the full cost tensor, when the caller wants it.
 */
int kvr_bootstrap(const double *d_wait_s, const int32_t *d_ctx_tokens, int64_t n,
                  const int32_t *d_idx, int64_t n_resamples, int64_t m,
                  const kvr_prices *p, const kvr_policy_grid *g,
                  int32_t *d_best, double *d_best_cost, double *d_cost,
                  void *d_ws, size_t *ws_bytes, void *hip_stream);

/*
 * Synchronise hip_stream and read the status word (the first bytes of the
 * workspace) of a call of any compute entry point here (kvr_cost_grid,
 * kvr_bootstrap, kvr_bootstrap_factored, kvr_capacity_replay,
 * kvr_controller_select, kvr_crossover_statistic): KVR_OK, KVR_E_DOMAIN, or
 * KVR_E_HIP if the synchronisation or the read failed.  d_ws NULL is
 * KVR_E_NULL.
 */
int kvr_workspace_status(const void *d_ws, void *hip_stream);

/*
 * Bootstrap calibration by the multiplicity-count closed form: a second
 * method for the same result as kvr_bootstrap (Eq. 1 with Eq. 3 integrated
 * over the sorted waits, the SORTED path's closed form, with the number of
 * times each resample draws a base sample as its weight).  The base sample is
 * sorted once; per resample the work is O(m + n + n_t1*n_t2*n_lam) instead of
 * O(m*n_t1*n_t2*n_lam).  Arguments, outputs, layouts and errors are those of
 * kvr_bootstrap, except n <= 2^31 - 2.  The prefix sums of T*w round
 * differently from the brute force's per-sample sums, so costs agree with it
 * within rounding (about 1e-12 relative on the bench workloads) and the
 * selection is the same up to rounding-level near ties.
 */
int kvr_bootstrap_factored(const double *d_wait_s, const int32_t *d_ctx_tokens, int64_t n,
                           const int32_t *d_idx, int64_t n_resamples, int64_t m,
                           const kvr_prices *p, const kvr_policy_grid *g, int32_t *d_best,
                           double *d_best_cost, double *d_cost, void *d_ws, size_t *ws_bytes,
                           void *hip_stream);

/*
 * Eq. 3 timer (host only): t2(lambda) = +inf if lambda <= lambda_crit =
 * C2/W_ref, else (beta_3 - beta_2) / alpha_2(lambda) with alpha_2(lambda) =
 * (lambda - lambda_crit) * beta_3 / C2.  With per-token prices both terms scale
 * with T, so the timer is the same for every context size.  Writes *t2_out;
 * KVR_E_PRICE for an invalid price vector, KVR_E_GRID for a load that is not
 * finite and >= 0, KVR_E_NULL for NULL pointers.
 */
int kvr_eq3_timer(const kvr_prices *p, double lambda, double *t2_out);

/*
 * Finite-capacity admission replay (Appendix D; the replay behind Table 6 and
 * the replay columns of Table 3).  Each row is one sequence of suspensions:
 * every request is offloaded to host DRAM at suspension; the host tier holds
 * C2 contexts (p->host_slots_c2, an integer >= 1); a request that arrives
 * while a slot is free is admitted, one that finds the tier full recomputes
 * at resume (beta_3), and residents are never displaced.  Under host timer t2
 * an admitted request whose wait exceeds t2 is discarded at arrival + t2
 * (recompute at resume); otherwise it is restored from host (beta_2) and
 * leaves at arrival + wait.  Departures at or before an arrival free their
 * slots first.  No holding price is charged: capacity is enforced directly.
 *   d_arrival_s     device, float64 [n_reps][n]: suspension times, seconds,
 *                   finite, >= 0, non-decreasing within a row.
 *   d_wait_s        device, float64 [n_reps][n]: waits, finite, >= 0.
 *   d_ctx_tokens    device, int32 [n_reps][n] or NULL (every context 1 token).
 *   p               host: b2, b3 and host_slots_c2 are used (all fields must be
 *                   valid; C2 not an integer >= 1 is KVR_E_PRICE; a nonzero
 *                   offload_per_token is KVR_E_METHOD).
 *   t2[n_t2]        host: host timers, > 0 (+INFINITY = host-retain), any order.
 *   d_cost          device, float64 [n_reps][n_t2]: mean GPU-s per request,
 *                   (b2*R + b3*(Ttot - R)) / n with R the restored tokens.
 *   d_restored_tokens, d_admitted  device, int64 [n_reps][n_t2] or NULL:
 *                   tokens restored from host, requests admitted (exact).
 *   Sizes: 1 <= n <= 8192, 1 <= n_t2 <= 4096, n_reps * n_t2 <= 2^31 - 1.
 *   Workspace: two-phase sizing as above.
 */
int kvr_capacity_replay(const double *d_arrival_s, const double *d_wait_s,
                        const int32_t *d_ctx_tokens, int64_t n_reps, int64_t n,
                        const kvr_prices *p, const double *t2, int32_t n_t2,
                        double *d_cost, int64_t *d_restored_tokens, int64_t *d_admitted,
                        void *d_ws, size_t *ws_bytes, void *hip_stream);

/* Result of kvr_controller_select, written to device memory by the library.
 * Every field is 8 bytes wide (120 bytes, no padding).  In each pair, index 0
 * is the Eq. 3 timer branch and index 1 is host-retain. */
typedef struct {
    int64_t branch;              /* KVR_RETAIN (also on equal totals) or KVR_EXPIRE */
    int64_t restored_tokens[2];  /* tokens restored from host over the whole sample */
    int64_t admitted[2];         /* requests admitted to the host tier */
    int64_t total_tokens;        /* context tokens over the whole sample */
    int64_t n_short;             /* waits w <= t* */
    int64_t n_requests;          /* n_reps * n */
    double t2_s;                 /* Eq. 3 timer at lambda; +inf at or below lambda_crit */
    double total_cost[2];        /* b2*R + b3*(Ttot - R), GPU-s, summed over the sample */
    double cost_per_request[2];  /* total_cost / n_requests */
    double t_star_s;             /* break-even time t* = beta_3 / alpha_1 */
    double p_short;              /* n_short / n_requests, i.e. P(W <= t*) */
} kvr_controller_out;

/*
 * Regime-aware controller (Section 3.4; calibrated once and frozen across
 * loads, Appendix F).  Replays the calibration sample with finite host
 * capacity exactly as kvr_capacity_replay does, under the Eq. 3 timer
 * t2(lambda) and under host-retain; totals each branch's GPU opportunity cost
 * over the whole sample, b2*R + b3*(Ttot - R); freezes the cheaper branch.
 * Equal totals keep host-retain (at or below lambda_crit the two branches are
 * one policy).  At run time a frozen KVR_EXPIRE branch needs only the offered
 * load: kvr_eq3_timer gives its timer.  The same call reports the summary
 * statistic of Section 4.3 / Figure 4(d): the share of calibration waits at
 * or below the break-even time t* = beta_3 / alpha_1.
 *   d_arrival_s, d_wait_s, d_ctx_tokens, n_reps, n: the calibration sample,
 *                   laid out and validated as in kvr_capacity_replay (its
 *                   arrivals are expected to be drawn at the load lambda).
 *   p               host: every field is used (alpha_1 for t*); C2 must be an
 *                   integer >= 1 (else KVR_E_PRICE); a nonzero
 *                   offload_per_token is KVR_E_METHOD.
 *   lambda          host: calibration load, suspended requests per second,
 *                   finite and >= 0 (else KVR_E_GRID).
 *   d_out           device: one kvr_controller_out, written by the call.
 *   Sizes: 1 <= n <= 8192, n_reps * 2 <= 2^31 - 1.  Workspace: two-phase
 *   sizing as above.
 */
int kvr_controller_select(const double *d_arrival_s, const double *d_wait_s,
                          const int32_t *d_ctx_tokens, int64_t n_reps, int64_t n,
                          const kvr_prices *p, double lambda, kvr_controller_out *d_out,
                          void *d_ws, size_t *ws_bytes, void *hip_stream);

/*
 * The crossover statistic of Section 4.3 / Figure 4(d) on any wait sample:
 * the share of waits at or below t* = beta_3 / alpha_1 (a rank query; the
 * library counts rather than sorts).
 *   d_wait_s        device, float64 [n]: waits, finite and >= 0 (else
 *                   KVR_E_DOMAIN through the workspace status word).
 *   p               host: a1 and b3 give t*; every field must be valid.
 *   d_count         device, int64 [1]: the number of waits w <= t* (exact).
 *   d_fraction      device, float64 [1] or NULL: d_count / n.
 *   Sizes: 1 <= n <= 2^40.  Workspace: two-phase sizing as above.
 */
int kvr_crossover_statistic(const double *d_wait_s, int64_t n, const kvr_prices *p,
                            int64_t *d_count, double *d_fraction, void *d_ws, size_t *ws_bytes,
                            void *hip_stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): kvr_cost_grid
 * without a workspace argument.  The workspace is a file-scope device array of
 * KVR_NOALLOC_SCRATCH_BYTES inside the library, one copy per GPU, held from
 * the library's load until the process ends; the call allocates and frees
 * nothing.  Arguments, checks, layouts and results are those of kvr_cost_grid,
 * with these differences:
 *   - The workspace kvr_cost_grid would need (its d_ws == NULL size) must fit
 *     KVR_NOALLOC_SCRATCH_BYTES, else KVR_E_SIZE and nothing is launched.  To
 *     fit, KVR_BRUTE may sum a sample in fewer splits than kvr_cost_grid does;
 *     costs then agree with kvr_cost_grid's to rounding (the splits are added
 *     in another grouping), and are bit-identical whenever kvr_cost_grid's own
 *     workspace fits.  About 1.6 million waits fit KVR_SORTED.
 *   - d_status      device, int32 [1] or NULL: written at the end of the
 *                   call's work on hip_stream with KVR_OK or KVR_E_DOMAIN (the
 *                   device-detected errors that kvr_workspace_status reports
 *                   for kvr_cost_grid).
 *   - Every call on one GPU uses that GPU's single copy of the array: calls
 *     queued on one stream are ordered, but calls that overlap in time on one
 *     GPU (different streams, different host threads) race and give
 *     meaningless results.  The array keeps the last call's contents; the
 *     kernels clear whatever must start at zero.
 *   - hip_stream must belong to a device of index < 64.
 */
#define KVR_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
int kvr_cost_grid_noalloc(const double *d_wait_s, const int32_t *d_ctx_tokens, int64_t n,
                          const kvr_prices *p, const kvr_policy_grid *g, int32_t method,
                          double *d_cost, int32_t *d_perm, int32_t *d_status, void *hip_stream);

/*
 * Instrumentation for benchmarks.  After this call, every kvr_cost_grid,
 * kvr_cost_grid_noalloc, kvr_bootstrap, kvr_bootstrap_factored,
 * kvr_capacity_replay and kvr_controller_select call made from the same host
 * thread records ev_begin (a hipEvent_t) on its stream right before its main
 * stage and ev_end right after it, so hipEventElapsedTime(ev_begin, ev_end) is
 * that stage's device time.  The stage is the brute-force grid kernel alone
 * (kvr_cost_grid and kvr_cost_grid_noalloc with KVR_BRUTE, kvr_bootstrap), the
 * whole sorted path from its first kernel (KVR_SORTED), the whole factored
 * path (kvr_bootstrap_factored), the replay
 * (kvr_capacity_replay), or the replay, count and final kernels
 * (kvr_controller_select).  kvr_set_profile_events(NULL, NULL)
 * stops it.  These two handles, kept per host thread, are the only state the
 * library holds between calls; the events stay owned by the caller.
 * Returns KVR_E_NULL if exactly one of the two is NULL.
 */
int kvr_set_profile_events(void *ev_begin, void *ev_end);

/* Static English text for a status code (never NULL). */
const char *kvr_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* KVR_H */
