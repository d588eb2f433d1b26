/*
 * TEST INFRASTRUCTURE — NOT PART OF THE PRODUCT PATH.
 *
 * Plain, slow CPU reference ("oracle") for the calibration replay of
 * "Adaptive KV Retention for LLM Agents at Human-Approval Timescales".
 * Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may
 * load this library.  It shares no code, header, table or constant with the
 * HIP library under paper_2608_30830_amd/, and includes nothing from it.
 *
 * Built with: gcc -O2 -ffp-contract=off -fopenmp -shared -fPIC (no fast-math),
 * so every operation below is one IEEE binary64 round-to-nearest-even step.
 *
 * What is computed (policies outer, samples inner):
 *
 *   Section 3.1, Eq. (1): a context that stays in state j for l seconds costs
 *   alpha_j * l + beta_j GPU-seconds; state 1 = HBM (beta_1 = 0), 2 = host
 *   DRAM (resume cost beta_2 = restore), 3 = discarded (alpha_3 = 0, resume
 *   cost beta_3 = recompute).  Prices are per token, so a context of T tokens
 *   pays T times each price.
 *
 *   Section 3.3, Eq. (3): lambda_crit = C2 / W_ref (Little's law saturation),
 *   alpha_2(lambda) = max(0, lambda - lambda_crit) * beta_3 / C2.
 *
 *   Section 3.4 and Appendix D: a suspended context stays in HBM for t1
 *   seconds, then moves to host DRAM and receives a one-shot host timer t2;
 *   if it has not resumed when the timer fires (deadline e = t1 + t2 from
 *   suspension) the host copy is discarded.  Resume at wait w pays beta_2 if
 *   the host copy is still there (w <= e), beta_3 otherwise; a resume while
 *   still in HBM (w <= t1) pays nothing.  t2 = +inf is host-retain.
 *
 *   Per sample:  c = T * ( a1*min(w,t1)
 *                          + [w > t1] * ( a2*(min(w,e) - t1) + (w <= e ? b2 : b3) + boff ) )
 *   boff is an optional per-token charge for the device-to-host copy made at
 *   offload.  The paper leaves that copy uncharged (Section 3.2: transfer time
 *   overlaps GPU work; Eq. 1 has resume costs only), so boff = 0 is the
 *   paper's model; a positive boff charges it once per offloaded request.
 *   Per policy (t1_a, t2_k, lambda_l): mean of c over the sample (GPU-s per
 *   request, the unit of Table 6), summed with Neumaier compensation.
 *   Selection (Section 3.4, the calibration replay freezes the cheaper
 *   branch): per load, arg-min over the flat policy index f = a*K2 + k, exact
 *   ties going to the larger f (longer retention; Section 1 notes that
 *   expiration only adds churn when elapsed age is uninformative).
 *
 *   The closed form (oracle_closed_form_grid) is an independent second
 *   derivation of the same mean from prefix sums over the samples sorted by
 *   wait; it exists to pin the double loop, and for bootstrap rows it uses
 *   per-sample multiplicities instead of gathering.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* Appendix B: price vector per token.
 *   alpha_1: a context's share of the usable HBM, charged across the GPUs
 *            (GPU-s per second of residency);
 *   beta_2:  host-to-device restore time over the host link, per GPU;
 *   beta_3:  re-prefill time at the measured prefill rate, per GPU. */
void oracle_prices_from_platform(double kv_bytes_per_token, double hbm_usable_bytes,
                                 double host_link_bytes_per_s, double prefill_tokens_per_s,
                                 double n_gpu, double *a1, double *b2, double *b3)
{
    *a1 = n_gpu * kv_bytes_per_token / hbm_usable_bytes;
    *b2 = n_gpu * kv_bytes_per_token / host_link_bytes_per_s;
    *b3 = n_gpu / prefill_tokens_per_s;
}

/* Eq. (3): lambda_crit and the per-token congestion price a2 for each load. */
double oracle_lambda_crit(double c2, double w_ref)
{
    return c2 / w_ref;
}

void oracle_congestion_prices(const double *lam, int32_t n_lam, double b3,
                              double c2, double w_ref, double *a2_out)
{
    double lc = oracle_lambda_crit(c2, w_ref);
    for (int32_t l = 0; l < n_lam; ++l) {
        double p = lam[l] - lc;
        if (!(p > 0.0)) p = 0.0;
        a2_out[l] = (p * b3) / c2;
    }
}

/* Eq. (3) timer: t2(lambda) = inf if lambda <= lambda_crit,
 * else (beta_3 - beta_2) / alpha_2(lambda).  Per-token prices give the same
 * timer for every context size, since both numerator and denominator scale
 * with T. */
double oracle_eq3_timer(double lam, double b2, double b3, double c2, double w_ref)
{
    double a2;
    oracle_congestion_prices(&lam, 1, b3, c2, w_ref, &a2);
    if (!(a2 > 0.0)) return INFINITY;
    return (b3 - b2) / a2;
}

/* The per-sample cost written out state by state (Eq. 1 summed over the
 * states visited, Appendix D one-shot timer semantics). */
static double sample_cost(double w, double T, double t1, double e,
                          double a1, double a2, double b2, double b3, double boff)
{
    double hbm_time = (w < t1) ? w : t1;          /* seconds in HBM        */
    double cost = a1 * hbm_time;                   /* alpha_1 * l, beta_1=0 */
    if (w > t1) {                                  /* offloaded at t1       */
        double host_end = (w < e) ? w : e;         /* resume or deadline    */
        double host = a2 * (host_end - t1);        /* alpha_2(lambda) * l   */
        double resume = (w <= e) ? b2 : b3;        /* restore or recompute  */
        cost = cost + (host + resume + boff);      /* boff: the offload copy */
    }
    return T * cost;
}

/* Neumaier-compensated running sum. */
typedef struct { double s, c; } nsum;
static inline void nsum_add(nsum *a, double x)
{
    double t = a->s + x;
    if (fabs(a->s) >= fabs(x)) a->c += (a->s - t) + x;
    else a->c += (x - t) + a->s;
    a->s = t;
}
static inline double nsum_get(const nsum *a) { return a->s + a->c; }

/*
 * Full cost grid, one resample.
 *   wait_s[n], ctx[n]: the base sample.
 *   idx: NULL for the base sample itself (m must equal n), else m indices.
 *   cost_out: [n_lam][n_t1][n_t2], mean GPU-s per request.
 * Deadlines e = t1 + t2 and the per-token a2 are derived exactly as above.
 */
void oracle_cost_grid(const double *wait_s, const int32_t *ctx, int64_t n,
                      const int32_t *idx, int64_t m,
                      double a1, double b2, double b3, double boff, double c2, double w_ref,
                      const double *t1, int32_t n_t1,
                      const double *t2, int32_t n_t2,
                      const double *lam, int32_t n_lam,
                      double *cost_out)
{
    (void)n;
    double *a2 = (double *)malloc(sizeof(double) * (size_t)(n_lam > 0 ? n_lam : 1));
    oracle_congestion_prices(lam, n_lam, b3, c2, w_ref, a2);
    int64_t n_pol = (int64_t)n_lam * n_t1 * n_t2;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t p = 0; p < n_pol; ++p) {
        int32_t l = (int32_t)(p / ((int64_t)n_t1 * n_t2));
        int32_t a = (int32_t)((p / n_t2) % n_t1);
        int32_t k = (int32_t)(p % n_t2);
        double e = t1[a] + t2[k];
        nsum acc = {0.0, 0.0};
        for (int64_t j = 0; j < m; ++j) {
            int64_t i = idx ? (int64_t)idx[j] : j;
            nsum_add(&acc, sample_cost(wait_s[i], (double)ctx[i], t1[a], e,
                                       a1, a2[l], b2, b3, boff));
        }
        cost_out[p] = nsum_get(&acc) / (double)m;
    }
    free(a2);
}

/*
 * Selection over a batch of cost grids [batch][n_lam][n_t1*n_t2]:
 * best flat index f = a*n_t2 + k with the smallest cost, exact ties to the
 * larger f.  branch = 0 (RETAIN) iff the chosen host timer is +inf, else 1.
 */
void oracle_select(const double *cost, int64_t batch, int32_t n_lam,
                   int32_t n_t1, int32_t n_t2, const double *t2,
                   int32_t *best, double *best_cost, int32_t *branch)
{
    int64_t P = (int64_t)n_t1 * n_t2;
    for (int64_t b = 0; b < batch; ++b)
        for (int32_t l = 0; l < n_lam; ++l) {
            const double *row = cost + (b * n_lam + l) * P;
            int64_t bi = 0;
            double bc = row[0];
            for (int64_t f = 1; f < P; ++f)
                if (row[f] <= bc) { bc = row[f]; bi = f; }
            best[b * n_lam + l] = (int32_t)bi;
            best_cost[b * n_lam + l] = bc;
            if (branch)
                branch[b * n_lam + l] = isinf(t2[bi % n_t2]) ? 0 : 1;
        }
}

/* Stable ascending order of the waits (numeric comparison, so -0.0 and +0.0
 * are equal and keep input order).  Plain top-down merge sort. */
static void merge_sort_rec(const double *w, int32_t *a, int32_t *tmp, int64_t lo, int64_t hi)
{
    if (hi - lo < 2) return;
    int64_t mid = lo + (hi - lo) / 2;
    merge_sort_rec(w, a, tmp, lo, mid);
    merge_sort_rec(w, a, tmp, mid, hi);
    int64_t i = lo, j = mid, o = lo;
    while (i < mid && j < hi) {
        if (w[a[j]] < w[a[i]]) tmp[o++] = a[j++];   /* strict: ties keep left */
        else tmp[o++] = a[i++];
    }
    while (i < mid) tmp[o++] = a[i++];
    while (j < hi) tmp[o++] = a[j++];
    memcpy(a + lo, tmp + lo, sizeof(int32_t) * (size_t)(hi - lo));
}

void oracle_stable_order(const double *wait_s, int64_t n, int32_t *perm)
{
    int32_t *tmp = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n > 0 ? n : 1));
    for (int64_t i = 0; i < n; ++i) perm[i] = (int32_t)i;
    merge_sort_rec(wait_s, perm, tmp, 0, n);
    free(tmp);
}

/* Number of sorted waits <= x. */
static int64_t upper_bound(const double *sw, int64_t n, double x)
{
    int64_t lo = 0, hi = n;
    while (lo < hi) {
        int64_t mid = lo + (hi - lo) / 2;
        if (sw[mid] <= x) lo = mid + 1; else hi = mid;
    }
    return lo;
}

/*
 * Closed form of the same mean (second derivation).  With the samples sorted
 * by wait and per-sample multiplicities c_i (1 for the base sample, the
 * number of times a bootstrap row draws i otherwise):
 *   N(x) = sum_{w_i <= x} c_i T_i,  S(x) = sum_{w_i <= x} c_i T_i w_i,
 *   Ttot = N(inf),
 *   m*C = a1*[S(t1) + t1*(Ttot - N(t1))]
 *       + a2*[(S(e) - S(t1)) - t1*(N(e) - N(t1)) + (e - t1)*(Ttot - N(e))]
 *       + b2*(N(e) - N(t1)) + b3*(Ttot - N(e)) + boff*(Ttot - N(t1)),
 * where the (e - t1)*(Ttot - N(e)) term is dropped when e = +inf (no sample
 * lies past an infinite deadline).  Integer sums N are exact in int64.
 *
 *   perm: stable order of the base waits (oracle_stable_order).
 *   idx/m: NULL and m = n for the base sample, else one bootstrap row.
 *   cost_out: [n_lam][n_t1][n_t2].
 */
void oracle_closed_form_grid(const double *wait_s, const int32_t *ctx, int64_t n,
                             const int32_t *perm, const int32_t *idx, int64_t m,
                             double a1, double b2, double b3, double boff, double c2,
                             double w_ref, const double *t1, int32_t n_t1,
                             const double *t2, int32_t n_t2,
                             const double *lam, int32_t n_lam,
                             double *cost_out)
{
    int64_t *mult = (int64_t *)calloc((size_t)(n > 0 ? n : 1), sizeof(int64_t));
    double *sw = (double *)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
    int64_t *N = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n + 1));
    double *S = (double *)malloc(sizeof(double) * (size_t)(n + 1));
    double *a2 = (double *)malloc(sizeof(double) * (size_t)(n_lam > 0 ? n_lam : 1));
    if (idx) { for (int64_t j = 0; j < m; ++j) mult[idx[j]] += 1; }
    else { for (int64_t i = 0; i < n; ++i) mult[i] = 1; }
    N[0] = 0; S[0] = 0.0;
    for (int64_t j = 0; j < n; ++j) {
        int64_t i = perm[j];
        sw[j] = wait_s[i];
        int64_t cT = mult[i] * (int64_t)ctx[i];
        N[j + 1] = N[j] + cT;
        S[j + 1] = S[j] + (double)cT * wait_s[i];
    }
    oracle_congestion_prices(lam, n_lam, b3, c2, w_ref, a2);
    double Ttot = (double)N[n];
    for (int32_t a = 0; a < n_t1; ++a) {
        int64_t p1 = upper_bound(sw, n, t1[a]);
        double N1 = (double)N[p1], S1 = S[p1];
        double hbm = S1 + t1[a] * (Ttot - N1);
        for (int32_t k = 0; k < n_t2; ++k) {
            double e = t1[a] + t2[k];
            int64_t pe = upper_bound(sw, n, e);
            double Ne = (double)N[pe], Se = S[pe];
            double hold = (Se - S1) - t1[a] * (Ne - N1);
            if (!isinf(e)) hold = hold + (e - t1[a]) * (Ttot - Ne);
            double fixed = a1 * hbm + b2 * (Ne - N1) + b3 * (Ttot - Ne) + boff * (Ttot - N1);
            for (int32_t l = 0; l < n_lam; ++l)
                cost_out[((int64_t)l * n_t1 + a) * n_t2 + k] =
                    (fixed + a2[l] * hold) / (double)m;
        }
    }
    free(mult); free(sw); free(N); free(S); free(a2);
}

/* Closed-form selection for every bootstrap row (used to check all rows of a
 * large batch): best[R][n_lam], best_cost[R][n_lam]. */
void oracle_closed_form_bootstrap(const double *wait_s, const int32_t *ctx, int64_t n,
                                  const int32_t *idx, int64_t n_rows, int64_t m,
                                  double a1, double b2, double b3, double boff, double c2,
                                  double w_ref, const double *t1, int32_t n_t1,
                                  const double *t2, int32_t n_t2,
                                  const double *lam, int32_t n_lam,
                                  int32_t *best, double *best_cost)
{
    int32_t *perm = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n > 0 ? n : 1));
    oracle_stable_order(wait_s, n, perm);
    int64_t P = (int64_t)n_t1 * n_t2;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t r = 0; r < n_rows; ++r) {
        double *cost = (double *)malloc(sizeof(double) * (size_t)(P * n_lam));
        oracle_closed_form_grid(wait_s, ctx, n, perm, idx + r * m, m, a1, b2, b3, boff,
                                c2, w_ref, t1, n_t1, t2, n_t2, lam, n_lam, cost);
        oracle_select(cost, 1, n_lam, n_t1, n_t2, t2, best + r * n_lam,
                      best_cost + r * n_lam, NULL);
        free(cost);
    }
    free(perm);
}

int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Thread count of later parallel loops (timing of the oracle only). */
void oracle_set_num_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/*
 * Finite-capacity admission replay (Appendix D; the evaluation behind
 * Table 6).  Requests suspend at their arrival times (ascending) and resume
 * after their waits; every request is offloaded to host DRAM at suspension.
 * The host tier has C2 slots: a request that arrives when a slot is free is
 * admitted, one that finds the tier full is not admitted and recomputes at
 * resume; residents are never displaced.  Under a host timer t2 an admitted
 * request whose wait exceeds t2 is discarded at arrival + t2 (its slot frees
 * then) and recomputes at resume; otherwise it is restored from host at
 * arrival + wait.  t2 = +inf is host-retain.  Departures at or before an
 * arrival free their slots before that arrival is admitted; a resume at the
 * instant its timer fires counts as a restore.  No holding price is charged:
 * capacity is enforced directly.
 *
 *   arrival_s[n] ascending, wait_s[n], ctx[n] (NULL: every context 1 token).
 *   restored_tokens_out: sum of T over restored requests (exact integer).
 *   Returns the mean cost per request, (b2*R + b3*(Ttot - R)) / n with
 *   R = restored_tokens_out, which is also how the GPU path reports it.
 */
typedef struct { double *v; int64_t size; } minheap;

static void heap_push(minheap *h, double x)
{
    int64_t i = h->size++;
    h->v[i] = x;
    while (i > 0) {
        int64_t p = (i - 1) / 2;
        if (!(h->v[i] < h->v[p])) break;
        double t = h->v[i]; h->v[i] = h->v[p]; h->v[p] = t;
        i = p;
    }
}

static void heap_pop(minheap *h)
{
    h->v[0] = h->v[--h->size];
    int64_t i = 0;
    for (;;) {
        int64_t l = 2 * i + 1, r = l + 1, s = i;
        if (l < h->size && h->v[l] < h->v[s]) s = l;
        if (r < h->size && h->v[r] < h->v[s]) s = r;
        if (s == i) break;
        double t = h->v[i]; h->v[i] = h->v[s]; h->v[s] = t;
        i = s;
    }
}

double oracle_capacity_replay(const double *arrival_s, const double *wait_s, const int32_t *ctx,
                              int64_t n, int64_t c2, double t2, double b2, double b3,
                              int64_t *restored_tokens_out, int64_t *admitted_out)
{
    minheap h;
    h.v = (double *)malloc(sizeof(double) * (size_t)(c2 > 0 ? c2 : 1));
    h.size = 0;
    int64_t restored = 0, total = 0, admitted = 0;
    for (int64_t i = 0; i < n; ++i) {
        const double a = arrival_s[i], w = wait_s[i];
        const int64_t T = ctx ? (int64_t)ctx[i] : 1;
        total += T;
        while (h.size > 0 && h.v[0] <= a) heap_pop(&h);     /* resumed or expired by now */
        if (h.size < c2) {
            admitted += 1;
            if (w <= t2) {                                   /* resumes before the timer */
                restored += T;
                heap_push(&h, a + w);
            } else {                                         /* discarded at the timer   */
                heap_push(&h, a + t2);
            }
        }                                                    /* else: tier full, recompute */
    }
    free(h.v);
    if (restored_tokens_out) *restored_tokens_out = restored;
    if (admitted_out) *admitted_out = admitted;
    return (b2 * (double)restored + b3 * (double)(total - restored)) / (double)n;
}

/* Many replays: rows of arrivals/waits [reps][n] x host timers [n_t2];
 * outputs [reps][n_t2]. */
void oracle_capacity_replay_batch(const double *arrival_s, const double *wait_s,
                                  const int32_t *ctx, int64_t reps, int64_t n, int64_t c2,
                                  const double *t2, int32_t n_t2, double b2, double b3,
                                  double *cost_out, int64_t *restored_out)
{
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t q = 0; q < reps * n_t2; ++q) {
        int64_t r = q / n_t2, k = q % n_t2;
        int64_t rest = 0;
        cost_out[q] = oracle_capacity_replay(arrival_s + r * n, wait_s + r * n,
                                             ctx ? ctx + r * n : NULL, n, c2, t2[k], b2, b3,
                                             &rest, NULL);
        if (restored_out) restored_out[q] = rest;
    }
}

/*
 * Regime-aware controller (Section 3.4; frozen across loads as in Appendix F).
 * The same calibration sample -- n_reps sequences of n suspensions -- is
 * replayed with finite capacity under the two host branches: the Eq. 3 timer
 * t2(lambda) and host-retain (t2 = +inf).  Each branch's GPU opportunity cost
 * is totalled over every request of the sample, b2*R + b3*(Ttot - R) with R
 * the tokens restored from host, and the cheaper branch is frozen; equal
 * totals keep host-retain (the timer only adds churn then, and below
 * lambda_crit the two branches are the same policy).  The sample's summary
 * statistic of Section 4.3 / Figure 4(d) is the fraction of its waits at or
 * below the break-even time t* = beta_3 / alpha_1.
 *
 *   i64_out[8]: branch (0 retain, 1 expire), R[timer], R[retain],
 *               admitted[timer], admitted[retain], Ttot, #(w <= t*), n_reps*n.
 *   f64_out[7]: t2(lambda), total cost[timer], total cost[retain],
 *               cost per request[timer], cost per request[retain], t*, P(W <= t*).
 */
void oracle_controller_select(const double *arrival_s, const double *wait_s, const int32_t *ctx,
                              int64_t n_reps, int64_t n, int64_t c2, double lam, double a1,
                              double b2, double b3, double w_ref, int64_t *i64_out,
                              double *f64_out)
{
    const double t2 = oracle_eq3_timer(lam, b2, b3, (double)c2, w_ref);
    const double tstar = b3 / a1;
    const double timers[2] = {t2, INFINITY};
    int64_t restored[2] = {0, 0}, admitted[2] = {0, 0}, total = 0, n_short = 0;
    for (int64_t r = 0; r < n_reps; ++r) {
        const double *A = arrival_s + r * n, *W = wait_s + r * n;
        const int32_t *C = ctx ? ctx + r * n : NULL;
        for (int k = 0; k < 2; ++k) {
            int64_t rest = 0, adm = 0;
            oracle_capacity_replay(A, W, C, n, c2, timers[k], b2, b3, &rest, &adm);
            restored[k] += rest;
            admitted[k] += adm;
        }
        for (int64_t i = 0; i < n; ++i) {
            total += C ? (int64_t)C[i] : 1;
            if (W[i] <= tstar) n_short += 1;
        }
    }
    const int64_t requests = n_reps * n;
    double cost[2];
    for (int k = 0; k < 2; ++k)
        cost[k] = b2 * (double)restored[k] + b3 * (double)(total - restored[k]);
    i64_out[0] = (cost[0] < cost[1]) ? 1 : 0;
    i64_out[1] = restored[0];
    i64_out[2] = restored[1];
    i64_out[3] = admitted[0];
    i64_out[4] = admitted[1];
    i64_out[5] = total;
    i64_out[6] = n_short;
    i64_out[7] = requests;
    f64_out[0] = t2;
    f64_out[1] = cost[0];
    f64_out[2] = cost[1];
    f64_out[3] = cost[0] / (double)requests;
    f64_out[4] = cost[1] / (double)requests;
    f64_out[5] = tstar;
    f64_out[6] = (double)n_short / (double)requests;
}

/* The crossover statistic of Section 4.3 / Figure 4(d) on a bare wait sample:
 * the number of waits at or below t* = beta_3 / alpha_1. */
int64_t oracle_crossover_count(const double *wait_s, int64_t n, double a1, double b3)
{
    const double t_star = b3 / a1;
    int64_t c = 0;
    for (int64_t i = 0; i < n; ++i)
        if (wait_s[i] <= t_star) c += 1;
    return c;
}
