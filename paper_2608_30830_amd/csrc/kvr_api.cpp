// C ABI of the calibration-replay library: validation on the host, derivation
// of the load-dependent prices (Eq. 3), workspace planning and launches.
// Built as a plain host translation unit (IEEE semantics for every check).
#include "kvr.h"
#include "kvr_factored.h"
#include "kvr_internal.h"

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <limits>
#include <vector>

namespace {

using kvr::GridPlan;
using kvr::PriceDev;
using kvr::SampleSrc;
using kvr::Tables;

constexpr int64_t kMaxPolicies = int64_t(1) << 24;
constexpr int32_t kMaxLoads = 4096;
constexpr int64_t kMaxBatch = int64_t(1) << 40;
constexpr size_t kStatusBytes = 256;
size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Sample splits per resample for the grid kernel (measured on MI355X: 1,024
// SIMDs, 4 resident grid waves each).  With at least 32K waves already there
// is no split (the selection is fused into the grid kernel).  Otherwise the
// samples are cut into splits of >= 2,048 samples, or of >= 512 samples when
// that is what it takes to give every resident slot a wave; never more than
// 16 rounds of waves, and never more than part_cap bytes (1 GiB unless the
// caller's workspace is bounded) of split partials.
constexpr int64_t kPartCapBytes = int64_t(1) << 30;
int64_t choose_splits(int64_t base_waves, int64_t m, int64_t partial_doubles_per_split,
                      int64_t part_cap)
{
    constexpr int64_t kSlots = 4096, kFull = 32768, kMaxRounds = 16;
    if (base_waves >= kFull) return 1;
    int64_t ns = std::max<int64_t>(1, m / 2048);
    if (base_waves * ns < kSlots)
        ns = std::max<int64_t>(1, std::min<int64_t>(m / 512, cdiv(kSlots, base_waves)));
    ns = std::min<int64_t>(ns, cdiv(kMaxRounds * kSlots, base_waves));
    const int64_t mem_cap = std::max<int64_t>(1, part_cap / 8 / partial_doubles_per_split);
    return std::max<int64_t>(1, std::min<int64_t>(ns, mem_cap));
}

bool pos_finite(double x) { return std::isfinite(x) && x > 0.0; }

int check_prices(const kvr_prices *p)
{
    if (!p) return KVR_E_NULL;
    if (!pos_finite(p->a1_per_token) || !pos_finite(p->b2_per_token) ||
        !pos_finite(p->b3_per_token) || !pos_finite(p->host_slots_c2) || !pos_finite(p->w_ref_s))
        return KVR_E_PRICE;
    if (!std::isfinite(p->offload_per_token) || p->offload_per_token < 0.0) return KVR_E_PRICE;
    return KVR_OK;
}

// Prices of the grid kernels.  The optional offload charge is paid once by
// every request with w > t1, which are exactly the requests that pay b2 (host
// copy restored) or b3 (discarded, recomputed), so it is added to both; the
// congestion price a2 keeps the plain b3 of Eq. 3.
PriceDev device_prices(const kvr_prices *p)
{
    return PriceDev{p->a1_per_token, p->b2_per_token + p->offload_per_token,
                    p->b3_per_token + p->offload_per_token};
}

int check_grid(const kvr_policy_grid *g)
{
    if (!g) return KVR_E_NULL;
    if (!g->t1 || !g->t2 || !g->lam) return KVR_E_NULL;
    if (g->n_t1 < 1 || g->n_t2 < 1 || g->n_lam < 1 || g->n_lam > kMaxLoads) return KVR_E_SIZE;
    if ((int64_t)g->n_t1 * g->n_t2 > kMaxPolicies) return KVR_E_SIZE;
    for (int32_t a = 0; a < g->n_t1; ++a) {
        const double v = g->t1[a];
        if (!std::isfinite(v) || v < 0.0) return KVR_E_GRID;
        if (a > 0 && !(v > g->t1[a - 1])) return KVR_E_GRID;
    }
    for (int32_t k = 0; k < g->n_t2; ++k) {
        const double v = g->t2[k];
        if (std::isnan(v) || !(v > 0.0)) return KVR_E_GRID;
        if (std::isinf(v) && k != g->n_t2 - 1) return KVR_E_GRID;
        if (k > 0 && !(v > g->t2[k - 1])) return KVR_E_GRID;
    }
    for (int32_t l = 0; l < g->n_lam; ++l) {
        const double v = g->lam[l];
        if (!std::isfinite(v) || v < 0.0) return KVR_E_GRID;
    }
    return KVR_OK;
}

// Eq. 3 per token: lambda_crit = C2 / W_ref, a2 = max(0, lambda - lambda_crit) * b3 / C2.
void congestion_prices(const kvr_prices &p, const kvr_policy_grid &g, int32_t Lpad,
                       std::vector<double> &a2)
{
    const double lc = p.host_slots_c2 / p.w_ref_s;
    a2.assign((size_t)Lpad, 0.0);
    for (int32_t l = 0; l < g.n_lam; ++l) {
        double d = g.lam[l] - lc;
        if (!(d > 0.0)) d = 0.0;
        a2[(size_t)l] = (d * p.b3_per_token) / p.host_slots_c2;
    }
}

struct BrutePlan {
    GridPlan gp;
    int32_t Lpad;
    bool fused;              // nsplit == 1: costs finalised inside the grid kernel
    // workspace offsets
    size_t off_t1, off_t2, off_a2, off_X, off_G, off_xgp, off_cand, off_part, off_cost, total;
    size_t off_rec, off_lb, off_S;
    int64_t r3_bins;         // finite grid deadlines (bins kept per resample)
    int r3_nsplit;
    int64_t r3_split_len;
    int64_t max_blocks;      // largest launch grid of the plan
};

int choose_tile(int32_t L)
{
    const int cands[4] = {4, 8, 16, 32};
    int best = 32;
    int64_t best_cost = std::numeric_limits<int64_t>::max();
    for (int c : cands) {
        // issue slots per sample: ~5 per tile (forming h, the staged reads, the
        // loop) plus one FMA per load
        const int64_t cost = cdiv(L, c) * (c + 5);
        if (cost < best_cost) {
            best_cost = cost;
            best = c;
        }
    }
    return best;
}

BrutePlan plan_brute(int64_t R, int64_t n, int64_t m, const kvr_policy_grid &g, bool bootstrap,
                     bool want_cost, int64_t part_cap = kPartCapBytes)
{
    const int32_t K1 = g.n_t1, K2 = g.n_t2, L = g.n_lam;
    BrutePlan bp{};
    GridPlan &gp = bp.gp;
    const int64_t P = (int64_t)K1 * K2;
    gp.LT = choose_tile(L);
    gp.ntiles = (int)cdiv(L, gp.LT);
    gp.nblk = (int)cdiv(P, kvr::kWave);
    gp.R = R;
    bp.Lpad = gp.ntiles * gp.LT;
    // a group of 64 lanes spans at most two t1 rows only when K2 >= 64; it never
    // straddles a resample when P is a multiple of 64 or there is one resample
    if (K2 < kvr::kWave) gp.mode = kvr::kModePerLane;
    else if (P % kvr::kWave == 0 || R == 1) gp.mode = kvr::kModeRows1;
    else gp.mode = kvr::kModeRows2;
    gp.ngroups = (gp.mode == kvr::kModePerLane) ? R * gp.nblk : cdiv(R * P, kvr::kWave);
    const int64_t base_waves = gp.ngroups * gp.ntiles;
    const int64_t target = choose_splits(base_waves, m, R * gp.ntiles * gp.LT * P, part_cap);
    const int64_t split_len = cdiv(cdiv(m, target), kvr::kChunk) * kvr::kChunk;
    const int64_t nsplit = cdiv(m, split_len);
    gp.nsplit = (int)nsplit;
    gp.split_len = split_len;
    gp.wpb = 1;
    bp.fused = (nsplit == 1);

    size_t off = kStatusBytes;
    auto take = [&](size_t bytes) {
        size_t o = off;
        off += align256(bytes);
        return o;
    };
    bp.off_t1 = take(sizeof(double) * K1);
    bp.off_t2 = take(sizeof(double) * K2);
    bp.off_a2 = take(sizeof(double) * bp.Lpad);
    bp.off_X = take(sizeof(double) * R * K1);
    bp.off_G = take(sizeof(double) * R * K1);
    int64_t part_len = 0;
    const int parts = kvr::xg_parts(R, K1, m, &part_len);
    bp.off_xgp = take(sizeof(double) * 2 * parts * R * K1);
    // recompute-share bins: same IEEE sums as the device's deadlines
    bp.r3_bins = 0;
    for (int32_t a = 0; a < K1; ++a)
        for (int32_t k = 0; k < K2; ++k)
            if (std::isfinite((g.t1[a] + 0.0) + g.t2[k])) ++bp.r3_bins;
    bp.r3_nsplit = kvr::r3_splits(R, m, &bp.r3_split_len);
    bp.off_rec = take(sizeof(kvr::SampleRec) * n);
    bp.off_lb = take(sizeof(int32_t) * P);
    bp.off_S = take(sizeof(uint64_t) * R * bp.r3_bins);
    bp.off_cand = bp.off_part = bp.off_cost = 0;
    if (bp.fused) {
        if (bootstrap) bp.off_cand = take(sizeof(kvr::ArgminCand) * gp.ngroups * 2 * L);
    } else {
        bp.off_part = take(sizeof(double) * nsplit * R * gp.ntiles * gp.LT * P);
        if (bootstrap && !want_cost) bp.off_cost = take(sizeof(double) * R * L * P);
    }
    bp.total = off;
    // the largest launch grid of the plan, in blocks (every launch takes a
    // 32-bit grid; the callers' bounds keep these products inside int64)
    const int64_t rows = R * gp.ntiles * gp.LT;
    const int64_t grids[] = {gp.ngroups * gp.nsplit * gp.ntiles,
                             R * cdiv(K1, 8) * parts,
                             cdiv(R * K1, 256),
                             cdiv(R * bp.r3_bins, 256),
                             R * bp.r3_nsplit,
                             cdiv(rows * P, 256),
                             cdiv(R * gp.ntiles * P, 256),
                             cdiv(R * L, 4),
                             R * L};
    bp.max_blocks = 0;
    for (int64_t v : grids) bp.max_blocks = std::max(bp.max_blocks, v);
    return bp;
}

template <typename T> T *at(void *ws, size_t off) { return reinterpret_cast<T *>(static_cast<char *>(ws) + off); }

kvr::R3Ws r3_view(void *ws, const BrutePlan &bp)
{
    kvr::R3Ws v{};
    v.rec = at<kvr::SampleRec>(ws, bp.off_rec);
    v.lb = at<int32_t>(ws, bp.off_lb);
    v.S = at<unsigned long long>(ws, bp.off_S);
    v.nbins = bp.r3_bins;
    v.nsplit = bp.r3_nsplit;
    v.split_len = bp.r3_split_len;
    return v;
}

// Workspace of the one-launch brute force for one small sample
// (kvr::small_path_fits): after bp's tables, the pre-pass blocks' rows of the
// recompute histogram over the F finite deadlines, each policy's deadline
// bin, the per-block X/G partials, the histogram's suffix sums, X and G, the
// grid blocks' split partials (always written, even for one split) and the
// arrival counters.
struct SmallPlan {
    size_t off_hist, off_lb, off_xgp, off_S, off_XG, off_part, off_ctr, total;
    size_t part_bytes;
    int nctr;
};

bool small_plan_applies(const BrutePlan &bp, const kvr_policy_grid &g, int64_t n)
{
    return kvr::small_path_fits(g.n_t1, g.n_t2, bp.r3_bins, n) &&
           bp.gp.ngroups * bp.gp.ntiles <= kvr::kSmallMaxGroupTiles;
}

// Splits of the small-sample path: blocks of kSmallWaves waves add their
// splits in LDS, so splits can be as short as one staged chunk; about 4,096
// waves (four per SIMD) in all.
void small_splits(BrutePlan &bp, int64_t m, int64_t part_cap)
{
    kvr::GridPlan &gp = bp.gp;
    const int64_t base_waves = gp.ngroups * gp.ntiles;
    int64_t ns = std::max<int64_t>(1, std::min<int64_t>(4096 / base_waves, cdiv(m, kvr::kChunk)));
    const int64_t per_group = gp.ntiles * gp.LT * (int64_t)gp.nblk * kvr::kWave;   // doubles per split group
    const int64_t cap_groups = std::max<int64_t>(1, part_cap / 8 / std::max<int64_t>(1, per_group));
    ns = std::min<int64_t>(ns, cap_groups * kvr::kSmallWaves);
    gp.split_len = cdiv(cdiv(m, ns), kvr::kChunk) * kvr::kChunk;
    gp.nsplit = (int)cdiv(m, gp.split_len);
    gp.wpb = kvr::kSmallWaves;
    bp.fused = false;
}

SmallPlan plan_small(const BrutePlan &bp, int64_t n, const kvr_policy_grid &g)
{
    SmallPlan sp{};
    const int64_t P = (int64_t)g.n_t1 * g.n_t2;
    size_t off = bp.off_a2 + align256(sizeof(double) * bp.Lpad);
    auto take = [&](size_t bytes) {
        size_t o = off;
        off += align256(bytes);
        return o;
    };
    sp.off_hist = take(sizeof(uint64_t) * std::max<int64_t>(1, bp.r3_bins) *
                       kvr::small_sample_blocks(n));
    sp.off_lb = take(sizeof(int32_t) * P);
    sp.off_xgp = take(sizeof(double) * 2 * g.n_t1 * kvr::small_sample_blocks(n));
    sp.off_S = take(sizeof(uint64_t) * std::max<int64_t>(1, bp.r3_bins));
    sp.off_XG = take(sizeof(double) * 2 * g.n_t1);
    const int64_t nbatch = cdiv(cdiv(bp.gp.nsplit, bp.gp.wpb), kvr::kSmallBatchGroups);
    sp.nctr = (int)(1 + bp.gp.ngroups * bp.gp.ntiles * (1 + nbatch));
    sp.off_ctr = take(sizeof(unsigned) * sp.nctr);
    const int64_t nsg = cdiv(bp.gp.nsplit, bp.gp.wpb);
    sp.part_bytes = sizeof(double) * (size_t)nsg * bp.gp.ntiles * bp.gp.LT * P;
    sp.off_part = take(sp.part_bytes);   // last: the part a workspace bound trims
    sp.total = off;
    return sp;
}

int hip_ok(hipError_t e) { return e == hipSuccess ? KVR_OK : KVR_E_HIP; }

#define KVR_TRY(expr)                       \
    do {                                    \
        int rc_ = hip_ok(expr);             \
        if (rc_ != KVR_OK) return rc_;      \
    } while (0)

// Uploads t1, t2 (canonical zeros) and the padded a2 table and clears the status
// word and zero[0..nzero) (one launch when the tables are small).
int stage_tables(void *ws, size_t off_t1, size_t off_t2, size_t off_a2, int32_t Lpad,
                 const kvr_prices &p, const kvr_policy_grid &g, hipStream_t s, Tables &tb,
                 unsigned *zero = nullptr, int nzero = 0)
{
    std::vector<double> t1(g.t1, g.t1 + g.n_t1), t2(g.t2, g.t2 + g.n_t2), a2;
    for (double &v : t1) v = v + 0.0;
    congestion_prices(p, g, Lpad, a2);
    double *const dst[3] = {at<double>(ws, off_t1), at<double>(ws, off_t2), at<double>(ws, off_a2)};
    const double *const src[3] = {t1.data(), t2.data(), a2.data()};
    const int64_t cnt[3] = {g.n_t1, g.n_t2, Lpad};
    KVR_TRY(kvr::launch_stage(static_cast<int *>(ws), dst, src, cnt, zero, nzero, s));
    tb.t1 = at<double>(ws, off_t1);
    tb.t2 = at<double>(ws, off_t2);
    tb.a2 = at<double>(ws, off_a2);
    tb.K1 = g.n_t1;
    tb.K2 = g.n_t2;
    tb.L = g.n_lam;
    tb.Lpad = Lpad;
    return KVR_OK;
}

// Optional profiling events of the calling host thread (kvr_set_profile_events).
thread_local hipEvent_t g_prof_begin = nullptr;
thread_local hipEvent_t g_prof_end = nullptr;

int prof_mark(hipEvent_t ev, hipStream_t s)
{
    if (ev == nullptr) return KVR_OK;
    return hipEventRecord(ev, s) == hipSuccess ? KVR_OK : KVR_E_HIP;
}

#define KVR_MARK(ev, s)                          \
    do {                                         \
        int rc_ = prof_mark((ev), (s));          \
        if (rc_ != KVR_OK) return rc_;           \
    } while (0)

int check_workspace(void *d_ws, size_t have, size_t need)
{
    if (have < need) return KVR_E_WORKSPACE;
    if ((reinterpret_cast<uintptr_t>(d_ws) & 255u) != 0) return KVR_E_WORKSPACE;
    return KVR_OK;
}

}  // namespace

extern "C" {

int kvr_prices_from_platform(double kv_bytes_per_token, double hbm_usable_bytes,
                             double host_link_bytes_per_s, double prefill_tokens_per_s,
                             double n_gpu, double host_slots_c2, double w_ref_s, kvr_prices *out)
{
    if (!out) return KVR_E_NULL;
    if (!pos_finite(kv_bytes_per_token) || !pos_finite(hbm_usable_bytes) ||
        !pos_finite(host_link_bytes_per_s) || !pos_finite(prefill_tokens_per_s) ||
        !pos_finite(n_gpu) || !pos_finite(host_slots_c2) || !pos_finite(w_ref_s))
        return KVR_E_PRICE;
    out->a1_per_token = n_gpu * kv_bytes_per_token / hbm_usable_bytes;
    out->b2_per_token = n_gpu * kv_bytes_per_token / host_link_bytes_per_s;
    out->b3_per_token = n_gpu / prefill_tokens_per_s;
    out->host_slots_c2 = host_slots_c2;
    out->w_ref_s = w_ref_s;
    out->offload_per_token = 0.0;
    return KVR_OK;
}

}  // extern "C"

// kvr_cost_grid with an optional bound on the workspace: with fit_bytes > 0
// the brute-force plan takes fewer sample splits when its split partials would
// otherwise push the workspace beyond fit_bytes (same result up to the order
// in which the splits are summed).
int kvr::cost_grid_entry(const double *d_wait_s, const int32_t *d_ctx_tokens, int64_t n,
                         const kvr_prices *p, const kvr_policy_grid *g, int32_t method,
                         double *d_cost, int32_t *d_perm, void *d_ws, size_t *ws_bytes,
                         size_t fit_bytes, void *hip_stream)
{
    if (!ws_bytes) return KVR_E_NULL;
    int rc;
    if ((rc = check_prices(p)) != KVR_OK) return rc;
    if ((rc = check_grid(g)) != KVR_OK) return rc;
    if (method != KVR_BRUTE && method != KVR_SORTED) return KVR_E_METHOD;
    if (method == KVR_BRUTE && d_perm != nullptr) return KVR_E_METHOD;
    if (n < 1 || n > INT32_MAX) return KVR_E_SIZE;

    size_t need;
    BrutePlan bp{};
    SmallPlan sp{};
    bool small = false;
    size_t off_t1 = kStatusBytes, off_t2 = 0, off_a2 = 0, off_sort = 0;
    int32_t Lpad = g->n_lam;
    if (method == KVR_BRUTE) {
        bp = plan_brute(1, n, n, *g, false, true);
        small = small_plan_applies(bp, *g, n);
        if (small) {
            small_splits(bp, n, kPartCapBytes);
            sp = plan_small(bp, n, *g);
        }
        need = small ? sp.total : bp.total;
        // the split partials are carved last: fewer splits when they alone
        // push the workspace past fit_bytes
        const size_t part = small ? sp.part_bytes : (bp.fused ? 0 : bp.total - bp.off_part);
        if (fit_bytes > 0 && need > fit_bytes && part > 0 && need - part < fit_bytes) {
            const int64_t cap = (int64_t)(fit_bytes - (need - part));
            bp = plan_brute(1, n, n, *g, false, true, cap);
            if (small) {
                small_splits(bp, n, cap);
                sp = plan_small(bp, n, *g);
            }
            need = small ? sp.total : bp.total;
        }
        if (bp.max_blocks > INT32_MAX) return KVR_E_SIZE;
    } else {
        off_t2 = off_t1 + align256(sizeof(double) * g->n_t1);
        off_a2 = off_t2 + align256(sizeof(double) * g->n_t2);
        off_sort = off_a2 + align256(sizeof(double) * Lpad);
        need = off_sort + kvr::sort_ws_bytes(n);
    }
    if (d_ws == nullptr) {
        *ws_bytes = need;
        return KVR_OK;
    }
    if (!d_wait_s || !d_ctx_tokens || !d_cost) return KVR_E_NULL;
    if ((rc = check_workspace(d_ws, *ws_bytes, need)) != KVR_OK) return rc;

    hipStream_t s = static_cast<hipStream_t>(hip_stream);
    int *status = static_cast<int *>(d_ws);
    const PriceDev pr = device_prices(p);
    Tables tb{};
    if (method == KVR_BRUTE && small) {
        kvr::SmallWs sw{};
        sw.hist = at<unsigned long long>(d_ws, sp.off_hist);
        sw.lb = at<int32_t>(d_ws, sp.off_lb);
        sw.xgp = at<double>(d_ws, sp.off_xgp);
        sw.S = at<unsigned long long>(d_ws, sp.off_S);
        sw.XG = at<double>(d_ws, sp.off_XG);
        sw.partials = at<double>(d_ws, sp.off_part);
        sw.ctr = at<unsigned>(d_ws, sp.off_ctr);
        sw.nbins = bp.r3_bins;
        sw.nsb = kvr::small_sample_blocks(n);
        sw.npb = kvr::small_policy_blocks((int64_t)g->n_t1 * g->n_t2);
        if ((rc = stage_tables(d_ws, bp.off_t1, bp.off_t2, bp.off_a2, bp.Lpad, *p, *g, s, tb, sw.ctr,
                               sp.nctr)) != KVR_OK)
            return rc;
        SampleSrc src{d_wait_s, d_ctx_tokens, nullptr, n, n};
        KVR_MARK(g_prof_begin, s);
        KVR_TRY(kvr::launch_small(src, tb, pr, bp.gp, sw, d_cost, status, s));
        KVR_MARK(g_prof_end, s);
        return KVR_OK;
    }
    if (method == KVR_BRUTE) {
        if ((rc = stage_tables(d_ws, bp.off_t1, bp.off_t2, bp.off_a2, bp.Lpad, *p, *g, s, tb)) != KVR_OK)
            return rc;
        SampleSrc src{d_wait_s, d_ctx_tokens, nullptr, n, n};
        double *X = at<double>(d_ws, bp.off_X), *G = at<double>(d_ws, bp.off_G);
        const kvr::R3Ws r3 = r3_view(d_ws, bp);
        const bool fuse = kvr::r3_fuses_xg(g->n_t1, r3.nsplit, r3.nbins);
        KVR_TRY(kvr::launch_r3(src, 1, tb, r3, fuse ? X : nullptr, fuse ? G : nullptr, status, s));
        if (!fuse)
            KVR_TRY(kvr::launch_xg(src, 1, tb, X, G, at<double>(d_ws, bp.off_xgp), r3.rec, status, s));
        double *part = bp.fused ? nullptr : at<double>(d_ws, bp.off_part);
        KVR_MARK(g_prof_begin, s);
        KVR_TRY(kvr::launch_grid(src, tb, pr, bp.gp, X, G, r3, bp.fused ? d_cost : nullptr,
                                 nullptr, part, status, s));
        KVR_MARK(g_prof_end, s);
        if (!bp.fused)
            KVR_TRY(kvr::launch_reduce_partials(bp.gp, tb, pr, n, X, G, r3, part, d_cost, s));
        return KVR_OK;
    }
    if ((rc = stage_tables(d_ws, off_t1, off_t2, off_a2, Lpad, *p, *g, s, tb)) != KVR_OK) return rc;
    kvr::SortWs sws{};
    kvr::sort_ws_carve(at<char>(d_ws, off_sort), n, sws);
    KVR_MARK(g_prof_begin, s);
    KVR_TRY(kvr::launch_sorted_path(d_wait_s, d_ctx_tokens, n, tb, pr, sws, d_cost, d_perm, status, s));
    KVR_MARK(g_prof_end, s);
    return KVR_OK;
}

extern "C" {

int kvr_cost_grid(const double *d_wait_s, const int32_t *d_ctx_tokens, int64_t n,
                  const kvr_prices *p, const kvr_policy_grid *g, int32_t method, double *d_cost,
                  int32_t *d_perm, void *d_ws, size_t *ws_bytes, void *hip_stream)
{
    return kvr::cost_grid_entry(d_wait_s, d_ctx_tokens, n, p, g, method, d_cost, d_perm, d_ws,
                                ws_bytes, 0, hip_stream);
}

int kvr_select_policy(const double *d_cost, int64_t batch, int32_t n_lam, int32_t n_t1,
                      int32_t n_t2, int32_t last_t2_is_inf, int32_t *d_best, double *d_best_cost,
                      int32_t *d_branch, void *hip_stream)
{
    if (!d_cost || !d_best || !d_best_cost) return KVR_E_NULL;
    if (batch < 1 || n_lam < 1 || n_t1 < 1 || n_t2 < 1 || n_lam > kMaxLoads) return KVR_E_SIZE;
    if ((int64_t)n_t1 * n_t2 > kMaxPolicies) return KVR_E_SIZE;
    if (batch > INT32_MAX / n_lam) return KVR_E_SIZE;
    if (last_t2_is_inf != 0 && last_t2_is_inf != 1) return KVR_E_GRID;
    KVR_TRY(kvr::launch_select(d_cost, batch, n_lam, (int64_t)n_t1 * n_t2, n_t2, last_t2_is_inf,
                               d_best, d_best_cost, d_branch, static_cast<hipStream_t>(hip_stream)));
    return KVR_OK;
}

int kvr_bootstrap(const double *d_wait_s, const int32_t *d_ctx_tokens, int64_t n,
                  const int32_t *d_idx, int64_t n_resamples, int64_t m, const kvr_prices *p,
                  const kvr_policy_grid *g, int32_t *d_best, double *d_best_cost, double *d_cost,
                  void *d_ws, size_t *ws_bytes, void *hip_stream)
{
    if (!ws_bytes) return KVR_E_NULL;
    int rc;
    if ((rc = check_prices(p)) != KVR_OK) return rc;
    if ((rc = check_grid(g)) != KVR_OK) return rc;
    if (n < 1 || n > INT32_MAX || n_resamples < 1 || m < 1 || m > INT32_MAX) return KVR_E_SIZE;
    if (n_resamples > kMaxBatch / m) return KVR_E_SIZE;
    if (n_resamples * g->n_lam > INT32_MAX) return KVR_E_SIZE;
    const bool want_cost = d_cost != nullptr;
    BrutePlan bp = plan_brute(n_resamples, n, m, *g, true, want_cost);
    if (bp.max_blocks > INT32_MAX) return KVR_E_SIZE;
    if (d_ws == nullptr) {
        *ws_bytes = bp.total;
        return KVR_OK;
    }
    if (!d_wait_s || !d_ctx_tokens || !d_idx || !d_best || !d_best_cost) return KVR_E_NULL;
    if ((rc = check_workspace(d_ws, *ws_bytes, bp.total)) != KVR_OK) return rc;

    hipStream_t s = static_cast<hipStream_t>(hip_stream);
    int *status = static_cast<int *>(d_ws);
    const PriceDev pr = device_prices(p);
    Tables tb{};
    if ((rc = stage_tables(d_ws, bp.off_t1, bp.off_t2, bp.off_a2, bp.Lpad, *p, *g, s, tb)) != KVR_OK)
        return rc;
    SampleSrc src{d_wait_s, d_ctx_tokens, d_idx, n, m};
    double *X = at<double>(d_ws, bp.off_X), *G = at<double>(d_ws, bp.off_G);
    const kvr::R3Ws r3 = r3_view(d_ws, bp);
    const bool fuse = kvr::r3_fuses_xg(g->n_t1, r3.nsplit, r3.nbins);
    KVR_TRY(kvr::launch_r3(src, n_resamples, tb, r3, fuse ? X : nullptr, fuse ? G : nullptr, status,
                           s));
    if (!fuse)
        KVR_TRY(kvr::launch_xg(src, n_resamples, tb, X, G, at<double>(d_ws, bp.off_xgp), r3.rec,
                               status, s));
    const int64_t P = (int64_t)g->n_t1 * g->n_t2;
    if (bp.fused) {
        kvr::ArgminCand *cand = at<kvr::ArgminCand>(d_ws, bp.off_cand);
        KVR_MARK(g_prof_begin, s);
        KVR_TRY(kvr::launch_grid(src, tb, pr, bp.gp, X, G, r3, d_cost, cand, nullptr, status, s));
        KVR_MARK(g_prof_end, s);
        KVR_TRY(kvr::launch_reduce_cands(cand, bp.gp, P, g->n_lam, d_best, d_best_cost, s));
        return KVR_OK;
    }
    double *part = at<double>(d_ws, bp.off_part);
    double *cost = want_cost ? d_cost : at<double>(d_ws, bp.off_cost);
    KVR_MARK(g_prof_begin, s);
    KVR_TRY(kvr::launch_grid(src, tb, pr, bp.gp, X, G, r3, nullptr, nullptr, part, status, s));
    KVR_MARK(g_prof_end, s);
    KVR_TRY(kvr::launch_reduce_partials(bp.gp, tb, pr, m, X, G, r3, part, cost, s));
    KVR_TRY(kvr::launch_select(cost, n_resamples, g->n_lam, P, g->n_t2, 0, d_best, d_best_cost,
                               nullptr, s));
    return KVR_OK;
}

int kvr_bootstrap_factored(const double *d_wait_s, const int32_t *d_ctx_tokens, int64_t n,
                           const int32_t *d_idx, int64_t n_resamples, int64_t m,
                           const kvr_prices *p, const kvr_policy_grid *g, int32_t *d_best,
                           double *d_best_cost, double *d_cost, void *d_ws, size_t *ws_bytes,
                           void *hip_stream)
{
    if (!ws_bytes) return KVR_E_NULL;
    int rc;
    if ((rc = check_prices(p)) != KVR_OK) return rc;
    if ((rc = check_grid(g)) != KVR_OK) return rc;
    if (n < 1 || n > INT32_MAX - 1 || n_resamples < 1 || m < 1 || m > INT32_MAX) return KVR_E_SIZE;
    if (n_resamples > kMaxBatch / m) return KVR_E_SIZE;
    if (n_resamples * g->n_lam > INT32_MAX) return KVR_E_SIZE;
    const int64_t P = (int64_t)g->n_t1 * g->n_t2;
    const int32_t Lpad = (int32_t)(cdiv(g->n_lam, 32) * 32);
    const int64_t nqs = kvr::factored_query_slots(n, g->n_t1, P);
    const int64_t Rb = kvr::factored_batch(nqs, n_resamples);
    size_t off = kStatusBytes;
    auto take = [&](size_t bytes) {
        size_t o = off;
        off += align256(bytes);
        return o;
    };
    const size_t off_t1 = take(sizeof(double) * g->n_t1);
    const size_t off_t2 = take(sizeof(double) * g->n_t2);
    const size_t off_a2 = take(sizeof(double) * Lpad);
    const size_t off_sort = take(kvr::sort_ws_bytes(n));
    const size_t off_rank = take(sizeof(int32_t) * n);
    const size_t off_Ts = take(sizeof(int32_t) * n);
    const size_t off_sw = take(sizeof(double) * n);
    const size_t off_u1 = take(sizeof(int32_t) * g->n_t1);
    const size_t off_ue = take(sizeof(int32_t) * P);
    const size_t off_qslot = take(sizeof(int32_t) * (n + 1));
    const size_t off_qbits = take(sizeof(uint32_t) * ((n + 32) / 32));
    const size_t off_qbase = take(sizeof(int32_t) * ((n + 32) / 32));
    const size_t off_TQ = take(sizeof(double) * 2 * Rb * nqs);
    const size_t off_tot = take(sizeof(uint64_t) * Rb);
    const size_t need = off;
    if (d_ws == nullptr) {
        *ws_bytes = need;
        return KVR_OK;
    }
    if (!d_wait_s || !d_ctx_tokens || !d_idx || !d_best || !d_best_cost) return KVR_E_NULL;
    if ((rc = check_workspace(d_ws, *ws_bytes, need)) != KVR_OK) return rc;

    hipStream_t s = static_cast<hipStream_t>(hip_stream);
    int *status = static_cast<int *>(d_ws);
    const PriceDev pr = device_prices(p);
    Tables tb{};
    if ((rc = stage_tables(d_ws, off_t1, off_t2, off_a2, Lpad, *p, *g, s, tb)) != KVR_OK) return rc;
    kvr::FactoredWs fw{};
    kvr::sort_ws_carve(at<char>(d_ws, off_sort), n, fw.sort);
    fw.rank = at<int32_t>(d_ws, off_rank);
    fw.Ts = at<int32_t>(d_ws, off_Ts);
    fw.sw = at<double>(d_ws, off_sw);
    fw.u1 = at<int32_t>(d_ws, off_u1);
    fw.ue = at<int32_t>(d_ws, off_ue);
    fw.qslot = at<int32_t>(d_ws, off_qslot);
    fw.qbits = at<uint32_t>(d_ws, off_qbits);
    fw.qbase = at<int32_t>(d_ws, off_qbase);
    fw.nqs = nqs;
    fw.TQ = at<double2>(d_ws, off_TQ);
    fw.tot = at<unsigned long long>(d_ws, off_tot);
    fw.Rb = Rb;
    SampleSrc src{d_wait_s, d_ctx_tokens, d_idx, n, m};
    KVR_MARK(g_prof_begin, s);
    KVR_TRY(kvr::launch_factored(src, n_resamples, tb, pr, fw, d_best, d_best_cost, d_cost, status,
                                 s));
    KVR_MARK(g_prof_end, s);
    return KVR_OK;
}

int kvr_eq3_timer(const kvr_prices *p, double lambda, double *t2_out)
{
    if (!t2_out) return KVR_E_NULL;
    int rc;
    if ((rc = check_prices(p)) != KVR_OK) return rc;
    if (!std::isfinite(lambda) || lambda < 0.0) return KVR_E_GRID;
    const double lc = p->host_slots_c2 / p->w_ref_s;
    double d = lambda - lc;
    if (!(d > 0.0)) d = 0.0;
    const double a2 = (d * p->b3_per_token) / p->host_slots_c2;
    *t2_out = (a2 > 0.0) ? (p->b3_per_token - p->b2_per_token) / a2
                         : std::numeric_limits<double>::infinity();
    return KVR_OK;
}

int kvr_capacity_replay(const double *d_arrival_s, const double *d_wait_s,
                        const int32_t *d_ctx_tokens, int64_t n_reps, int64_t n,
                        const kvr_prices *p, const double *t2, int32_t n_t2, double *d_cost,
                        int64_t *d_restored_tokens, int64_t *d_admitted, void *d_ws,
                        size_t *ws_bytes, void *hip_stream)
{
    if (!ws_bytes || !t2) return KVR_E_NULL;
    int rc;
    if ((rc = check_prices(p)) != KVR_OK) return rc;
    if (p->offload_per_token != 0.0) return KVR_E_METHOD;   // no offload charge in the replay
    const double c2d = p->host_slots_c2;
    if (!(c2d >= 1.0) || c2d != std::floor(c2d) || c2d > 9.0e15) return KVR_E_PRICE;
    if (n_reps < 1 || n < 1 || n > 8192 || n_t2 < 1 || n_t2 > kMaxLoads) return KVR_E_SIZE;
    if (n_reps > INT32_MAX / n_t2) return KVR_E_SIZE;
    for (int32_t k = 0; k < n_t2; ++k)
        if (std::isnan(t2[k]) || !(t2[k] > 0.0)) return KVR_E_GRID;
    const size_t need = kStatusBytes + kvr::replay_ws_bytes(n_reps, n, n_t2);
    if (d_ws == nullptr) {
        *ws_bytes = need;
        return KVR_OK;
    }
    if (!d_arrival_s || !d_wait_s || !d_cost) return KVR_E_NULL;
    if ((rc = check_workspace(d_ws, *ws_bytes, need)) != KVR_OK) return rc;
    hipStream_t s = static_cast<hipStream_t>(hip_stream);
    int *status = static_cast<int *>(d_ws);
    KVR_TRY(kvr::launch_clear_status(status, s));
    KVR_MARK(g_prof_begin, s);
    KVR_TRY(kvr::launch_replay(d_arrival_s, d_wait_s, d_ctx_tokens, n_reps, n, t2, n_t2,
                               (int64_t)c2d, p->b2_per_token, p->b3_per_token,
                               at<char>(d_ws, kStatusBytes), d_cost, d_restored_tokens,
                               d_admitted, status, s));
    KVR_MARK(g_prof_end, s);
    return KVR_OK;
}

int kvr_controller_select(const double *d_arrival_s, const double *d_wait_s,
                          const int32_t *d_ctx_tokens, int64_t n_reps, int64_t n,
                          const kvr_prices *p, double lambda, kvr_controller_out *d_out,
                          void *d_ws, size_t *ws_bytes, void *hip_stream)
{
    if (!ws_bytes) return KVR_E_NULL;
    int rc;
    double t2 = 0.0;
    if ((rc = kvr_eq3_timer(p, lambda, &t2)) != KVR_OK) return rc;
    if (p->offload_per_token != 0.0) return KVR_E_METHOD;   // no offload charge in the replay
    const double c2d = p->host_slots_c2;
    if (!(c2d >= 1.0) || c2d != std::floor(c2d) || c2d > 9.0e15) return KVR_E_PRICE;
    if (n_reps < 1 || n < 1 || n > 8192 || n_reps > INT32_MAX / 2) return KVR_E_SIZE;
    const double t_star = p->b3_per_token / p->a1_per_token;
    const int64_t reps = n_reps;
    const size_t off_replay = kStatusBytes;
    const size_t off_cost = off_replay + align256(kvr::replay_ws_bytes(reps, n, 2));
    const size_t off_rest = off_cost + align256(sizeof(double) * 2 * (size_t)reps);
    const size_t off_adm = off_rest + align256(sizeof(int64_t) * 2 * (size_t)reps);
    const size_t off_cnt = off_adm + align256(sizeof(int64_t) * 2 * (size_t)reps);
    const size_t need = off_cnt + align256(kvr::count_ws_bytes());
    if (d_ws == nullptr) {
        *ws_bytes = need;
        return KVR_OK;
    }
    if (!d_arrival_s || !d_wait_s || !d_out) return KVR_E_NULL;
    if ((rc = check_workspace(d_ws, *ws_bytes, need)) != KVR_OK) return rc;
    hipStream_t s = static_cast<hipStream_t>(hip_stream);
    int *status = static_cast<int *>(d_ws);
    int64_t *rest = at<int64_t>(d_ws, off_rest), *adm = at<int64_t>(d_ws, off_adm);
    const double timers[2] = {t2, std::numeric_limits<double>::infinity()};
    KVR_TRY(kvr::launch_clear_status(status, s));
    KVR_MARK(g_prof_begin, s);
    KVR_TRY(kvr::launch_replay(d_arrival_s, d_wait_s, d_ctx_tokens, reps, n, timers, 2,
                               (int64_t)c2d, p->b2_per_token, p->b3_per_token,
                               at<char>(d_ws, off_replay), at<double>(d_ws, off_cost), rest, adm,
                               status, s));
    KVR_TRY(kvr::launch_short_count(d_wait_s, d_ctx_tokens, reps * n, t_star,
                                    at<char>(d_ws, off_cnt), status, s));
    KVR_TRY(kvr::launch_controller_final(rest, adm, reps, reps * n, at<char>(d_ws, off_cnt), t2,
                                         t_star, p->b2_per_token, p->b3_per_token, d_out, s));
    KVR_MARK(g_prof_end, s);
    return KVR_OK;
}

int kvr_crossover_statistic(const double *d_wait_s, int64_t n, const kvr_prices *p,
                            int64_t *d_count, double *d_fraction, void *d_ws, size_t *ws_bytes,
                            void *hip_stream)
{
    if (!ws_bytes) return KVR_E_NULL;
    int rc;
    if ((rc = check_prices(p)) != KVR_OK) return rc;
    if (n < 1 || n > kMaxBatch) return KVR_E_SIZE;
    const size_t need = kStatusBytes + align256(kvr::count_ws_bytes());
    if (d_ws == nullptr) {
        *ws_bytes = need;
        return KVR_OK;
    }
    if (!d_wait_s || !d_count) return KVR_E_NULL;
    if ((rc = check_workspace(d_ws, *ws_bytes, need)) != KVR_OK) return rc;
    hipStream_t s = static_cast<hipStream_t>(hip_stream);
    int *status = static_cast<int *>(d_ws);
    void *cnt = at<char>(d_ws, kStatusBytes);
    KVR_TRY(kvr::launch_clear_status(status, s));
    KVR_TRY(kvr::launch_short_count(d_wait_s, nullptr, n, p->b3_per_token / p->a1_per_token, cnt,
                                    status, s));
    KVR_TRY(kvr::launch_fraction(cnt, n, d_count, d_fraction, s));
    return KVR_OK;
}

int kvr_set_profile_events(void *ev_begin, void *ev_end)
{
    if ((ev_begin == nullptr) != (ev_end == nullptr)) return KVR_E_NULL;
    g_prof_begin = static_cast<hipEvent_t>(ev_begin);
    g_prof_end = static_cast<hipEvent_t>(ev_end);
    return KVR_OK;
}

int kvr_workspace_status(const void *d_ws, void *hip_stream)
{
    if (!d_ws) return KVR_E_NULL;
    hipStream_t s = static_cast<hipStream_t>(hip_stream);
    int word = 0;
    if (hipMemcpyAsync(&word, d_ws, sizeof(int), hipMemcpyDeviceToHost, s) != hipSuccess)
        return KVR_E_HIP;
    if (hipStreamSynchronize(s) != hipSuccess) return KVR_E_HIP;
    return word == 0 ? KVR_OK : KVR_E_DOMAIN;
}

const char *kvr_status_string(int status)
{
    switch (status) {
    case KVR_OK: return "ok";
    case KVR_E_NULL: return "a required pointer is NULL";
    case KVR_E_SIZE: return "a count is out of range or a product overflows";
    case KVR_E_GRID: return "invalid timer or load grid";
    case KVR_E_PRICE: return "a price, C2 or W_ref is not finite and positive";
    case KVR_E_WORKSPACE: return "workspace too small or not 256-byte aligned";
    case KVR_E_DOMAIN: return "bad sample or index detected on the device";
    case KVR_E_HIP: return "HIP runtime error";
    case KVR_E_METHOD: return "unknown method or option not supported by the method";
    default: return "unknown status";
    }
}

}  // extern "C"
