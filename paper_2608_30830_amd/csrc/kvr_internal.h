// Internal declarations shared by the library's HIP sources (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kvr.h"

namespace kvr {

constexpr int kWave = 64;          // CDNA wavefront width
constexpr int kChunk = 128;        // samples staged in LDS per buffer (grid kernel)
constexpr int kStatusDomain = 1;   // value of the workspace status word on a domain error
constexpr int kSmallWaves = 8;     // waves per block of the small-sample kernel
constexpr int kSmallMaxGroupTiles = 4096;   // (group, load tile)s of one small-sample launch
constexpr int kSmallBatchGroups = 8;        // split groups per batch in that launch

// Where a call's samples come from: the base arrays, optionally through
// bootstrap index rows idx[R][m].
struct SampleSrc {
    const double *w;     // [n] waits, seconds
    const int32_t *T;    // [n] context tokens
    const int32_t *idx;  // [R][m] or nullptr (then m == n, R == 1)
    int64_t n;
    int64_t m;
};

// Prices and derived scalars of one call.
struct PriceDev {
    double a1, b2, b3;
};

// Derived tables staged in the workspace.
struct Tables {
    const double *t1;    // [K1]
    const double *t2;    // [K2]
    const double *a2;    // [Lpad] per-token congestion prices, zero-padded
    int32_t K1, K2, L, Lpad;
};

// Grid-kernel modes (how 64-lane groups map onto policies and resamples).
enum { kModePerLane = 0, kModeRows1 = 1, kModeRows2 = 2 };

// Brute-force launch plan.
struct GridPlan {
    int LT;              // loads per tile (4, 8, 16 or 32)
    int ntiles;          // ceil(L / LT)
    int nblk;            // groups per resample, kModePerLane: ceil(K1*K2 / 64)
    int nsplit;          // sample splits per resample
    int wpb;             // splits per block: 1 (grid_kernel), or kSmallWaves (the
                         // small-sample kernel adds a block's splits in LDS)
    int mode;            // kModePerLane, kModeRows1 or kModeRows2
    int64_t ngroups;     // 64-lane groups: R*nblk (per lane) or ceil(R*K1*K2 / 64)
    int64_t split_len;   // samples per split (multiple of kChunk)
    int64_t R;           // resamples
};

// One wave's best policy for one (group, resample slot, load); laid out
// [ngroups][2][L], slot 1 used only by groups that straddle two resamples.
struct ArgminCand {
    double cost;
    int32_t f;
    int32_t pad;
};

// One base sample for the pre-passes over the draws: the number of grid
// deadlines below its wait, its context size (>= 1) and its wait (finite,
// >= 0; bad values replaced as fetch_sample replaces them).
struct SampleRec {
    int32_t bin;
    int32_t T;
    double w;
};

// Recompute share R3 per (resample, deadline), counted through deadline bins
// (kvr_r3.hip).  S[r][x] is R3 of every policy f with lb[f] == x; policies
// with lb[f] >= nbins (infinite deadlines) have R3 = 0.
struct R3Ws {
    SampleRec *rec;           // [n] per base sample: deadline bin, clamped context size and
                              // wait, cleaned as fetch_sample cleans them (one 16-byte gather)
    int32_t *lb;              // [K1*K2] grid deadlines strictly below each policy's
    unsigned long long *S;    // [R][nbins] suffix sums of T over bins 1..nbins
    int64_t nbins;            // F, the number of finite grid deadlines
    int nsplit;               // draw splits per resample
    int64_t split_len;
};

// kvr_cost_grid (same arguments, checks and results) with an optional bound on
// the workspace: fit_bytes > 0 makes the brute-force plan take fewer sample
// splits where its split partials would push the workspace beyond fit_bytes.
int cost_grid_entry(const double *d_wait_s, const int32_t *d_ctx_tokens, int64_t n,
                    const kvr_prices *p, const kvr_policy_grid *g, int32_t method,
                    double *d_cost, int32_t *d_perm, void *d_ws, size_t *ws_bytes,
                    size_t fit_bytes, void *hip_stream);

// ---- launches (all asynchronous on `stream`) --------------------------------
hipError_t launch_clear_status(int *status, hipStream_t stream);
// out[0] = KVR_OK or KVR_E_DOMAIN from a workspace status word.
hipError_t launch_export_status(const int *status, int32_t *out, hipStream_t stream);
hipError_t launch_upload(double *dst, const double *host_src, int64_t count, hipStream_t stream);
// Clears the status word and zero[0..nzero), and stores three host tables.
hipError_t launch_stage(int *status, double *const dst[3], const double *const src[3],
                        const int64_t cnt[3], unsigned *zero, int nzero, hipStream_t stream);

// X and G per (resample, t1); with few resamples the samples are cut into
// parts (partials in xgp[parts][R][K1][2], summed in part order).
int xg_parts(int64_t R, int K1, int64_t m, int64_t *part_len);
hipError_t launch_xg(const SampleSrc &src, int64_t R, const Tables &tb, double *X, double *G,
                     double *xgp, const SampleRec *rec, int *status, hipStream_t stream);

int r3_splits(int64_t R, int64_t m, int64_t *split_len);
// With X and G given (one t1 timer, one histogram block per resample: see
// r3_fuses_xg), the histogram pass also forms X and G, and xg_kernel is not
// needed.
bool r3_fuses_xg(int K1, int nsplit, int64_t nbins);
hipError_t launch_r3(const SampleSrc &src, int64_t R, const Tables &tb, const R3Ws &ws,
                     double *X, double *G, int *status, hipStream_t stream);

hipError_t launch_grid(const SampleSrc &src, const Tables &tb, const PriceDev &pr,
                       const GridPlan &plan, const double *X, const double *G, const R3Ws &r3,
                       double *cost_out, ArgminCand *cand, double *partials, int *status,
                       hipStream_t stream);

// Sums the split partials in place (split order) and writes mean costs.
hipError_t launch_reduce_partials(const GridPlan &plan, const Tables &tb, const PriceDev &pr,
                                  int64_t m, const double *X, const double *G, const R3Ws &r3,
                                  double *partials, double *cost_out, hipStream_t stream);

hipError_t launch_reduce_cands(const ArgminCand *cand, const GridPlan &plan, int64_t P, int L,
                               int32_t *best, double *best_cost, hipStream_t stream);

hipError_t launch_select(const double *cost, int64_t batch, int L, int64_t P, int K2,
                         int last_inf, int32_t *best, double *best_cost, int32_t *branch,
                         hipStream_t stream);

// Finite-capacity admission replay (n <= kReplayMaxN requests per sequence).
size_t replay_ws_bytes(int64_t reps, int64_t n, int K);
hipError_t launch_replay(const double *arrival, const double *wait, const int32_t *ctx,
                         int64_t reps, int64_t n, const double *h_t2, int K, int64_t c2, double b2,
                         double b3, void *ws, double *cost, int64_t *restored,
                         int64_t *admitted, int *status, hipStream_t stream);

// Controller tail: share of waits <= t_star and token total over N waits,
// then the branch totals from the replay's per-row counts [reps][2].
size_t count_ws_bytes();
hipError_t launch_short_count(const double *wait, const int32_t *ctx, int64_t N, double t_star,
                              void *count_ws, int *status, hipStream_t stream);
hipError_t launch_fraction(const void *count_ws, int64_t N, int64_t *count, double *fraction,
                           hipStream_t stream);
hipError_t launch_controller_final(const int64_t *restored, const int64_t *admitted,
                                   int64_t reps, int64_t n_requests, const void *count_ws,
                                   double t2, double t_star, double b2, double b3,
                                   kvr_controller_out *out, hipStream_t stream);

// Brute-force grid of one sample with few t1 timers and deadlines in one
// launch after the table staging (kvr_small.hip).  Workspace of that launch:
struct SmallWs {
    unsigned long long *hist;   // [nsb][nbins] pre-pass blocks' recompute histograms
    int32_t *lb;                // [K1*K2] grid deadlines strictly below each policy's
    double *xgp;                // [nsb][K1][2] pre-pass blocks' X and G
    unsigned long long *S;      // [nbins] suffix sums of the histogram
    double *XG;                 // [K1][2] X and G of the sample
    double *partials;           // [ceil(nsplit / kSmallWaves)][ntiles][LT][K1*K2]
    unsigned *ctr;              // arrival counters, zero at launch: the pre-pass, each
                                // (group, tile), each batch of a (group, tile)'s split groups
    int64_t nbins;              // F, the number of finite grid deadlines
    int nsb, npb;               // pre-pass sample blocks and policy blocks
};
bool small_path_fits(int K1, int K2, int64_t nbins, int64_t n);
int small_sample_blocks(int64_t n);
int small_policy_blocks(int64_t P);
hipError_t launch_small(const SampleSrc &src, const Tables &tb, const PriceDev &pr,
                        const GridPlan &plan, const SmallWs &ws, double *cost_out, int *status,
                        hipStream_t stream);

// Sorted path.
struct SortWs {
    uint64_t *keys[2];
    int32_t *vals[2];
    uint32_t *hist;       // [256][nblocks]
    uint32_t *counts;     // [256] digit totals of the current pass
    int64_t *Nsum;        // [n] inclusive prefix of T (sorted order), or the sums of T over
                          // each run of 64 sorted positions when the closed form queries
    double *Ssum;         // [n] the same for T*w
    int64_t *blkN;        // [nblocks_scan]
    double *blkS;         // [nblocks_scan]
    int nblocks;          // sort tiles
    int kpt;              // keys per thread of a sort tile (tile = 256 * kpt keys)
    int nblocks_scan;     // scan tiles
};

size_t sort_ws_bytes(int64_t n);
void sort_ws_carve(void *base, int64_t n, SortWs &ws);
// Stable radix sort of the waits only: afterwards ws.keys[*cur_out] holds the
// sorted key bits (fl(w + 0.0)) and ws.vals[*cur_out] the base index at each
// sorted position.
hipError_t launch_sort_keys(const double *w, const int32_t *T, int64_t n, SortWs &ws, int *cur_out,
                            int *status, hipStream_t stream);
hipError_t launch_sorted_path(const double *w, const int32_t *T, int64_t n, const Tables &tb,
                              const PriceDev &pr, SortWs &ws, double *cost_out,
                              int32_t *perm_out, int *status, hipStream_t stream);

}  // namespace kvr
