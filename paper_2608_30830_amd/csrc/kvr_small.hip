// The brute-force grid of one sample with few GPU-tier timers and few
// deadlines in one launch after the table staging.  Small grids are bound by
// their launches, not by their arithmetic, so the load-independent sums of
// Eq. 1 that the large path forms in separate launches (X and G per t1, the
// recompute share R3 per deadline through deadline bins, see kvr_r3.hip), the
// grid itself and the final combination all run as blocks of one kernel.
//
// Blocks (kSmallWaves waves each), in launch order:
//  * pre-pass, sample blocks b < nsb: kSmallPer consecutive samples.  Each
//    sample's deadline bin c(w) (the number of grid deadlines below it, by
//    binary searches in LDS copies of the timer tables) adds T to an LDS
//    histogram of bins 1..F, stored as the block's row hist[b][F];
//    X(t1) = sum T*min(w, t1) and G(t1) = sum T*[w > t1] are added over the
//    block in a fixed order into partials xgp[b][a][2];
//  * pre-pass, policy blocks: each policy's lb = c(e);
//  * grid blocks: one (group of 64 policies, tile of LT loads) and kSmallWaves
//    consecutive sample splits, one per wave, whose accumulators are added in
//    wave order in LDS into one partial per block (per split group).
// No block waits for another.  Each block counts itself done on a counter
// after its results are visible device-wide.  The pre-pass block that
// completes the pre-pass adds the histogram rows (block order), takes their
// suffix sums and adds X and G (block order), publishes them, and counts one
// more on every (group, tile).  The grid block that completes a batch of
// kSmallBatch split groups of its (group, tile) adds their partials in split
// order into the batch's first slot and counts the batch on the (group,
// tile).  Whichever block completes a (group, tile) -- its last batch's, or
// that pre-pass block -- forms its mean costs: the batch sums added in batch
// order plus a1*X + b2*(G - R3) + b3*R3.  Every sum is taken in a fixed order,
// so the result does not depend on the order in which blocks finish.
#include "kvr_device.h"

namespace kvr {

constexpr int kSmallThreads = kSmallWaves * kWave;             // 512
constexpr int kSmallSPT = 2;                                   // samples per thread (pre-pass)
constexpr int kSmallPer = kSmallThreads * kSmallSPT;           // samples per pre-pass block
constexpr int kSmallMaxK1 = 8;
constexpr int kSmallMaxK2 = 4096;
constexpr int kSmallMaxBins = 4096;
constexpr int kFinFlight = 16;   // histogram rows and split partials in flight per thread
constexpr int kSmallBatch = kSmallBatchGroups;   // split groups added by their batch's last block

int small_sample_blocks(int64_t n) { return (int)((n + kSmallPer - 1) / kSmallPer); }

int small_policy_blocks(int64_t P) { return (int)((P + kSmallThreads - 1) / kSmallThreads); }

// The pre-pass block that completes the pre-pass adds all histogram rows:
// kept to 65,536 words (65,536 waits with 1,024 deadlines, or 256 blocks of 256).
bool small_path_fits(int K1, int K2, int64_t nbins, int64_t n)
{
    const int64_t nsb = small_sample_blocks(n);
    return K1 <= kSmallMaxK1 && K2 <= kSmallMaxK2 && nbins <= kSmallMaxBins && nsb <= 256 &&
           nsb * nbins <= 65536;
}

// Grid deadlines fl(t1[a] + t2[k]) strictly below x, from LDS tables (each
// t1 row is non-decreasing in t2).
__device__ __forceinline__ int32_t small_bin(const double *t1, int K1, const double *t2, int K2,
                                             double x)
{
    int32_t c = 0;
    for (int a = 0; a < K1; ++a) {
        int lo = 0, hi = K2;
        while (lo < hi) {
            const int mid = (lo + hi) >> 1;
            if (t1[a] + t2[mid] < x) lo = mid + 1;
            else hi = mid;
        }
        c += lo;
    }
    return c;
}

// LDS of one block, shared by the roles (a block takes one role).
struct SmallPrepLds {
    double t1[kSmallMaxK1];
    union {
        double t2[kSmallMaxK2];
            int list[kSmallMaxGroupTiles];            // after the pre-pass: the (group, tile)s
    };                                            // this block completes
    unsigned long long h[kSmallMaxBins];          // histogram, then the suffix sums
    double wred[kSmallWaves][2 * kSmallMaxK1];    // per-wave X and G
    unsigned long long wtot[kSmallWaves];
};
static_assert(sizeof(int) * kSmallMaxGroupTiles <= sizeof(double) * kSmallMaxK2,
              "the completion list shares the t2 table's LDS");

template <int LT, int MODE>
struct SmallGridLds {
    static constexpr bool kStaged = MODE != kModePerLane;
    union {
        struct {
            // per-lane d: (w, T) per sample; staged: (T, d) per sample for the
            // group's two t1 rows (A, B), so a lane reads one 16-byte record per sample
            double2 wt[kStaged ? 1 : kSmallWaves][2][kStaged ? 1 : kChunk];
            double2 td[kStaged ? kSmallWaves : 1][2][kStaged ? kChunk : 1][2];
        } st;
        double red[LT][kWave];   // after the last chunk: the waves' accumulators
    };
};

template <int LT, int MODE>
constexpr size_t small_lds_bytes()
{
    return sizeof(SmallPrepLds) > sizeof(SmallGridLds<LT, MODE>) ? sizeof(SmallPrepLds)
                                                                 : sizeof(SmallGridLds<LT, MODE>);
}

// Values passed between blocks of one launch are stored and loaded as
// agent-scope relaxed atomics, which gfx950 serves coherently across the
// XCDs' L2 caches; an agent-scope fence would instead write back and
// invalidate a whole L2 at every block's arrival (measured on MI355X: the
// mix-64k call took 0.18 ms with such fences, 0.045 ms without).
__device__ __forceinline__ void put_u64(unsigned long long *p, unsigned long long v)
{
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned long long get_u64(const unsigned long long *p)
{
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void put_f64(double *p, double v)
{
    put_u64(reinterpret_cast<unsigned long long *>(p), (unsigned long long)__double_as_longlong(v));
}
__device__ __forceinline__ double get_f64(const double *p)
{
    return __longlong_as_double((long long)get_u64(reinterpret_cast<const unsigned long long *>(p)));
}
__device__ __forceinline__ void put_i32(int32_t *p, int32_t v)
{
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int32_t get_i32(const int32_t *p)
{
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Every memory operation this thread issued has completed (vector memory
// counter at zero; the others are not waited for), and the compiler keeps
// the thread's accesses on their side of this point.
__device__ __forceinline__ void release_order()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_s_waitcnt(0 | (0x7 << 4) | (0xf << 8));
}
__device__ __forceinline__ void acquire_order()
{
    __builtin_amdgcn_s_waitcnt(0 | (0x7 << 4) | (0xf << 8));
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

__device__ __forceinline__ unsigned arrive(unsigned *ctr)
{
    return __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Counts this block done on *ctr after every thread's stores (put_*) have
// completed; every thread gets the count before this block's add.
__device__ __forceinline__ unsigned block_arrive(unsigned *ctr, unsigned *slot)
{
    release_order();
    __syncthreads();
    if (threadIdx.x == 0) *slot = arrive(ctr);
    __syncthreads();
    const unsigned old = *slot;
    acquire_order();
    return old;
}

// Sum of the partials of n consecutive slots starting at slot s0, in slot
// order (slot = split group; a slot holds [ntiles][LT][P]), loads in flight.
__device__ __forceinline__ double sum_slots(const double *p0, int s0, int n, int slice)
{
    const double *p = p0 + s0 * slice;
    double s = get_f64(p);
    int q = 1;
    for (; q + kFinFlight <= n; q += kFinFlight) {   // loads in flight, added in slot order
        const double *pq = p + q * slice;
        double v[kFinFlight];
#pragma unroll
        for (int u = 0; u < kFinFlight; ++u) v[u] = get_f64(pq + u * slice);
#pragma unroll
        for (int u = 0; u < kFinFlight; ++u) s += v[u];
    }
    for (; q < n; ++q) s += get_f64(p + q * slice);
    return s;
}

// The (policy, load) items of one (group of 64 policies, tile of LT loads):
// thread (q, lane) takes policy grp*64 + lane and loads q, q + kSmallWaves, ...
// (the partials hold fewer than 2^31 values: the plan caps them at 1 GiB).
template <int LT, typename Fn>
__device__ __forceinline__ void for_items(int gt, const GridPlan &plan, const Tables &tb, Fn fn)
{
    const int64_t P = (int64_t)tb.K1 * tb.K2;
    const int grp = gt / plan.ntiles, tile = gt % plan.ntiles;
    const int lane = (int)threadIdx.x % kWave, q0 = (int)threadIdx.x / kWave;
    const int64_t f = (int64_t)grp * kWave + lane;
    if (f >= P) return;
    for (int ll = q0; ll < LT; ll += kSmallWaves) {
        const int l = tile * LT + ll;
        if (l >= tb.L) break;
        fn(f, l, ((int64_t)tile * LT + ll) * P + f);
    }
}

// A batch's split groups [s0, s0 + n) added into slot s0.
template <int LT>
__device__ void small_batch(int gt, int s0, int n, const GridPlan &plan, const Tables &tb,
                            const SmallWs &ws)
{
    const int slice = (int)(plan.ntiles * LT * (int64_t)tb.K1 * tb.K2);
    for_items<LT>(gt, plan, tb, [&](int64_t, int, int64_t off) {
        const double *p0 = ws.partials + off;
        put_f64(ws.partials + off + (int64_t)s0 * slice, sum_slots(p0, s0, n, slice));
    });
}

// Mean costs of one (group, tile): the batch sums (slots 0, kSmallBatch, ...)
// added in batch order, plus the load-independent terms.
template <int LT>
__device__ void small_finish(int gt, const GridPlan &plan, const Tables &tb, const PriceDev &pr,
                             double md, int nsg, const SmallWs &ws, double *__restrict__ cost_out)
{
    const int64_t P = (int64_t)tb.K1 * tb.K2;
    const int slice = (int)(plan.ntiles * LT * P);
    const int nbatch = (nsg + kSmallBatch - 1) / kSmallBatch;
    for_items<LT>(gt, plan, tb, [&](int64_t f, int l, int64_t off) {
        const int a = (int)(f / tb.K2);
        const double x = get_f64(&ws.XG[a * 2]), g = get_f64(&ws.XG[a * 2 + 1]);
        const int32_t xb = get_i32(&ws.lb[f]);
        const double r3 = (xb < ws.nbins) ? (double)get_u64(&ws.S[xb]) : 0.0;
        const double base = pr.a1 * x + (pr.b2 * (g - r3) + pr.b3 * r3);
        const double s = sum_slots(ws.partials + off, 0, nbatch, kSmallBatch * slice);
        cost_out[(int64_t)l * P + f] = (base + s) / md;
    });
}

// Pre-pass block: sample block b < nsb, else policy block b - nsb.
__device__ void small_prep(SmallPrepLds &sm, const double *__restrict__ w,
                           const int32_t *__restrict__ T, int64_t n, const Tables &tb,
                           const SmallWs &ws, int b, int *status)
{
    const int K1 = tb.K1, K2 = tb.K2;
    const int lane = (int)threadIdx.x % kWave, wv = (int)threadIdx.x / kWave;
    for (int i = threadIdx.x; i < K2; i += kSmallThreads) sm.t2[i] = tb.t2[i];
    if ((int)threadIdx.x < K1) sm.t1[threadIdx.x] = tb.t1[threadIdx.x];
    if (b >= ws.nsb) {   // policies: lb = deadlines below their own
        __syncthreads();
        const int64_t f = (int64_t)(b - ws.nsb) * kSmallThreads + threadIdx.x;
        if (f < (int64_t)K1 * K2) {
            const int a = (int)(f / K2), k = (int)(f % K2);
            put_i32(&ws.lb[f], small_bin(sm.t1, K1, sm.t2, K2, sm.t1[a] + sm.t2[k]));
        }
        return;
    }
    for (int64_t i = threadIdx.x; i < ws.nbins; i += kSmallThreads) sm.h[i] = 0ull;
    __syncthreads();
    double xs[kSmallMaxK1], gs[kSmallMaxK1];
#pragma unroll
    for (int a = 0; a < kSmallMaxK1; ++a) {
        xs[a] = 0.0;
        gs[a] = 0.0;
    }
    const int64_t j0 = (int64_t)b * kSmallPer;
    bool bad = false;
#pragma unroll
    for (int q = 0; q < kSmallSPT; ++q) {
        const int64_t j = j0 + q * kSmallThreads + threadIdx.x;
        if (j >= n) break;
        double x = w[j];
        int32_t t = T[j];
        // finite and >= 0 (or -0.0), tested on the bits; the grid blocks read
        // the same sample and replace it the same way
        const uint64_t bits = (uint64_t)__double_as_longlong(x);
        if (!(bits < 0x7ff0000000000000ull || bits == 0x8000000000000000ull)) {
            bad = true;
            x = 0.0;
        }
        if (t < 1) {
            bad = true;
            t = 1;
        }
        x = x + 0.0;   // -0.0 -> +0.0
        const double Td = (double)t;
        const int32_t c = small_bin(sm.t1, K1, sm.t2, K2, x);
        if (c >= 1) atomicAdd(&sm.h[c - 1], (unsigned long long)t);   // bin 0 is never read
#pragma unroll
        for (int a = 0; a < kSmallMaxK1; ++a) {
            if (a < K1) {
                xs[a] = fma(Td, fmin(x, sm.t1[a]), xs[a]);
                gs[a] += (x > sm.t1[a]) ? Td : 0.0;
            }
        }
    }
    if (bad) flag_domain(status);
    // X and G: a fixed butterfly within each wave, then the waves in order
#pragma unroll
    for (int a = 0; a < kSmallMaxK1; ++a) {
        if (a < K1) {
            const double xa = wave_sum(xs[a]), ga = wave_sum(gs[a]);
            if (lane == 0) {
                sm.wred[wv][a] = xa;
                sm.wred[wv][kSmallMaxK1 + a] = ga;
            }
        }
    }
    __syncthreads();
    if ((int)threadIdx.x < 2 * K1) {
        const int a = (int)threadIdx.x % K1, which = (int)threadIdx.x / K1;
        double v = 0.0;
        for (int q = 0; q < kSmallWaves; ++q) v += sm.wred[q][which * kSmallMaxK1 + a];
        put_f64(&ws.xgp[((int64_t)b * K1 + a) * 2 + which], v);
    }
    // this block's row of the histogram (integer sums; rows are added by the
    // block that completes the pre-pass, so no atomics contend across blocks)
    for (int64_t i = threadIdx.x; i < ws.nbins; i += kSmallThreads)
        put_u64(&ws.hist[(int64_t)b * ws.nbins + i], sm.h[i]);
}

// The block that completes the pre-pass: the histogram rows added in block
// order and suffix-summed (S[x] = sum of bins x.. in stored index), X and G
// added in block order; both published to the workspace.
__device__ void small_prep_total(SmallPrepLds &sm, const Tables &tb, const SmallWs &ws)
{
    const int nsb = ws.nsb;
    for (int64_t i = threadIdx.x; i < ws.nbins; i += kSmallThreads) {
        unsigned long long v = 0ull;
        int b = 0;
        for (; b + kFinFlight <= nsb; b += kFinFlight) {   // rows in flight, added in block order
            unsigned long long u[kFinFlight];
#pragma unroll
            for (int q = 0; q < kFinFlight; ++q) u[q] = get_u64(&ws.hist[(int64_t)(b + q) * ws.nbins + i]);
#pragma unroll
            for (int q = 0; q < kFinFlight; ++q) v += u[q];
        }
        for (; b < nsb; ++b) v += get_u64(&ws.hist[(int64_t)b * ws.nbins + i]);
        sm.h[i] = v;
    }
    if ((int)threadIdx.x < 2 * tb.K1) {
        const int a = (int)threadIdx.x % tb.K1, which = (int)threadIdx.x / tb.K1;
        double v = 0.0;
        int b = 0;
        for (; b + kFinFlight <= nsb; b += kFinFlight) {   // in flight, added in block order
            double u[kFinFlight];
#pragma unroll
            for (int q = 0; q < kFinFlight; ++q) u[q] = get_f64(&ws.xgp[((int64_t)(b + q) * tb.K1 + a) * 2 + which]);
#pragma unroll
            for (int q = 0; q < kFinFlight; ++q) v += u[q];
        }
        for (; b < nsb; ++b) v += get_f64(&ws.xgp[((int64_t)b * tb.K1 + a) * 2 + which]);
        put_f64(&ws.XG[a * 2 + which], v);
    }
    __syncthreads();
    // suffix sums in chunks of one value per thread from the top down, in place
    unsigned long long carry = 0;
    const int lane = threadIdx.x % kWave, wv = threadIdx.x / kWave;
    for (int64_t top = ws.nbins; top > 0; top -= kSmallThreads) {
        const int64_t pos = top - 1 - threadIdx.x;
        unsigned long long v = pos >= 0 ? sm.h[pos] : 0ull;
        for (int off = 1; off < kWave; off <<= 1) {
            const unsigned long long o = __shfl_up(v, off, kWave);
            if (lane >= off) v += o;
        }
        if (lane == kWave - 1) sm.wtot[wv] = v;
        __syncthreads();
        unsigned long long before = carry, all = carry;
        for (int q = 0; q < kSmallWaves; ++q) {
            if (q < wv) before += sm.wtot[q];
            all += sm.wtot[q];
        }
        if (pos >= 0) sm.h[pos] = v + before;
        carry = all;
        __syncthreads();
    }
    for (int64_t i = threadIdx.x; i < ws.nbins; i += kSmallThreads) put_u64(&ws.S[i], sm.h[i]);
}

// Grid block: the holding term of Eq. 1 at the Eq. 3 price, one fp64 FMA per
// (sample, policy, load), as in grid_kernel (kvr_grid.hip) for one resample;
// wave wv takes split sg * kSmallWaves + wv, and the waves' accumulators are
// added in wave order into the block's partial.
template <int LT, int MODE>
__device__ void small_grid(SmallGridLds<LT, MODE> &sm, const SampleSrc &src, const Tables &tb,
                           const GridPlan &plan, const SmallWs &ws, int64_t logical, int nsg,
                           int *status)
{
    constexpr bool kStaged = MODE != kModePerLane;
    constexpr int kPer = kChunk / kWave;   // samples each lane stages per chunk
    const int wv = (int)threadIdx.x / kWave, lane = (int)threadIdx.x % kWave;
    auto &wt = sm.st.wt[kStaged ? 0 : wv];
    auto &td = sm.st.td[kStaged ? wv : 0];
    const int tile = (int)(logical % plan.ntiles);
    const int64_t rest = logical / plan.ntiles;
    const int sg = (int)(rest % nsg);
    const int64_t grp = rest / nsg;
    const int split = sg * kSmallWaves + wv;

    const int64_t P = (int64_t)tb.K1 * tb.K2;
    const int64_t FA = grp * kWave;
    const int64_t FB = (FA + kWave - 1 < P) ? FA + kWave - 1 : P - 1;
    int64_t f = FA + lane;
    const bool valid = f < P;
    if (!valid) f = FB;
    const int a = (int)(f / tb.K2);
    const int k = (int)(f % tb.K2);
    const double t1 = tb.t1[a];
    const double e = t1 + tb.t2[k];   // deadline from suspension
    const double ep = e - t1;         // host time before discard
    // the group's (at most two) t1 rows
    const int aA = (int)(FA / tb.K2), aB = (int)(FB / tb.K2);
    const double t1A = tb.t1[aA], t1B = tb.t1[aB];
    const int sel = (a == aA) ? 0 : 1;

    double a2[LT], acc[LT];
#pragma unroll
    for (int l = 0; l < LT; ++l) {
        a2[l] = tb.a2[tile * LT + l];
        acc[l] = 0.0;
    }
    int64_t j0 = (int64_t)split * plan.split_len;   // a block's last waves may have no samples
    if (j0 > src.m) j0 = src.m;
    int64_t j1 = j0 + plan.split_len;
    if (j1 > src.m) j1 = src.m;
    // every wave takes the same number of chunks (the block's barriers),
    // padding the short ones with zeros
    const int64_t nch = (plan.split_len + kChunk - 1) / kChunk;

    Sample pre[kPer];
    auto load_chunk = [&](int64_t c) {
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            const int64_t j = j0 + c * kChunk + q * kWave + lane;
            if (j < j1) {
                pre[q] = fetch_sample(src, 0, j, status);
            } else {  // padding: contributes exact zeros
                pre[q].w = 0.0;
                pre[q].T = 0.0;
            }
        }
    };
    auto store_chunk = [&](int b) {
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            const int s = q * kWave + lane;
            if (kStaged) {
                td[b][s][0] = make_double2(pre[q].T, fmax(pre[q].w, t1A) - t1A);
                td[b][s][1] = make_double2(pre[q].T, fmax(pre[q].w, t1B) - t1B);
            } else {
                wt[b][s] = make_double2(pre[q].w, pre[q].T);
            }
        }
    };

    if (nch > 0) {
        load_chunk(0);
        store_chunk(0);
    }
    __syncthreads();
    for (int64_t c = 0; c < nch; ++c) {
        const int cur = (int)(c & 1);
        if (c + 1 < nch) load_chunk(c + 1);
#pragma unroll 8
        for (int j = 0; j < kChunk; ++j) {
            double Tj, d;
            if (kStaged) {                            // this lane's t1 row
                const double2 s = td[cur][j][sel];
                Tj = s.x;
                d = s.y;
            } else {
                const double2 s = wt[cur][j];
                Tj = s.y;
                d = fmax(s.x, t1) - t1;               // 0 when w <= t1
            }
            const double h = Tj * fmin(d, ep);        // T * host seconds held
#pragma unroll
            for (int l = 0; l < LT; ++l) acc[l] = fma(a2[l], h, acc[l]);
        }
        if (c + 1 < nch) store_chunk(cur ^ 1);
        __syncthreads();
    }
    // the block's splits in wave order, then one partial
    for (int q = 1; q < kSmallWaves; ++q) {
        if (wv == q) {
#pragma unroll
            for (int l = 0; l < LT; ++l) sm.red[l][lane] = acc[l];
        }
        __syncthreads();
        if (wv == 0) {
#pragma unroll
            for (int l = 0; l < LT; ++l) acc[l] += sm.red[l][lane];
        }
        __syncthreads();
    }
    if (wv == 0 && valid) {
        const int64_t base_row = ((int64_t)sg * plan.ntiles + tile) * LT;
#pragma unroll
        for (int l = 0; l < LT; ++l) put_f64(&ws.partials[(base_row + l) * P + f], acc[l]);
    }
}

template <int LT, int MODE>
__global__ void __launch_bounds__(kSmallThreads) __attribute__((amdgpu_waves_per_eu(4)))
small_fused_kernel(SampleSrc src, Tables tb, PriceDev pr, GridPlan plan, SmallWs ws,
                   double *__restrict__ cost_out, int *status)
{
    __shared__ __align__(16) unsigned char lds[small_lds_bytes<LT, MODE>()];
    __shared__ unsigned arrived;
    __shared__ int nfin, one;
    const int nprep = ws.nsb + ws.npb;
    const int nsg = (plan.nsplit + kSmallWaves - 1) / kSmallWaves;
    const int *fin;   // the (group, tile)s this block completes, nfin of them
    if ((int)blockIdx.x < nprep) {
        auto &sm = *reinterpret_cast<SmallPrepLds *>(lds);
        small_prep(sm, src.w, src.T, src.m, tb, ws, (int)blockIdx.x, status);
        if (block_arrive(&ws.ctr[0], &arrived) != (unsigned)(nprep - 1)) return;
        // the pre-pass is complete: totals, then one more on every (group, tile)
        small_prep_total(sm, tb, ws);
        release_order();   // S, X and G stored before any (group, tile) counts them
        if (threadIdx.x == 0) nfin = 0;
        __syncthreads();
        const int ngt = (int)(plan.ngroups * plan.ntiles);
        const unsigned nbatch = (unsigned)((nsg + kSmallBatch - 1) / kSmallBatch);
        for (int gt = threadIdx.x; gt < ngt; gt += kSmallThreads) {
            if (arrive(&ws.ctr[1 + gt]) == nbatch) sm.list[atomicAdd(&nfin, 1)] = gt;
        }
        __syncthreads();
        acquire_order();
        fin = sm.list;
    } else {
        const int64_t logical = (int64_t)blockIdx.x - nprep;
        auto &sm = *reinterpret_cast<SmallGridLds<LT, MODE> *>(lds);
        small_grid<LT, MODE>(sm, src, tb, plan, ws, logical, nsg, status);
        const int64_t rest = logical / plan.ntiles;
        const int gt = (int)((rest / nsg) * plan.ntiles + logical % plan.ntiles);
        const int sg = (int)(rest % nsg), s0 = sg - sg % kSmallBatch;
        const int nb = nsg - s0 < kSmallBatch ? nsg - s0 : kSmallBatch;
        const int nbatch = (nsg + kSmallBatch - 1) / kSmallBatch;
        const int ngt = (int)(plan.ngroups * plan.ntiles);
        // the batch's last block adds it up
        if (block_arrive(&ws.ctr[1 + ngt + (int64_t)gt * nbatch + s0 / kSmallBatch], &arrived) !=
            (unsigned)(nb - 1))
            return;
        if (nb > 1) small_batch<LT>(gt, s0, nb, plan, tb, ws);
        // nbatch batches and the pre-pass's one: the last of them finishes
        if (block_arrive(&ws.ctr[1 + gt], &arrived) != (unsigned)nbatch) return;
        if (threadIdx.x == 0) {
            one = gt;
            nfin = 1;
        }
        __syncthreads();
        fin = &one;
    }
    const int nf = nfin;
    for (int i = 0; i < nf; ++i) small_finish<LT>(fin[i], plan, tb, pr, (double)src.m, nsg, ws, cost_out);
}

template <int LT, int MODE>
static hipError_t launch_small_m(const SampleSrc &src, const Tables &tb, const PriceDev &pr,
                                 const GridPlan &plan, const SmallWs &ws, double *cost_out,
                                 int *status, hipStream_t stream)
{
    const int64_t nsg = (plan.nsplit + kSmallWaves - 1) / kSmallWaves;
    const int64_t nblocks = ws.nsb + ws.npb + plan.ngroups * nsg * plan.ntiles;
    hipLaunchKernelGGL((small_fused_kernel<LT, MODE>), dim3((unsigned)nblocks), dim3(kSmallThreads),
                       0, stream, src, tb, pr, plan, ws, cost_out, status);
    return hipGetLastError();
}

template <int LT>
static hipError_t launch_small_t(const SampleSrc &src, const Tables &tb, const PriceDev &pr,
                                 const GridPlan &plan, const SmallWs &ws, double *cost_out,
                                 int *status, hipStream_t stream)
{
    switch (plan.mode) {
    case kModePerLane: return launch_small_m<LT, kModePerLane>(src, tb, pr, plan, ws, cost_out, status, stream);
    case kModeRows1: return launch_small_m<LT, kModeRows1>(src, tb, pr, plan, ws, cost_out, status, stream);
    default: return hipErrorInvalidValue;   // one resample never straddles two
    }
}

hipError_t launch_small(const SampleSrc &src, const Tables &tb, const PriceDev &pr,
                        const GridPlan &plan, const SmallWs &ws, double *cost_out, int *status,
                        hipStream_t stream)
{
    // the launch assumes one resample read directly, splits grouped by
    // kSmallWaves, a histogram within the LDS table and every counter cleared
    if (src.idx != nullptr || plan.R != 1 || plan.wpb != kSmallWaves || src.m != src.n ||
        !small_path_fits(tb.K1, tb.K2, ws.nbins, src.m) ||
        plan.ngroups * plan.ntiles > kSmallMaxGroupTiles || ws.nsb != small_sample_blocks(src.m) ||
        ws.npb != small_policy_blocks((int64_t)tb.K1 * tb.K2))
        return hipErrorInvalidValue;
    switch (plan.LT) {
    case 4: return launch_small_t<4>(src, tb, pr, plan, ws, cost_out, status, stream);
    case 8: return launch_small_t<8>(src, tb, pr, plan, ws, cost_out, status, stream);
    case 16: return launch_small_t<16>(src, tb, pr, plan, ws, cost_out, status, stream);
    case 32: return launch_small_t<32>(src, tb, pr, plan, ws, cost_out, status, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace kvr
