// Finite-capacity admission replay for gfx950 (Appendix D; the evaluation
// behind Table 6).
//
// Every request is offloaded to host DRAM at suspension.  The host tier has C2
// slots: a request that arrives while a slot is free is admitted, one that
// finds the tier full recomputes at resume, residents are never displaced.
// Under a host timer t2 an admitted request whose wait exceeds t2 leaves at
// arrival + t2 (discarded, recompute at resume); otherwise it leaves at
// arrival + wait (restored from host).  Departures at or before an arrival free
// their slots first.  A replay reports the tokens restored from host; the mean
// cost per request is (b2*R + b3*(Ttot - R)) / n.
//
// GPU formulation (no heap): the departures of a replay come from two
// monotone streams -- resumes, ordered by the key (fl(arrival + wait), index),
// and expiries, which follow arrival order because fl(arrival + t2) is
// monotone in the arrival.  The resume stream depends neither on the timer nor
// on admissions, so one block per request sequence sorts it once and also
// records, for every arrival j, the resume cursor rcur[j] = the number of
// resume keys below (a_j, j): the resumes that have happened when request j
// arrives (a request arriving later never resumes before j arrives, since its
// key is at least (a_j, j)).  It also records the place of request i in the
// resume order; the two travel packed in one 32-bit word per request.
//
// The expiry stream depends on the timer but not on admissions: a second
// per-sequence pass records, for every timer and arrival j, how many earlier
// requests have reached their timer by a_j (a binary search, the arrivals
// being sorted) and whether j itself resumes before its timer.
//
// The merge runs one lane per (timer, sequence) pair, 64 or 40 pairs per wave,
// and keeps two lane-private bitsets in LDS: rbits[p] for "the request at
// resume place p was admitted and resumes before its timer", set at its
// admission through its place, and ebits[i] for "request i was admitted and
// is discarded at its timer".  At arrival j the departures that free slots
// are the set bits of rbits between the previous and the current resume
// cursor and of ebits between the previous and the current expiry cursor
// (popcounts over a two-word window of each).  The step loop reads only the
// packed per-arrival words, in register buffers of eight arrivals filled one
// buffer ahead of use: no load in it depends on another, and a wave's walk is
// bound by its own instruction stream rather than by chains of global loads.
#include "kvr_device.h"

namespace kvr {

constexpr int kReplayMaxN = 8192;
constexpr int kReplaySortThreads = 512;

// Sort key (resume time, request index): a total order, so ties in time keep
// index order.
__device__ __forceinline__ bool key_less(double ta, int ia, double tb, int ib)
{
    return ta < tb || (ta == tb && ia < ib);
}

// Keeps, of the pair (k, i) and (ok, oi), the smaller key under the total
// order when keep_low, else the larger.
__device__ __forceinline__ void keep_pair(double &k, int &i, double ok, int oi, bool keep_low)
{
    const bool mine_low = key_less(k, i, ok, oi);
    if (mine_low != keep_low) {
        k = ok;
        i = oi;
    }
}

// One compare-exchange stage of stride S < E among a thread's own elements
// (global index t*E + r; ascending blocks of `size`).
template <int E, int S>
__device__ __forceinline__ void reg_stage(double (&k)[E], int (&id)[E], int t, int size)
{
    if constexpr (S < E) {
#pragma unroll
        for (int r = 0; r < E; ++r) {
            const int q = r ^ S;
            if (q > r) {
                const bool asc = ((t * E + r) & size) == 0;
                const double kr = k[r], kq = k[q];
                const int ir = id[r], iq = id[q];
                const bool swap = key_less(kq, iq, kr, ir) == asc;
                k[r] = swap ? kq : kr;
                id[r] = swap ? iq : ir;
                k[q] = swap ? kr : kq;
                id[q] = swap ? ir : iq;
            }
        }
    }
}

// One block per request sequence (n <= MAXN): validate the row, bitonic-sort
// (fl(a + w), index) padded to MAXN with +inf, then write pr[j] = place of
// request j in the resume order (high 16 bits) | rcur[j] = number of keys
// below (a_j, j) (low 16 bits).  Thread t holds elements t*E .. t*E + E - 1 in
// registers: compare-exchange stages with stride < E stay in registers, those
// with stride < 64*E pair lanes of one wave (shuffles), and only the wider
// ones go through LDS with a block barrier.
template <int MAXN>
__global__ void __launch_bounds__(kReplaySortThreads) replay_sort_kernel(
    const double *__restrict__ arrival, const double *__restrict__ wait,
    const int32_t *__restrict__ ctx, int n, uint32_t *__restrict__ pr, int *status)
{
    constexpr int E = MAXN / kReplaySortThreads;
    constexpr int kPer = (MAXN + kReplaySortThreads - 1) / kReplaySortThreads;
    static_assert(E >= 1 && E * kReplaySortThreads == MAXN, "MAXN must be a multiple of 512");
    __shared__ double key[MAXN];
    __shared__ uint16_t idx[MAXN];
    const int64_t row = blockIdx.x;
    const double *A = arrival + row * n;
    const double *W = wait + row * n;
    const int t = threadIdx.x;
    // coalesced loads and checks into LDS, then each thread takes E consecutive keys
    for (int e = t; e < MAXN; e += blockDim.x) {
        if (e < n) {
            const double a = A[e], w = W[e];
            const uint64_t ba = (uint64_t)__double_as_longlong(a);
            const uint64_t bw = (uint64_t)__double_as_longlong(w);
            // finite and >= 0 (or -0.0), arrivals non-decreasing, contexts >= 1
            bool bad = !(ba < 0x7ff0000000000000ull || ba == 0x8000000000000000ull) ||
                       !(bw < 0x7ff0000000000000ull || bw == 0x8000000000000000ull);
            if (e > 0 && !(A[e - 1] <= a)) bad = true;
            if (ctx != nullptr && ctx[row * n + e] < 1) bad = true;
            if (bad) flag_domain(status);
            key[e] = a + w;
        } else {   // padding sorts last: +inf with indices above every request
            key[e] = INFINITY;
        }
    }
    __syncthreads();
    double k[E];
    int id[E];
#pragma unroll
    for (int r = 0; r < E; ++r) {
        id[r] = t * E + r;
        k[r] = key[t * E + r];
    }
    __syncthreads();
    for (int size = 2; size <= MAXN; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            if (stride < E) {
                if (stride == 1) reg_stage<E, 1>(k, id, t, size);
                else if (stride == 2) reg_stage<E, 2>(k, id, t, size);
                else if (stride == 4) reg_stage<E, 4>(k, id, t, size);
                else reg_stage<E, 8>(k, id, t, size);
            } else if (stride < kWave * E) {
                const int m = stride / E;   // partner lane offset
#pragma unroll
                for (int r = 0; r < E; ++r) {
                    const int e = t * E + r;
                    const double ok = __shfl_xor(k[r], m, kWave);
                    const int oi = __shfl_xor(id[r], m, kWave);
                    const bool lower = (e & stride) == 0, asc = (e & size) == 0;
                    keep_pair(k[r], id[r], ok, oi, lower == asc);
                }
            } else {
#pragma unroll
                for (int r = 0; r < E; ++r) {
                    key[t * E + r] = k[r];
                    idx[t * E + r] = (uint16_t)id[r];
                }
                __syncthreads();
#pragma unroll
                for (int r = 0; r < E; ++r) {
                    const int e = t * E + r;
                    const double ok = key[e ^ stride];
                    const int oi = idx[e ^ stride];
                    const bool lower = (e & stride) == 0, asc = (e & size) == 0;
                    keep_pair(k[r], id[r], ok, oi, lower == asc);
                }
                __syncthreads();
            }
        }
    }
#pragma unroll
    for (int r = 0; r < E; ++r) {
        key[t * E + r] = k[r];
        idx[t * E + r] = (uint16_t)id[r];
    }
    __syncthreads();
    // rcur: keys below (a_j, j), by a fixed-step search over all MAXN sorted
    // keys (the +inf padding is never below a finite target); the kPer
    // searches of a thread advance together, so their LDS reads overlap
    double ta[kPer];
    int pos[kPer];
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
        const int j = t + q * kReplaySortThreads;
        ta[q] = (j < n) ? A[j] : 0.0;
        pos[q] = 0;
    }
    for (int step = MAXN / 2; step > 0; step >>= 1) {
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            const int j = t + q * kReplaySortThreads;
            const int m = pos[q] + step - 1;
            if (key_less(key[m], idx[m], ta[q], j)) pos[q] += step;
        }
    }
    uint32_t rc[kPer];
#pragma unroll
    for (int q = 0; q < kPer; ++q) rc[q] = (uint32_t)pos[q];
    __syncthreads();
    uint16_t *place = reinterpret_cast<uint16_t *>(key);   // keys are no longer needed
    for (int p = t; p < n; p += blockDim.x) place[idx[p]] = (uint16_t)p;
    __syncthreads();
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
        const int j = t + q * kReplaySortThreads;
        if (j < n) pr[row * n + j] = ((uint32_t)place[j] << 16) | rc[q];
    }
}

constexpr int kRing = 8;   // arrivals per register buffer in the merge

// One block per request sequence (n <= MAXN): the arrivals into LDS, then for
// every timer k and arrival j the packed word
//   ec = min(j, #{i : fl(a_i + t2_k) <= a_j}) | [w_j <= t2_k] << 15,
// laid out [timer][reps][n] for the kc timers t2s[0..kc): how many earlier
// requests have reached their timer
// when j arrives (a prefix, since fl(a_i + t2) is non-decreasing in i) and
// whether j itself resumes before its timer.
template <int MAXN>
__global__ void __launch_bounds__(kReplaySortThreads) replay_expiry_kernel(
    const double *__restrict__ arrival, const double *__restrict__ wait, int n,
    const double *__restrict__ t2s, int kc, int64_t reps, uint16_t *__restrict__ ec)
{
    constexpr int kPer = (MAXN + kReplaySortThreads - 1) / kReplaySortThreads;
    __shared__ double A[MAXN];
    const int64_t row = blockIdx.x;
    const int t = threadIdx.x;
    for (int i = t; i < n; i += blockDim.x) A[i] = arrival[row * n + i];
    __syncthreads();
    // this thread's arrivals j = t + q*512 and their waits, read once
    double aj[kPer], wj[kPer];
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
        const int j = t + q * kReplaySortThreads;
        aj[q] = (j < n) ? A[j] : 0.0;
        wj[q] = (j < n) ? wait[row * n + j] : 0.0;
    }
    for (int k = 0; k < kc; ++k) {
        const double t2 = t2s[k];
        uint16_t *out = ec + ((int64_t)k * reps + row) * n;
        // #{i < j : fl(a_i + t2) <= a_j}, a prefix of [0, j) since the left
        // side is non-decreasing in i: fixed-step searches (steps MAXN/2 .. 1
        // sum to MAXN - 1 >= j) that advance together, so the kPer LDS reads
        // of a step overlap instead of forming kPer serial chains
        int pos[kPer];
#pragma unroll
        for (int q = 0; q < kPer; ++q) pos[q] = 0;
        for (int step = MAXN / 2; step > 0; step >>= 1) {
#pragma unroll
            for (int q = 0; q < kPer; ++q) {
                const int j = t + q * kReplaySortThreads;
                const int m = pos[q] + step - 1;   // < MAXN always
                if (m < j && A[m] + t2 <= aj[q]) pos[q] += step;
            }
        }
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            const int j = t + q * kReplaySortThreads;
            if (j < n) {
                const uint32_t stays = (wj[q] <= t2) ? 1u : 0u;
                out[j] = (uint16_t)((uint32_t)pos[q] | (stays << 15));
            }
        }
    }
}

// Set bits in [lo, hi) of the 64-bit window w1:w0, for 0 <= lo <= 32 and
// hi <= 64; zero when hi <= lo (lo = 32 only comes with an empty range).
__device__ __forceinline__ int count_window(uint32_t w0, uint32_t w1, int lo, int hi)
{
    const int width = hi - lo;
    const uint64_t win = ((uint64_t)w1 << 32) | w0;
    const uint64_t mask = width > 0 ? (~0ull >> (64 - width)) << lo : 0ull;
    return __popcll(win & mask);
}

// Set bits of a lane's column in [from, to) from the word after from's on
// (the rare case of a range longer than the two-word window).
template <int LPW>
__device__ __forceinline__ int count_tail(const uint32_t (*bits)[LPW], int lane, int from, int to)
{
    int c = 0;
    for (int b = ((from >> 5) + 1) << 5; b < to; b += 32) {
        uint32_t x = bits[b >> 5][lane];
        if (to - b < 32) x &= (1u << (to - b)) - 1u;
        c += __popc(x);
    }
    return c;
}

// One lane per (timer k0 + k, sequence) pair, k < kc, the pairs numbered
// timer-major and dealt LPW to a wave: 64, or 40 so that four waves, one per
// SIMD, fit in a CU's LDS (the other lanes leave at once: no lane touches
// another's LDS column and there is no barrier).  NW 32-bit words per bitset
// bound n <= 32*NW.  Lanes past the last pair walk the last one and write
// nothing.  The step loop reads only the packed per-arrival words (and the
// context sizes when CTX), kRing arrivals ahead, with no conditional loads.
template <int NW, int LPW, bool CTX>
__global__ void __launch_bounds__(kWave) replay_merge_kernel(
    const int32_t *__restrict__ ctx, int64_t reps, int n, int64_t c2,
    const uint32_t *__restrict__ pr, const uint16_t *__restrict__ ec, double b2, double b3,
    double *__restrict__ cost, int64_t *__restrict__ restored_out,
    int64_t *__restrict__ admitted_out, int k0, int kn, int K)
{
    __shared__ uint32_t rbits[NW][LPW];
    __shared__ uint32_t ebits[NW][LPW];
    const int lane = threadIdx.x;
    if (lane >= LPW) return;
    const int64_t pairs = reps * kn;
    const int64_t F = (int64_t)blockIdx.x * LPW + lane;
    const bool active = F < pairs;
    const int64_t Fa = active ? F : pairs - 1;
    const int k = (int)(Fa / reps);
    const int64_t row = Fa % reps;
    const int64_t rr = row;
    const int32_t *C = CTX ? ctx + rr * n : nullptr;
    const uint32_t *PR = pr + rr * n;
    const uint16_t *EC = ec + ((int64_t)k * reps + rr) * n;
    const int nw = (n + 31) >> 5;
    for (int q = 0; q < nw; ++q) {   // each lane clears only its own column
        rbits[q][lane] = 0u;
        ebits[q][lane] = 0u;
    }

    // Two buffers of kRing arrivals: one is processed while the other fills.
    int32_t ta[kRing], tb[kRing];
    uint32_t pa[kRing], pb[kRing], ea[kRing], eb[kRing];
    auto fill = [&](int32_t (&t)[kRing], uint32_t (&pw)[kRing], uint32_t (&ew)[kRing], int j0) {
#pragma unroll
        for (int u = 0; u < kRing; ++u) {
            const int jj = (j0 + u < n) ? j0 + u : n - 1;
            t[u] = CTX ? C[jj] : 1;
            pw[u] = PR[jj];
            ew[u] = EC[jj];
        }
    };

    // occupancy is at most n, so C2 above n is the same as n + 1
    const int cap = (c2 > (int64_t)n) ? n + 1 : (int)c2;
    int occ = 0, admitted = 0;
    int64_t restored = 0, total = 0;
    int rdone = 0;   // resume places already applied
    int edone = 0;   // requests (arrival order) whose timer has been applied
    auto run = [&](const int32_t (&t)[kRing], const uint32_t (&pw)[kRing],
                   const uint32_t (&ew)[kRing], int j0) {
#pragma unroll
        for (int u = 0; u < kRing; ++u) {
            const int j = j0 + u;
            if (j < n) {   // uniform across the wave
                const int p = (int)(pw[u] >> 16), rc = (int)(pw[u] & 0xffffu);
                const int ex = (int)(ew[u] & 0x7fffu);
                const bool stays = (ew[u] >> 15) != 0u;
                // departures at or before this arrival: set bits of rbits in
                // [rdone, rc) (resumes) and of ebits in [edone, ex) (timers);
                // the two words from each range's start are always read, so a
                // range of up to 33 bits, which nearly every step has, takes
                // no branch.  The second word's row is clamped to the last
                // row: a range ends at n <= 32*NW, so past the last row its
                // window bits are never counted.
                const int rq = ((rdone < n) ? rdone : n - 1) >> 5;
                const int eq = ((edone < n) ? edone : n - 1) >> 5;
                const int rq1 = (rq + 1 < NW) ? rq + 1 : rq;
                const int eq1 = (eq + 1 < NW) ? eq + 1 : eq;
                const uint32_t r0 = rbits[rq][lane], r1 = rbits[rq1][lane];
                const uint32_t e0 = ebits[eq][lane], e1 = ebits[eq1][lane];
                const int rhi = rc - (rq << 5), ehi = ex - (eq << 5);
                int gone = count_window(r0, r1, rdone - (rq << 5), rhi < 64 ? rhi : 64) +
                           count_window(e0, e1, edone - (eq << 5), ehi < 64 ? ehi : 64);
                if (rhi > 64 || ehi > 64)
                    gone += count_tail<LPW>(rbits, lane, (rq << 5) + 32, rc) +
                            count_tail<LPW>(ebits, lane, (eq << 5) + 32, ex);
                occ -= gone;
                rdone = (rc > rdone) ? rc : rdone;
                edone = (ex > edone) ? ex : edone;
                const int32_t T = t[u] < 1 ? 1 : t[u];
                total += T;
                const bool in = occ < cap;
                occ += in ? 1 : 0;
                admitted += in ? 1 : 0;
                restored += (in && stays) ? T : 0;
                // admitted requests leave a bit: at their resume place if they
                // resume in time, else at their arrival index (an OR of zero
                // when not admitted)
                uint32_t *word = stays ? &rbits[p >> 5][lane] : &ebits[j >> 5][lane];
                const int bit = stays ? (p & 31) : (j & 31);
                __hip_atomic_fetch_or(word, in ? (1u << bit) : 0u, __ATOMIC_RELAXED,
                                      __HIP_MEMORY_SCOPE_WORKGROUP);
            }
        }
    };
    fill(ta, pa, ea, 0);
    for (int jb = 0; jb < n; jb += 2 * kRing) {
        fill(tb, pb, eb, jb + kRing);
        run(ta, pa, ea, jb);
        fill(ta, pa, ea, jb + 2 * kRing);
        run(tb, pb, eb, jb + kRing);
    }
    if (!active) return;
    const int64_t sim = row * K + k0 + k;
    cost[sim] = (b2 * (double)restored + b3 * (double)(total - restored)) / (double)n;
    if (restored_out) restored_out[sim] = restored;
    if (admitted_out) admitted_out[sim] = admitted;
}

// Timers per pass of the expiry and merge kernels: at most 1 GiB of packed
// expiry words.
static int replay_timer_chunk(int64_t reps, int64_t n, int K)
{
    int64_t kc = ((int64_t)1 << 30) / (2 * reps * n);
    if (kc < 1) kc = 1;
    return (int)(kc < K ? kc : K);
}

size_t replay_ws_bytes(int64_t reps, int64_t n, int K)
{
    auto a256 = [](size_t x) { return (x + 255) & ~(size_t)255; };
    const int kc = replay_timer_chunk(reps, n, K);
    return a256(sizeof(uint32_t) * reps * n) + a256(sizeof(uint16_t) * kc * reps * n) +
           a256(sizeof(double) * K);
}

// Lanes per merge wave.  A wave's step is bound by its own instruction
// stream, so two waves on one SIMD take twice as long: the time goes with the
// most waves any SIMD runs.  Each lane keeps 2*NW words of LDS and a CU (four
// SIMDs, 160 KiB of LDS; 256 CUs) holds only so many waves; 40-lane waves are
// taken when they put fewer waves on the busiest SIMD than 64-lane ones.
static int merge_lanes(int64_t reps, int kn, int nw)
{
    auto load = [&](int64_t lpw) {
        int64_t per_cu = (int64_t)160 * 1024 / (8 * (int64_t)nw * lpw);
        per_cu = per_cu < 4 ? per_cu : 4;
        const int64_t waves = (reps * kn + lpw - 1) / lpw;
        return (waves + 256 * per_cu - 1) / (256 * per_cu);
    };
    return load(40) < load(64) ? 40 : 64;
}

template <int MAXN, int NW>
static hipError_t launch_replay_n(const double *arrival, const double *wait, const int32_t *ctx,
                                  int64_t reps, int n, const double *t2, int K, int64_t c2,
                                  double b2, double b3, uint32_t *pr, uint16_t *ec, double *cost,
                                  int64_t *restored, int64_t *admitted, int *status,
                                  hipStream_t stream)
{
    hipLaunchKernelGGL(replay_sort_kernel<MAXN>, dim3((unsigned)reps), dim3(kReplaySortThreads), 0,
                       stream, arrival, wait, ctx, n, pr, status);
    const int kc = replay_timer_chunk(reps, n, K);
    for (int k0 = 0; k0 < K; k0 += kc) {
        const int kn = (K - k0 < kc) ? K - k0 : kc;
        hipLaunchKernelGGL(replay_expiry_kernel<MAXN>, dim3((unsigned)reps),
                           dim3(kReplaySortThreads), 0, stream, arrival, wait, n, t2 + k0, kn, reps,
                           ec);
        const int lpw = merge_lanes(reps, kn, NW);
        const unsigned blocks = (unsigned)((reps * kn + lpw - 1) / lpw);
        if (lpw == 40 && ctx != nullptr)
            hipLaunchKernelGGL((replay_merge_kernel<NW, 40, true>), dim3(blocks), dim3(kWave), 0,
                               stream, ctx, reps, n, c2, pr, ec, b2, b3, cost, restored, admitted,
                               k0, kn, K);
        else if (lpw == 40)
            hipLaunchKernelGGL((replay_merge_kernel<NW, 40, false>), dim3(blocks), dim3(kWave), 0,
                               stream, ctx, reps, n, c2, pr, ec, b2, b3, cost, restored, admitted,
                               k0, kn, K);
        else if (ctx != nullptr)
            hipLaunchKernelGGL((replay_merge_kernel<NW, 64, true>), dim3(blocks), dim3(kWave), 0,
                               stream, ctx, reps, n, c2, pr, ec, b2, b3, cost, restored, admitted,
                               k0, kn, K);
        else
            hipLaunchKernelGGL((replay_merge_kernel<NW, 64, false>), dim3(blocks), dim3(kWave), 0,
                               stream, ctx, reps, n, c2, pr, ec, b2, b3, cost, restored, admitted,
                               k0, kn, K);
        hipError_t err = hipGetLastError();
        if (err != hipSuccess) return err;
    }
    return hipGetLastError();
}

hipError_t launch_replay(const double *arrival, const double *wait, const int32_t *ctx,
                         int64_t reps, int64_t n, const double *h_t2, int K, int64_t c2, double b2,
                         double b3, void *ws, double *cost, int64_t *restored,
                         int64_t *admitted, int *status, hipStream_t stream)
{
    auto a256 = [](size_t x) { return (x + 255) & ~(size_t)255; };
    const int kc = replay_timer_chunk(reps, n, K);
    char *p = static_cast<char *>(ws);
    uint32_t *pr = reinterpret_cast<uint32_t *>(p);
    p += a256(sizeof(uint32_t) * reps * n);
    uint16_t *ec = reinterpret_cast<uint16_t *>(p);
    p += a256(sizeof(uint16_t) * kc * reps * n);
    double *t2 = reinterpret_cast<double *>(p);
    hipError_t err = launch_upload(t2, h_t2, K, stream);
    if (err != hipSuccess) return err;
    const int ni = (int)n;
    if (n <= 1024)
        return launch_replay_n<1024, 32>(arrival, wait, ctx, reps, ni, t2, K, c2, b2, b3, pr, ec,
                                         cost, restored, admitted, status, stream);
    if (n <= 4096)
        return launch_replay_n<4096, 128>(arrival, wait, ctx, reps, ni, t2, K, c2, b2, b3, pr, ec,
                                          cost, restored, admitted, status, stream);
    return launch_replay_n<kReplayMaxN, 256>(arrival, wait, ctx, reps, ni, t2, K, c2, b2, b3, pr,
                                             ec, cost, restored, admitted, status, stream);
}

}  // namespace kvr
