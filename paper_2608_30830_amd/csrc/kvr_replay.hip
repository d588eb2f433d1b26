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
// monotone streams -- resumes, ordered by fl(arrival + wait) (one sort per
// request sequence, shared by every timer), and expiries, which follow arrival
// order because fl(arrival + t2) is monotone in the arrival.  One lane runs one
// (sequence, timer) replay as a three-way merge of arrivals, resumes and
// expiries, keeping an admitted bit per request; a departure frees a slot only
// if its request was admitted and left by that stream.
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

// One block per request sequence: validate the row, then bitonic-sort
// (fl(arrival + wait), index) in LDS and write the sorted times and indices.
__global__ void __launch_bounds__(kReplaySortThreads) replay_sort_kernel(
    const double *__restrict__ arrival, const double *__restrict__ wait,
    const int32_t *__restrict__ ctx, int n, double *__restrict__ stime,
    int32_t *__restrict__ sidx, int *status)
{
    __shared__ double key[kReplayMaxN];
    __shared__ int32_t idx[kReplayMaxN];
    const int64_t row = blockIdx.x;
    const double *A = arrival + row * n;
    const double *W = wait + row * n;
    int np2 = 1;
    while (np2 < n) np2 <<= 1;
    for (int i = threadIdx.x; i < np2; i += blockDim.x) {
        if (i < n) {
            const double a = A[i], w = W[i];
            const uint64_t ba = (uint64_t)__double_as_longlong(a);
            const uint64_t bw = (uint64_t)__double_as_longlong(w);
            // finite and >= 0 (or -0.0), arrivals non-decreasing, contexts >= 1
            bool bad = !(ba < 0x7ff0000000000000ull || ba == 0x8000000000000000ull) ||
                       !(bw < 0x7ff0000000000000ull || bw == 0x8000000000000000ull);
            if (i > 0 && !(A[i - 1] <= a)) bad = true;
            if (ctx != nullptr && ctx[row * n + i] < 1) bad = true;
            if (bad) flag_domain(status);
            key[i] = a + w;
            idx[i] = i;
        } else {
            key[i] = INFINITY;
            idx[i] = 0x7fffffff;
        }
    }
    __syncthreads();
    for (int size = 2; size <= np2; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int i = threadIdx.x; i < np2; i += blockDim.x) {
                const int j = i ^ stride;
                if (j > i) {
                    const bool up = (i & size) == 0;
                    const bool gt = key_less(key[j], idx[j], key[i], idx[i]);
                    if (gt == up) {
                        const double tk = key[i];
                        key[i] = key[j];
                        key[j] = tk;
                        const int32_t ti = idx[i];
                        idx[i] = idx[j];
                        idx[j] = ti;
                    }
                }
            }
            __syncthreads();
        }
    }
    for (int i = threadIdx.x; i < n; i += blockDim.x) {
        stime[row * n + i] = key[i];
        sidx[row * n + i] = idx[i];
    }
}

// One lane per (sequence, timer): the three-way merge.
__global__ void __launch_bounds__(256) replay_merge_kernel(
    const double *__restrict__ arrival, const double *__restrict__ wait,
    const int32_t *__restrict__ ctx, int64_t reps, int n, const double *__restrict__ t2s, int K,
    int64_t c2, const double *__restrict__ stime, const int32_t *__restrict__ sidx,
    uint32_t *__restrict__ bits, double b2, double b3, double *__restrict__ cost,
    int64_t *__restrict__ restored_out, int64_t *__restrict__ admitted_out)
{
    const int64_t sim = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (sim >= reps * K) return;
    const int64_t row = sim / K;
    const double t2 = t2s[sim % K];
    const double *A = arrival + row * n;
    const double *W = wait + row * n;
    const int32_t *C = ctx ? ctx + row * n : nullptr;
    const double *ST = stime + row * n;
    const int32_t *SI = sidx + row * n;
    const int nwords = (n + 31) / 32;
    uint32_t *B = bits + sim * nwords;

    int64_t occ = 0, restored = 0, admitted = 0, total = 0;
    int ir = 0, ie = 0;
    uint32_t word = 0;   // admitted bits of requests 32*(j/32) .. j-1
    auto was_admitted = [&](int i, int j) -> bool {
        const uint32_t w32 = ((i >> 5) == (j >> 5)) ? word : B[i >> 5];
        return (w32 >> (i & 31)) & 1u;
    };
    for (int j = 0; j < n; ++j) {
        const double a = A[j];
        // resumes at or before a (only requests that arrived before j)
        while (ir < n) {
            const int i = SI[ir];
            if (i >= j || ST[ir] > a) break;
            if (W[i] <= t2 && was_admitted(i, j)) --occ;
            ++ir;
        }
        // expiries at or before a, in arrival order
        while (ie < j) {
            if (A[ie] + t2 > a) break;
            if (W[ie] > t2 && was_admitted(ie, j)) --occ;
            ++ie;
        }
        int32_t T = C ? C[j] : 1;
        if (T < 1) T = 1;
        total += T;
        if (occ < c2) {
            ++occ;
            ++admitted;
            word |= 1u << (j & 31);
            if (W[j] <= t2) restored += T;
        }
        if ((j & 31) == 31 || j == n - 1) {
            B[j >> 5] = word;
            word = 0;
        }
    }
    cost[sim] = (b2 * (double)restored + b3 * (double)(total - restored)) / (double)n;
    if (restored_out) restored_out[sim] = restored;
    if (admitted_out) admitted_out[sim] = admitted;
}

size_t replay_ws_bytes(int64_t reps, int64_t n, int K)
{
    auto a256 = [](size_t x) { return (x + 255) & ~(size_t)255; };
    const int64_t nwords = (n + 31) / 32;
    return a256(sizeof(double) * reps * n) + a256(sizeof(int32_t) * reps * n) +
           a256(sizeof(uint32_t) * reps * K * nwords) + a256(sizeof(double) * K);
}

hipError_t launch_replay(const double *arrival, const double *wait, const int32_t *ctx,
                         int64_t reps, int64_t n, const double *h_t2, int K, int64_t c2, double b2,
                         double b3, void *ws, double *cost, int64_t *restored,
                         int64_t *admitted, int *status, hipStream_t stream)
{
    auto a256 = [](size_t x) { return (x + 255) & ~(size_t)255; };
    char *p = static_cast<char *>(ws);
    double *stime = reinterpret_cast<double *>(p);
    p += a256(sizeof(double) * reps * n);
    int32_t *sidx = reinterpret_cast<int32_t *>(p);
    p += a256(sizeof(int32_t) * reps * n);
    uint32_t *bits = reinterpret_cast<uint32_t *>(p);
    p += a256(sizeof(uint32_t) * reps * K * ((n + 31) / 32));
    double *t2 = reinterpret_cast<double *>(p);
    hipError_t err = launch_upload(t2, h_t2, K, stream);
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(replay_sort_kernel, dim3((unsigned)reps), dim3(kReplaySortThreads), 0,
                       stream, arrival, wait, ctx, (int)n, stime, sidx, status);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    const int64_t sims = reps * K;
    hipLaunchKernelGGL(replay_merge_kernel, dim3((unsigned)((sims + 255) / 256)), dim3(256), 0,
                       stream, arrival, wait, ctx, reps, (int)n, t2, K, c2, stime, sidx, bits, b2,
                       b3, cost, restored, admitted);
    return hipGetLastError();
}

}  // namespace kvr
