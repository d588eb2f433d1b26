// The brute-force grid of one sample with few GPU-tier timers and few
// deadlines, in four launches instead of ten: table staging, one pre-pass
// over the samples, the grid kernel (blocks of several waves that add their
// splits in LDS), and one finalize.  Small grids are bound by their launches, not by
// their arithmetic, so the load-independent sums of Eq. 1 that the large path
// computes in six launches (X and G per t1, the recompute share R3 per
// deadline; see kvr_r3.hip for the deadline bins) are gathered here in one.
//
// Pre-pass: block b < nsb takes kSmallPer consecutive samples.  Each sample's
// deadline bin c(w) (the number of grid deadlines below it, found by binary
// searches in LDS copies of the timer tables) adds T to an LDS histogram of
// bins 1..F, stored as the block's row hist[b][F]; X(t1) = sum T*min(w, t1)
// and G(t1) = sum T*[w > t1] are reduced over the block in a fixed order into
// partials xgp[b][a][2].  Blocks from nsb on give each policy its lb = c(e).
// Finalize: one thread per (policy, load) adds the grid kernel's split
// partials in split order and reads X, G and R3 from what its block formed in
// LDS: the rows added in block order, the histogram's suffix sums.
#include "kvr_device.h"

namespace kvr {

constexpr int kSmallThreads = 256;
constexpr int kSmallSPT = 4;                                   // samples per thread
constexpr int kSmallPer = kSmallThreads * kSmallSPT;           // samples per block
constexpr int kSmallMaxK1 = 8;
constexpr int kSmallMaxK2 = 4096;
constexpr int kSmallMaxBins = 4096;
constexpr int kFinFlight = 16;   // finalize: histogram rows and split partials in flight per thread

int small_sample_blocks(int64_t n) { return (int)((n + kSmallPer - 1) / kSmallPer); }

// Every finalize block adds all pre-pass rows of the histogram: kept to
// 65,536 words (65,536 waits with 1,024 deadlines, or 256 blocks of 256).
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

__global__ void __launch_bounds__(kSmallThreads) small_prep_kernel(
    const double *__restrict__ w, const int32_t *__restrict__ T, int64_t n, Tables tb, int nsb,
    int64_t nbins, unsigned long long *__restrict__ hist, int32_t *__restrict__ lb,
    double *__restrict__ xgp, int *status)
{
    __shared__ double lt1[kSmallMaxK1];
    __shared__ double lt2[kSmallMaxK2];
    __shared__ unsigned long long lh[kSmallMaxBins];
    __shared__ double red[kSmallThreads][2 * kSmallMaxK1];
    const int K1 = tb.K1, K2 = tb.K2;
    for (int i = threadIdx.x; i < K2; i += kSmallThreads) lt2[i] = tb.t2[i];
    if (threadIdx.x < K1) lt1[threadIdx.x] = tb.t1[threadIdx.x];
    if ((int)blockIdx.x >= nsb) {   // policies: lb = deadlines below their own
        __syncthreads();
        const int64_t f = (int64_t)(blockIdx.x - nsb) * kSmallThreads + threadIdx.x;
        if (f < (int64_t)K1 * K2) {
            const int a = (int)(f / K2), k = (int)(f % K2);
            lb[f] = small_bin(lt1, K1, lt2, K2, lt1[a] + lt2[k]);
        }
        return;
    }
    for (int64_t i = threadIdx.x; i < nbins; i += kSmallThreads) lh[i] = 0ull;
    __syncthreads();
    double xs[kSmallMaxK1], gs[kSmallMaxK1];
#pragma unroll
    for (int a = 0; a < kSmallMaxK1; ++a) {
        xs[a] = 0.0;
        gs[a] = 0.0;
    }
    const int64_t j0 = (int64_t)blockIdx.x * kSmallPer;
    bool bad = false;
#pragma unroll
    for (int q = 0; q < kSmallSPT; ++q) {
        const int64_t j = j0 + q * kSmallThreads + threadIdx.x;
        if (j >= n) break;
        double x = w[j];
        int32_t t = T[j];
        // finite and >= 0 (or -0.0), tested on the bits; the grid kernel reads
        // the same sample and replaces it the same way
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
        const int32_t b = small_bin(lt1, K1, lt2, K2, x);
        if (b >= 1) atomicAdd(&lh[b - 1], (unsigned long long)t);   // bin 0 is never read
#pragma unroll
        for (int a = 0; a < kSmallMaxK1; ++a) {
            if (a < K1) {
                xs[a] = fma(Td, fmin(x, lt1[a]), xs[a]);
                gs[a] += (x > lt1[a]) ? Td : 0.0;
            }
        }
    }
    if (bad) flag_domain(status);
    // X and G: fixed-order tree over the block
#pragma unroll
    for (int a = 0; a < kSmallMaxK1; ++a) {
        red[threadIdx.x][a] = xs[a];
        red[threadIdx.x][kSmallMaxK1 + a] = gs[a];
    }
    __syncthreads();
    for (int stride = kSmallThreads / 2; stride > 0; stride /= 2) {
        if ((int)threadIdx.x < stride) {
            for (int a = 0; a < K1; ++a) {
                red[threadIdx.x][a] += red[threadIdx.x + stride][a];
                red[threadIdx.x][kSmallMaxK1 + a] += red[threadIdx.x + stride][kSmallMaxK1 + a];
            }
        }
        __syncthreads();
    }
    if ((int)threadIdx.x < 2 * K1) {
        const int a = (int)threadIdx.x % K1, which = (int)threadIdx.x / K1;
        xgp[((int64_t)blockIdx.x * K1 + a) * 2 + which] = red[0][which * kSmallMaxK1 + a];
    }
    // this block's row of the histogram (integer sums; rows are added in the
    // finalize, so no block waits on another and no atomics contend)
    for (int64_t i = threadIdx.x; i < nbins; i += kSmallThreads) hist[(int64_t)blockIdx.x * nbins + i] = lh[i];
}

// One thread per (policy f, load l).  Partials [split group][tile][LT][P]
// from the grid kernel (one resample; a block's splits already added).  Each
// block first forms, in LDS, the histogram (rows added in block order), its
// suffix sums and X, G per t1 row (partials added in block order).
__global__ void __launch_bounds__(kSmallThreads) small_finalize_kernel(
    GridPlan plan, Tables tb, PriceDev pr, double md, int nsb, int64_t nbins,
    const unsigned long long *__restrict__ hist, const int32_t *__restrict__ lb,
    const double *__restrict__ xgp, const double *__restrict__ partials,
    double *__restrict__ cost_out)
{
    __shared__ unsigned long long S[kSmallMaxBins];
    __shared__ unsigned long long wtot[kSmallThreads / kWave];
    __shared__ double xg[kSmallMaxK1][2];
    for (int64_t i = threadIdx.x; i < nbins; i += kSmallThreads) {
        unsigned long long v = 0ull;
        int b = 0;
        for (; b + kFinFlight <= nsb; b += kFinFlight) {   // rows in flight, added in block order
            unsigned long long u[kFinFlight];
#pragma unroll
            for (int q = 0; q < kFinFlight; ++q) u[q] = hist[(int64_t)(b + q) * nbins + i];
#pragma unroll
            for (int q = 0; q < kFinFlight; ++q) v += u[q];
        }
        for (; b < nsb; ++b) v += hist[(int64_t)b * nbins + i];
        S[i] = v;
    }
    if ((int)threadIdx.x < 2 * tb.K1) {
        const int a = (int)threadIdx.x % tb.K1, which = (int)threadIdx.x / tb.K1;
        double v = 0.0;
        int b = 0;
        for (; b + kFinFlight <= nsb; b += kFinFlight) {   // in flight, added in block order
            double u[kFinFlight];
#pragma unroll
            for (int q = 0; q < kFinFlight; ++q) u[q] = xgp[((int64_t)(b + q) * tb.K1 + a) * 2 + which];
#pragma unroll
            for (int q = 0; q < kFinFlight; ++q) v += u[q];
        }
        for (; b < nsb; ++b) v += xgp[((int64_t)b * tb.K1 + a) * 2 + which];
        xg[a][which] = v;
    }
    __syncthreads();
    // suffix sums S[x] = sum of bins x.. (stored index), in chunks of one
    // value per thread from the top down, in place
    unsigned long long carry = 0;
    const int lane = threadIdx.x % kWave, wv = threadIdx.x / kWave;
    for (int64_t top = nbins; top > 0; top -= kSmallThreads) {
        const int64_t pos = top - 1 - threadIdx.x;
        unsigned long long v = pos >= 0 ? S[pos] : 0ull;
        for (int off = 1; off < kWave; off <<= 1) {
            const unsigned long long o = __shfl_up(v, off, kWave);
            if (lane >= off) v += o;
        }
        if (lane == kWave - 1) wtot[wv] = v;
        __syncthreads();
        unsigned long long before = carry, all = carry;
        for (int q = 0; q < kSmallThreads / kWave; ++q) {
            if (q < wv) before += wtot[q];
            all += wtot[q];
        }
        if (pos >= 0) S[pos] = v + before;
        carry = all;
        __syncthreads();
    }
    const int64_t P = (int64_t)tb.K1 * tb.K2;
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (gid >= P * tb.L) return;
    const int64_t f = gid % P;
    const int l = (int)(gid / P);
    const int a = (int)(f / tb.K2);
    const double x = xg[a][0], g = xg[a][1];
    const int32_t xb = lb[f];
    const double r3 = (xb < nbins) ? (double)S[xb] : 0.0;
    const double base = pr.a1 * x + (pr.b2 * (g - r3) + pr.b3 * r3);
    const int64_t row = l;   // tile l / LT, value l % LT
    const int64_t slice = (int64_t)plan.ntiles * plan.LT * P;
    const int64_t nsg = (plan.nsplit + plan.wpb - 1) / plan.wpb;
    const double *p0 = partials + row * P + f;
    double s = p0[0];
    int64_t q = 1;
    for (; q + kFinFlight <= nsg; q += kFinFlight) {   // loads in flight, added in split order
        double v[kFinFlight];
#pragma unroll
        for (int u = 0; u < kFinFlight; ++u) v[u] = p0[(q + u) * slice];
#pragma unroll
        for (int u = 0; u < kFinFlight; ++u) s += v[u];
    }
    for (; q < nsg; ++q) s += p0[q * slice];
    cost_out[(int64_t)l * P + f] = (base + s) / md;
}

hipError_t launch_small_prep(const double *w, const int32_t *T, int64_t n, const Tables &tb,
                             int64_t nbins, unsigned long long *hist, int32_t *lb, double *xgp,
                             int *status, hipStream_t stream)
{
    const int nsb = small_sample_blocks(n);
    const int64_t P = (int64_t)tb.K1 * tb.K2;
    const int64_t npb = (P + kSmallThreads - 1) / kSmallThreads;
    hipLaunchKernelGGL(small_prep_kernel, dim3((unsigned)(nsb + npb)), dim3(kSmallThreads), 0,
                       stream, w, T, n, tb, nsb, nbins, hist, lb, xgp, status);
    return hipGetLastError();
}

hipError_t launch_small_finalize(const GridPlan &plan, const Tables &tb, const PriceDev &pr,
                                 int64_t m, int64_t nbins, const unsigned long long *hist,
                                 const int32_t *lb, const double *xgp, const double *partials,
                                 double *cost_out, hipStream_t stream)
{
    const int64_t items = (int64_t)tb.K1 * tb.K2 * tb.L;
    hipLaunchKernelGGL(small_finalize_kernel, dim3((unsigned)((items + kSmallThreads - 1) / kSmallThreads)),
                       dim3(kSmallThreads), 0, stream, plan, tb, pr, (double)m,
                       small_sample_blocks(m), nbins, hist, lb, xgp, partials, cost_out);
    return hipGetLastError();
}

}  // namespace kvr
