// Recompute share of the grid: R3(r, e) = sum over resample r of T * [w > e]
// for every deadline e = fl(t1 + t2) of the policy grid (the b3 branch of
// Eq. 1 under a one-shot host timer).  R3 does not depend on the load, and
// it is an integer, so it is counted here once per (resample, deadline)
// instead of being tested inside the grid kernel for every (sample, policy).
//
// Counting through deadline bins: let c(x) be the number of grid deadlines
// strictly below x.  For a policy with deadline e_p and lb_p = c(e_p),
// w > e_p holds exactly when c(w) > lb_p (every deadline below e_p is below
// w, and so is e_p; conversely w <= e_p leaves no deadline below w that is
// not below e_p).  So with hist[b] = sum of T over draws whose wait has
// c(w) = b, R3(e_p) = sum_{b > lb_p} hist[b], a suffix sum.  The deadlines
// are non-decreasing along each t1 row (t2 ascending) and along each t2
// column (t1 ascending), rounding being monotone, so c(x) is a sum of one
// binary search per row or per column, whichever are fewer: at most
// min(K1, K2) <= 4,096 searches per item, and no sort is needed.  A finite
// wait has c(w) <= F, the number of finite deadlines, and bin 0 never enters
// a suffix that is read (lb_p + 1 >= 1), so only bins 1..F are kept, stored
// at b - 1: S[r][x] = R3 of any policy with lb_p = x, and R3 = 0 when
// lb_p >= F (an infinite deadline).
//
// The sums are exact unsigned 64-bit integers: neither the atomics' order nor
// the reduction tree can change them, and they equal the grid kernel's former
// fp64 accumulation of the same integers bit for bit.
#include "kvr_device.h"

namespace kvr {

constexpr int kR3Threads = 1024;
constexpr int kR3BinsPerPass = 16384;  // 128 KiB of LDS counters per pass
constexpr int kR3BinsSmall = 2048;     // 16 KiB: grids with few deadlines
constexpr int kR3Unroll = 4;           // draws per thread and step, fetched together
constexpr int kR3LdsTable = 4096;      // timer-table entries staged in LDS (32 KiB)

// Number of grid deadlines fl(t1[a] + t2[k]) strictly below x, from timer
// tables t1[K1] and t2[K2] (in LDS when they fit there).
__device__ int32_t deadlines_below(const double *t1v, int K1, const double *t2v, int K2, double x)
{
    int32_t c = 0;
    if (K1 <= K2) {
        for (int a = 0; a < K1; ++a) {
            const double t1 = t1v[a];
            int lo = 0, hi = K2;   // first k with t1 + t2[k] >= x
            while (lo < hi) {
                const int mid = (lo + hi) >> 1;
                if (t1 + t2v[mid] < x) lo = mid + 1;
                else hi = mid;
            }
            c += lo;
        }
    } else {
        for (int k = 0; k < K2; ++k) {
            const double t2 = t2v[k];
            int lo = 0, hi = K1;   // first a with t1[a] + t2 >= x
            while (lo < hi) {
                const int mid = (lo + hi) >> 1;
                if (t1v[mid] + t2 < x) lo = mid + 1;
                else hi = mid;
            }
            c += lo;
        }
    }
    return c;
}

// Items 0..n-1: per base sample, one 16-byte record of its wait's bin, its
// (clamped) context size and its wait, read as fetch_sample reads them (bad
// waits count as 0, contexts below 1 as 1; the grid kernel flags both), so
// that the passes over the draws gather one record per draw.  Items
// n..n+P-1: per policy f = a*K2 + k, the number of grid deadlines strictly
// below its own.
__global__ void __launch_bounds__(256) r3_bins_kernel(const double *__restrict__ w,
                                                      const int32_t *__restrict__ T, int64_t n,
                                                      Tables tb, SampleRec *__restrict__ rec,
                                                      int32_t *__restrict__ lb)
{
    // the timer tables in LDS when both fit (every item searches them)
    __shared__ double lt[kR3LdsTable];
    const bool in_lds = tb.K1 + tb.K2 <= kR3LdsTable;   // uniform
    const double *t1v = tb.t1, *t2v = tb.t2;
    if (in_lds) {
        for (int q = threadIdx.x; q < tb.K1 + tb.K2; q += blockDim.x)
            lt[q] = q < tb.K1 ? tb.t1[q] : tb.t2[q - tb.K1];
        __syncthreads();
        t1v = lt;
        t2v = lt + tb.K1;
    }
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t P = (int64_t)tb.K1 * tb.K2;
    if (i < n) {
        double x = w[i];
        const uint64_t bits = (uint64_t)__double_as_longlong(x);
        if (!(bits < 0x7ff0000000000000ull || bits == 0x8000000000000000ull)) x = 0.0;
        int32_t t = T[i];
        if (t < 1) t = 1;
        SampleRec v;
        v.bin = deadlines_below(t1v, tb.K1, t2v, tb.K2, x + 0.0);
        v.T = t;
        v.w = x + 0.0;
        rec[i] = v;
    } else if (i - n < P) {
        const int64_t f = i - n;
        const int a = (int)(f / tb.K2), k = (int)(f % tb.K2);
        lb[f] = deadlines_below(t1v, tb.K1, t2v, tb.K2, t1v[a] + t2v[k]);
    }
}

__global__ void __launch_bounds__(256) r3_zero_kernel(unsigned long long *__restrict__ p,
                                                      int64_t count)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < count) p[i] = 0ull;
}

// One block per (resample, split of its draws): histogram of T over the
// stored bins 1..nbins (index b - 1) in LDS, one pass per range of PER bins
// (a small PER for grids with few deadlines leaves room for more resident
// blocks).  A resample with one split owns its row of hist and stores it;
// several splits add into a zeroed row.
template <int PER, bool XG>
__global__ void __launch_bounds__(kR3Threads) r3_hist_kernel(
    const int32_t *__restrict__ idx, int64_t n, int64_t m, const SampleRec *__restrict__ rec,
    int64_t nbins, int nsplit, int64_t split_len, unsigned long long *__restrict__ hist,
    const double *__restrict__ t1p, double *__restrict__ X, double *__restrict__ G, int *status)
{
    __shared__ unsigned long long lh[PER];
    constexpr int64_t per = PER;
    const int64_t r = blockIdx.x / nsplit;
    const int s = (int)(blockIdx.x % nsplit);
    const int64_t j0 = (int64_t)s * split_len;
    const int64_t j1 = (j0 + split_len < m) ? j0 + split_len : m;
    const int64_t B = blockDim.x;
    unsigned long long *row = hist + r * nbins;
    // XG (one t1 timer, one block per resample): X = sum T*min(w, t1) and
    // G = sum T*[w > t1] over the resample's draws, formed in the first pass
    // in each thread's draw order, then across the block in a fixed order
    double xs = 0.0, gs = 0.0;
    const double t1 = XG ? t1p[0] : 0.0;
    for (int64_t b0 = 0; b0 < nbins; b0 += per) {
        const int64_t nb = (nbins - b0 < per) ? nbins - b0 : per;
        for (int64_t x = threadIdx.x; x < nb; x += blockDim.x) lh[x] = 0ull;
        __syncthreads();
        for (int64_t j = j0 + threadIdx.x; j < j1; j += kR3Unroll * B) {
            // the kR3Unroll draws are loaded unconditionally (a position past
            // the split re-reads the split's last one and is dropped below)
            // and checked with selects and one branch for all, so the index
            // loads, and then the gathers, are in flight together
            int32_t raw[kR3Unroll];
            bool inr[kR3Unroll];
#pragma unroll
            for (int u = 0; u < kR3Unroll; ++u) {
                const int64_t jj = j + u * B;
                inr[u] = jj < j1;
                const int64_t jc = inr[u] ? jj : j1 - 1;
                raw[u] = (idx != nullptr) ? idx[r * m + jc] : (int32_t)jc;
            }
            bool bad = false;
            int32_t ic[kR3Unroll];
#pragma unroll
            for (int u = 0; u < kR3Unroll; ++u) {
                const bool out = raw[u] < 0 || (int64_t)raw[u] >= n;
                bad = bad || (inr[u] && out);
                ic[u] = out ? 0 : raw[u];               // a bad draw counts as sample 0
            }
            if (bad) flag_domain(status);
            SampleRec bt[kR3Unroll];
#pragma unroll
            for (int u = 0; u < kR3Unroll; ++u) {
                bt[u] = rec[ic[u]];
                if (!inr[u]) {   // bin 0 is never counted; T = 0 adds nothing to X, G
                    bt[u].bin = 0;
                    bt[u].T = 0;
                }
            }
#pragma unroll
            for (int u = 0; u < kR3Unroll; ++u) {
                const int64_t b = (int64_t)bt[u].bin - 1 - b0;   // bin 0 gives b < 0
                if (b >= 0 && b < nb) atomicAdd(&lh[b], (unsigned long long)bt[u].T);
            }
            if (XG && b0 == 0) {
#pragma unroll
                for (int u = 0; u < kR3Unroll; ++u) {
                    const double T = (double)bt[u].T;
                    xs = fma(T, fmin(bt[u].w, t1), xs);
                    gs += (bt[u].w > t1) ? T : 0.0;
                }
            }
        }
        __syncthreads();
        for (int64_t x = threadIdx.x; x < nb; x += blockDim.x) {
            const unsigned long long v = lh[x];
            if (nsplit == 1) row[b0 + x] = v;
            else if (v != 0ull) atomicAdd(&row[b0 + x], v);
        }
        __syncthreads();
    }
    if (XG) {   // butterfly within each wave, then the waves in order
        __shared__ double wx[kR3Threads / kWave], wg[kR3Threads / kWave];
        xs = wave_sum(xs);
        gs = wave_sum(gs);
        const int lane = threadIdx.x % kWave, wv = threadIdx.x / kWave;
        if (lane == 0) {
            wx[wv] = xs;
            wg[wv] = gs;
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            double a = 0.0, g = 0.0;
            for (int q = 0; q < kR3Threads / kWave; ++q) {
                a += wx[q];
                g += wg[q];
            }
            X[r] = a;
            G[r] = g;
        }
    }
}

bool r3_fuses_xg(int K1, int nsplit, int64_t nbins)
{
    return K1 == 1 && nsplit == 1 && nbins > 0;   // with no finite deadline the pass is skipped
}

// One block per resample: hist row -> suffix sums S[b] = sum_{b' >= b} hist[b'],
// in place, chunk by chunk from the top bin down.
__global__ void __launch_bounds__(kR3Threads) r3_suffix_kernel(unsigned long long *__restrict__ hist,
                                                               int64_t nbins)
{
    __shared__ unsigned long long wsum[kR3Threads / kWave];
    __shared__ unsigned long long carry_s;
    unsigned long long *row = hist + (int64_t)blockIdx.x * nbins;
    const int lane = threadIdx.x % kWave, wv = threadIdx.x / kWave;
    constexpr int nw = kR3Threads / kWave;
    if (threadIdx.x == 0) carry_s = 0ull;
    __syncthreads();
    for (int64_t top = nbins; top > 0; top -= kR3Threads) {
        // element handled by this thread: position top-1-tid (descending)
        const int64_t pos = top - 1 - threadIdx.x;
        unsigned long long v = (pos >= 0) ? row[pos] : 0ull;
        // inclusive scan in descending-position order within the wave
        for (int off = 1; off < kWave; off <<= 1) {
            const unsigned long long o = __shfl_up(v, off, kWave);
            if (lane >= off) v += o;
        }
        if (lane == kWave - 1) wsum[wv] = v;
        __syncthreads();
        unsigned long long before = carry_s;
        for (int q = 0; q < wv; ++q) before += wsum[q];
        v += before;
        if (pos >= 0) row[pos] = v;
        __syncthreads();
        if (threadIdx.x == 0) {
            unsigned long long t = carry_s;
            for (int q = 0; q < nw; ++q) t += wsum[q];
            carry_s = t;
        }
        __syncthreads();
    }
}

int r3_splits(int64_t R, int64_t m, int64_t *split_len)
{
    // enough blocks to cover the chip when there are few resamples, but never
    // fewer than 4,096 draws per block
    int64_t ns = (512 + R - 1) / R;
    const int64_t cap = (m + 4095) / 4096;
    if (ns > cap) ns = cap;
    if (ns < 1) ns = 1;
    *split_len = (m + ns - 1) / ns;
    return (int)ns;
}

hipError_t launch_r3(const SampleSrc &src, int64_t R, const Tables &tb, const R3Ws &ws,
                     double *X, double *G, int *status, hipStream_t stream)
{
    const int64_t P = (int64_t)tb.K1 * tb.K2;
    hipLaunchKernelGGL(r3_bins_kernel, dim3((unsigned)((src.n + P + 255) / 256)), dim3(256), 0,
                       stream, src.w, src.T, src.n, tb, ws.rec, ws.lb);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    if (ws.nbins == 0) return hipSuccess;   // every deadline infinite: R3 = 0
    if (ws.nsplit > 1) {
        const int64_t cnt = R * ws.nbins;
        hipLaunchKernelGGL(r3_zero_kernel, dim3((unsigned)((cnt + 255) / 256)), dim3(256), 0,
                           stream, ws.S, cnt);
        if ((err = hipGetLastError()) != hipSuccess) return err;
    }
    const bool xg = X != nullptr;   // r3_fuses_xg held on the host
    const double *t1 = tb.t1;
    const dim3 grid((unsigned)(R * ws.nsplit)), block(kR3Threads);
    if (ws.nbins <= kR3BinsSmall && xg)
        hipLaunchKernelGGL((r3_hist_kernel<kR3BinsSmall, true>), grid, block, 0, stream, src.idx,
                           src.n, src.m, ws.rec, ws.nbins, ws.nsplit, ws.split_len, ws.S, t1, X,
                           G, status);
    else if (ws.nbins <= kR3BinsSmall)
        hipLaunchKernelGGL((r3_hist_kernel<kR3BinsSmall, false>), grid, block, 0, stream, src.idx,
                           src.n, src.m, ws.rec, ws.nbins, ws.nsplit, ws.split_len, ws.S, t1,
                           nullptr, nullptr, status);
    else if (xg)
        hipLaunchKernelGGL((r3_hist_kernel<kR3BinsPerPass, true>), grid, block, 0, stream, src.idx,
                           src.n, src.m, ws.rec, ws.nbins, ws.nsplit, ws.split_len, ws.S, t1, X,
                           G, status);
    else
        hipLaunchKernelGGL((r3_hist_kernel<kR3BinsPerPass, false>), grid, block, 0, stream,
                           src.idx, src.n, src.m, ws.rec, ws.nbins, ws.nsplit, ws.split_len, ws.S,
                           t1, nullptr, nullptr, status);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    hipLaunchKernelGGL(r3_suffix_kernel, dim3((unsigned)R), dim3(kR3Threads), 0, stream, ws.S,
                       ws.nbins);
    return hipGetLastError();
}

}  // namespace kvr
