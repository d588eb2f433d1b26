// Bootstrap selection by the multiplicity-count closed form, a second method
// beside the brute-force grid (Eq. 1 and Eq. 3 integrated over sorted waits,
// as in the SORTED path, with bootstrap multiplicities as weights).
//
// With the base waits sorted once and, for one resample, c_i the number of
// times it draws base sample i, let N(x) = sum_{w_i <= x} c_i T_i and
// S(x) = sum_{w_i <= x} c_i T_i w_i, Ttot = N(inf).  Then for policy
// (t1, t2, lambda), e = t1 + t2:
//   m*C = a1*[S(t1) + t1*(Ttot - N(t1))]
//       + a2*[(S(e) - S(t1)) - t1*(N(e) - N(t1)) + (e - t1)*(Ttot - N(e))]
//       + b2*(N(e) - N(t1)) + b3*(Ttot - N(e)),
// dropping (e - t1)*(Ttot - N(e)) when e = +inf.  Per resample the work is a
// weighted histogram of its m draws over sorted positions, one prefix scan of
// length n, and O(1) per (policy, load): O(m + n + P*L) instead of the brute
// force's O(m*P*L).  N is exact (unsigned 64-bit); S, and so the costs, round
// differently from the brute force's per-sample sums, so the two methods
// agree within rounding and their selections up to rounding-level ties.
//
// Per batch of resamples: factored_hist_kernel (one block per resample,
// 32-bit LDS counters of multiplicity over ranges of sorted positions),
// factored_scan_kernel (one block per resample: weights c_i T_i and the N and
// S prefix sums in place), factored_policy_kernel (one block per (resample,
// tile of 32 loads): every policy, fused arg-min on the numerators m*C).
#include "kvr_device.h"
#include "kvr_factored.h"

namespace kvr {

constexpr int kFThreads = 1024;
constexpr int kFRanksPerPass = 32768;   // 128 KiB of 32-bit LDS counters per pass
constexpr int kFScanPer = 4;            // consecutive positions per thread in the scan
constexpr int kFLoads = 32;             // loads per policy-kernel block
constexpr int kFPolThreads = 256;

// Per sorted position k: the sorted wait and the context size there (below
// 1 counts as 1; sort_prep_kernel has flagged it); per base sample: its
// sorted position.
__global__ void __launch_bounds__(256) factored_rank_kernel(const uint64_t *__restrict__ skeys,
                                                            const int32_t *__restrict__ perm,
                                                            const int32_t *__restrict__ T, int64_t n,
                                                            double *__restrict__ sw,
                                                            int32_t *__restrict__ Ts,
                                                            int32_t *__restrict__ rank)
{
    const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= n) return;
    const int32_t i = perm[k];
    sw[k] = __longlong_as_double((long long)skeys[k]);
    int32_t t = T[i];
    Ts[k] = t < 1 ? 1 : t;
    rank[i] = (int32_t)k;
}

// Number of sorted waits <= x.
__device__ __forceinline__ int32_t count_le(const double *__restrict__ sw, int64_t n, double x)
{
    int64_t lo = 0, hi = n;
    while (lo < hi) {
        const int64_t mid = lo + (hi - lo) / 2;
        if (sw[mid] <= x) lo = mid + 1;
        else hi = mid;
    }
    return (int32_t)lo;
}

// Items 0..K1-1: u1[a] = #(w <= t1[a]); items K1..K1+P-1: ue[f] = #(w <= e_f).
__global__ void __launch_bounds__(256) factored_bounds_kernel(const double *__restrict__ sw,
                                                              int64_t n, Tables tb,
                                                              int32_t *__restrict__ u1,
                                                              int32_t *__restrict__ ue)
{
    const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t P = (int64_t)tb.K1 * tb.K2;
    if (g < tb.K1) {
        u1[g] = count_le(sw, n, tb.t1[g]);
    } else if (g - tb.K1 < P) {
        const int64_t f = g - tb.K1;
        const int a = (int)(f / tb.K2), k = (int)(f % tb.K2);
        ue[f] = count_le(sw, n, tb.t1[a] + tb.t2[k]);
    }
}

// One block per resample of the batch: row[1 + k] = the number of its draws of
// the base sample at sorted position k (exact: at most m < 2^31); row[0] = 0.
__global__ void __launch_bounds__(kFThreads) factored_hist_kernel(
    const int32_t *__restrict__ idx, int64_t n, int64_t m, int64_t r0,
    const int32_t *__restrict__ rank, unsigned long long *__restrict__ N, int *status)
{
    __shared__ uint32_t lh[kFRanksPerPass];
    const int64_t rb = blockIdx.x;
    const int64_t r = r0 + rb;
    unsigned long long *row = N + rb * (n + 1);
    for (int64_t k0 = 0; k0 < n; k0 += kFRanksPerPass) {
        const int64_t nk = (n - k0 < kFRanksPerPass) ? n - k0 : kFRanksPerPass;
        for (int64_t x = threadIdx.x; x < nk; x += blockDim.x) lh[x] = 0u;
        __syncthreads();
        for (int64_t j = threadIdx.x; j < m; j += blockDim.x) {
            int32_t ii = idx[r * m + j];
            if (ii < 0 || (int64_t)ii >= n) {
                flag_domain(status);
                ii = 0;
            }
            const int64_t kk = (int64_t)rank[ii] - k0;
            if (kk >= 0 && kk < nk) atomicAdd(&lh[kk], 1u);
        }
        __syncthreads();
        for (int64_t x = threadIdx.x; x < nk; x += blockDim.x) row[1 + k0 + x] = lh[x];
        __syncthreads();
    }
    if (threadIdx.x == 0) row[0] = 0ull;
}

// One block per resample of the batch: weights c_k T_k (exact) and inclusive
// prefix sums over positions 1..n of the weights (N) and of weight x sorted
// wait (S, fp64), in place.  Each thread sums kFScanPer consecutive positions
// in order, then the thread totals are scanned across the block: a fixed
// order, so S is reproducible.
__global__ void __launch_bounds__(kFThreads) factored_scan_kernel(unsigned long long *__restrict__ N,
                                                                  double *__restrict__ S,
                                                                  const double *__restrict__ sw,
                                                                  const int32_t *__restrict__ Ts,
                                                                  int64_t n)
{
    constexpr int nw = kFThreads / kWave;
    constexpr int kTile = kFThreads * kFScanPer;
    __shared__ unsigned long long wn[nw];
    __shared__ double wsd[nw];
    __shared__ unsigned long long carry_n;
    __shared__ double carry_s;
    const int64_t rb = blockIdx.x;
    unsigned long long *nrow = N + rb * (n + 1);
    double *srow = S + rb * (n + 1);
    const int lane = threadIdx.x % kWave, wv = threadIdx.x / kWave;
    if (threadIdx.x == 0) {
        carry_n = 0ull;
        carry_s = 0.0;
        srow[0] = 0.0;
    }
    __syncthreads();
    for (int64_t base = 0; base < n; base += kTile) {
        const int64_t k0 = base + (int64_t)threadIdx.x * kFScanPer;
        unsigned long long cw[kFScanPer];
        double sv[kFScanPer];
        unsigned long long tn = 0ull;
        double ts = 0.0;
#pragma unroll
        for (int q = 0; q < kFScanPer; ++q) {
            const int64_t k = k0 + q;
            const unsigned long long c = (k < n) ? nrow[1 + k] * (unsigned long long)Ts[k] : 0ull;
            cw[q] = c;
            sv[q] = (k < n) ? (double)c * sw[k] : 0.0;
            tn += c;
            ts += sv[q];
        }
        // inclusive scan of the thread totals within the wave, then across waves
        unsigned long long c = tn;
        double s = ts;
        for (int off = 1; off < kWave; off <<= 1) {
            const unsigned long long oc = __shfl_up(c, off, kWave);
            const double os = __shfl_up(s, off, kWave);
            if (lane >= off) {
                c += oc;
                s += os;
            }
        }
        if (lane == kWave - 1) {
            wn[wv] = c;
            wsd[wv] = s;
        }
        __syncthreads();
        unsigned long long bn = carry_n;
        double bs = carry_s;
        for (int q = 0; q < wv; ++q) {
            bn += wn[q];
            bs += wsd[q];
        }
        // this thread's exclusive offset, then its positions in order
        bn += c - tn;
        bs += s - ts;
#pragma unroll
        for (int q = 0; q < kFScanPer; ++q) {
            const int64_t k = k0 + q;
            bn += cw[q];
            bs += sv[q];
            if (k < n) {
                nrow[1 + k] = bn;
                srow[1 + k] = bs;
            }
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            unsigned long long t2 = carry_n;
            double s2 = carry_s;
            for (int q = 0; q < nw; ++q) {
                t2 += wn[q];
                s2 += wsd[q];
            }
            carry_n = t2;
            carry_s = s2;
        }
        __syncthreads();
    }
}

// One block per (resample of the batch, tile of kFLoads loads): every policy's
// closed-form total m*C for the tile's loads, the optional cost output, and
// the arg-min per load under the library's total order (smaller first, then
// larger flat index).  Dividing by m is monotone, so the arg-min compares the
// totals and only the selected one is divided.
__global__ void __launch_bounds__(kFPolThreads) factored_policy_kernel(
    const unsigned long long *__restrict__ N, const double *__restrict__ S, int64_t n, int64_t m,
    int64_t r0, int ntl, Tables tb, PriceDev pr, const int32_t *__restrict__ u1,
    const int32_t *__restrict__ ue, int32_t *__restrict__ best, double *__restrict__ best_cost,
    double *__restrict__ cost_out)
{
    constexpr int nw = kFPolThreads / kWave;
    __shared__ double rc[nw][kFLoads];
    __shared__ int32_t rf[nw][kFLoads];
    const int64_t rb = blockIdx.x / ntl;
    const int tile = (int)(blockIdx.x % ntl);
    const int64_t r = r0 + rb;
    const unsigned long long *nrow = N + rb * (n + 1);
    const double *srow = S + rb * (n + 1);
    const int64_t P = (int64_t)tb.K1 * tb.K2;
    const int l0 = tile * kFLoads;
    const int nl = (tb.L - l0 < kFLoads) ? tb.L - l0 : kFLoads;
    const double tot = (double)nrow[n];
    const double md = (double)m;
    double a2[kFLoads], bc[kFLoads];
    int32_t bf[kFLoads];
#pragma unroll
    for (int l = 0; l < kFLoads; ++l) {
        a2[l] = tb.a2[l0 + l];   // zero-padded to whole tiles
        bc[l] = INFINITY;
        bf[l] = -1;
    }
    for (int64_t f = threadIdx.x; f < P; f += blockDim.x) {
        const int a = (int)(f / tb.K2), k = (int)(f % tb.K2);
        const double t1 = tb.t1[a];
        const double e = t1 + tb.t2[k];
        const int32_t p1 = u1[a], pe = ue[f];
        const double n1 = (double)nrow[p1], ne = (double)nrow[pe];
        const double s1 = srow[p1], se = srow[pe];
        const double hbm = s1 + t1 * (tot - n1);
        double hold = (se - s1) - t1 * (ne - n1);
        if (!isinf(e)) hold = hold + (e - t1) * (tot - ne);
        const double fixed = pr.a1 * hbm + pr.b2 * (ne - n1) + pr.b3 * (tot - ne);
#pragma unroll
        for (int l = 0; l < kFLoads; ++l) {
            if (l < nl) {
                const double tc = fixed + a2[l] * hold;
                if (cost_out != nullptr) cost_out[(r * tb.L + l0 + l) * P + f] = tc / md;
                argmin_merge(bc[l], bf[l], tc, (int32_t)f);
            }
        }
    }
    const int lane = threadIdx.x % kWave, wv = threadIdx.x / kWave;
#pragma unroll
    for (int l = 0; l < kFLoads; ++l) {
        wave_argmin(bc[l], bf[l]);
        if (lane == 0) {
            rc[wv][l] = bc[l];
            rf[wv][l] = bf[l];
        }
    }
    __syncthreads();
    if ((int)threadIdx.x < nl) {
        const int l = threadIdx.x;
        double c = rc[0][l];
        int32_t f = rf[0][l];
        for (int q = 1; q < nw; ++q) argmin_merge(c, f, rc[q][l], rf[q][l]);
        best[r * tb.L + l0 + l] = f;
        best_cost[r * tb.L + l0 + l] = c / md;
    }
}

int64_t factored_batch(int64_t n, int64_t R)
{
    // at most 1 GiB of prefix rows (16 bytes per position) per batch
    int64_t rb = ((int64_t)1 << 30) / ((n + 1) * 16);
    if (rb < 1) rb = 1;
    return rb < R ? rb : R;
}

hipError_t launch_factored(const SampleSrc &src, int64_t R, const Tables &tb, const PriceDev &pr,
                           FactoredWs &ws, int32_t *best, double *best_cost, double *cost_out,
                           int *status, hipStream_t stream)
{
    const int64_t n = src.n, m = src.m;
    const int64_t P = (int64_t)tb.K1 * tb.K2;
    int cur = 0;
    hipError_t err = launch_sort_keys(src.w, src.T, n, ws.sort, &cur, status, stream);
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(factored_rank_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0,
                       stream, ws.sort.keys[cur], ws.sort.vals[cur], src.T, n, ws.sw, ws.Ts,
                       ws.rank);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    hipLaunchKernelGGL(factored_bounds_kernel, dim3((unsigned)((tb.K1 + P + 255) / 256)), dim3(256),
                       0, stream, ws.sw, n, tb, ws.u1, ws.ue);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    const int ntl = (tb.L + kFLoads - 1) / kFLoads;
    for (int64_t r0 = 0; r0 < R; r0 += ws.Rb) {
        const int64_t rb = (R - r0 < ws.Rb) ? R - r0 : ws.Rb;
        hipLaunchKernelGGL(factored_hist_kernel, dim3((unsigned)rb), dim3(kFThreads), 0, stream,
                           src.idx, n, m, r0, ws.rank, ws.N, status);
        hipLaunchKernelGGL(factored_scan_kernel, dim3((unsigned)rb), dim3(kFThreads), 0, stream,
                           ws.N, ws.S, ws.sw, ws.Ts, n);
        hipLaunchKernelGGL(factored_policy_kernel, dim3((unsigned)(rb * ntl)), dim3(kFPolThreads), 0,
                           stream, ws.N, ws.S, n, m, r0, ntl, tb, pr, ws.u1, ws.ue, best, best_cost,
                           cost_out);
        if ((err = hipGetLastError()) != hipSuccess) return err;
    }
    return hipSuccess;
}

}  // namespace kvr
