// Brute-force cost grid for gfx950 (CDNA4).
//
// Per request (Eq. 1 summed over the states visited, Eq. 3 congestion price,
// Appendix D one-shot timer) the cost of policy (t1, t2, lambda) is
//   T * ( a1*min(w,t1) + [w > t1] * ( a2(lambda)*(min(w,e) - t1) + (w <= e ? b2 : b3) ) ),
// e = t1 + t2.  Summed over a sample this splits into
//   a1*X(t1) + b2*(G(t1) - R3(e)) + b3*R3(e) + sum_i a2(lambda) * h_i(t1,e)
// with X(t1) = sum T*min(w,t1), G(t1) = sum T*[w > t1], R3(e) = sum T*[w > e]
// and h_i = T*(min(max(w,t1),e) - t1) >= 0 (zero when w <= t1).  The load
// axis is evaluated in full: every (sample, policy, load) gets one fp64 FMA
// acc[lambda] += a2(lambda) * h.  Terms that do not depend on the load are
// computed once per (sample, policy); terms that depend only on t1 (X, G) once
// per (sample, t1) by xg_kernel.
//
// Layout: one wave owns 64 consecutive policies (lane = flat policy index
// f = a*K2 + k) of one resample and one tile of up to 32 loads.  The samples
// are streamed through LDS in chunks of kChunk and read back as wave-uniform
// broadcasts, so each lane accumulates its own policy over the whole sample
// in a fixed order; no cross-lane reduction of costs is needed, and every
// policy of a call is summed in exactly the same order, which keeps policies
// with identical per-sample terms bit-identical (structural ties stay exact).
// No MFMA: nothing here is a dense contraction.
#include "kvr_internal.h"

#include <float.h>
#include <math.h>

namespace kvr {

// ------------------------------------------------------------------ common --
__device__ __forceinline__ void flag_domain(int *status)
{
    __hip_atomic_store(status, kStatusDomain, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

struct Sample {
    double w, T;
};

// Read sample j of a resample (row offset row_off into idx), replacing bad
// values by safe ones and flagging the status word.
__device__ __forceinline__ Sample fetch_sample(const SampleSrc &s, int64_t row_off, int64_t j,
                                               int *status)
{
    int64_t i = j;
    if (s.idx) {
        int32_t ii = s.idx[row_off + j];
        if (ii < 0 || (int64_t)ii >= s.n) {
            flag_domain(status);
            ii = 0;
        }
        i = ii;
    }
    double w = s.w[i];
    int32_t t = s.T[i];
    // finite and >= 0 (or -0.0), tested on the bits so that no floating-point
    // mode or NaN assumption can remove the check
    const uint64_t bits = (uint64_t)__double_as_longlong(w);
    if (!(bits < 0x7ff0000000000000ull || bits == 0x8000000000000000ull)) {
        flag_domain(status);
        w = 0.0;
    }
    if (t < 1) {
        flag_domain(status);
        t = 1;
    }
    Sample out;
    out.w = w + 0.0;  // -0.0 -> +0.0
    out.T = (double)t;
    return out;
}

template <typename V>
__device__ __forceinline__ V wave_sum(V v)
{
    for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
    return v;
}

// Total order used by every selection: smaller cost first, then larger f.
__device__ __forceinline__ void argmin_merge(double &bc, int32_t &bf, double oc, int32_t of)
{
    bool take = (oc < bc) || (oc == bc && of > bf);
    bc = take ? oc : bc;
    bf = take ? of : bf;
}

__device__ __forceinline__ void wave_argmin(double &bc, int32_t &bf)
{
    for (int off = kWave / 2; off > 0; off >>= 1) {
        double oc = __shfl_xor(bc, off, kWave);
        int32_t of = __shfl_xor(bf, off, kWave);
        argmin_merge(bc, bf, oc, of);
    }
}

// Hardware hands work-groups to the 8 XCDs round-robin; remap so that each
// XCD walks a contiguous range of logical blocks (same resample rows, same
// L2).
__device__ __forceinline__ int64_t xcd_logical_block(int64_t hw, int64_t nblocks)
{
    const int64_t nx = 8;
    int64_t x = hw % nx, q = nblocks / nx, rem = nblocks % nx;
    return x * q + (x < rem ? x : rem) + hw / nx;
}

// ------------------------------------------------------------ small kernels --
__global__ void clear_status_kernel(int *status)
{
    if (threadIdx.x == 0) status[0] = 0;
}

constexpr int kUploadMax = 384;
struct UploadPayload {
    double v[kUploadMax];
};

// Host tables travel as kernel arguments, so the caller's host buffers are
// captured at launch and no pinned staging or host synchronisation is needed.
__global__ void upload_kernel(double *dst, int n, UploadPayload p)
{
    for (int i = threadIdx.x; i < n; i += blockDim.x) dst[i] = p.v[i];
}

hipError_t launch_clear_status(int *status, hipStream_t stream)
{
    hipLaunchKernelGGL(clear_status_kernel, dim3(1), dim3(64), 0, stream, status);
    return hipGetLastError();
}

hipError_t launch_upload(double *dst, const double *host_src, int64_t count, hipStream_t stream)
{
    for (int64_t off = 0; off < count; off += kUploadMax) {
        int c = (int)((count - off) < kUploadMax ? (count - off) : kUploadMax);
        UploadPayload p;
        for (int i = 0; i < c; ++i) p.v[i] = host_src[off + i];
        for (int i = c; i < kUploadMax; ++i) p.v[i] = 0.0;
        hipLaunchKernelGGL(upload_kernel, dim3(1), dim3(256), 0, stream, dst + off, c, p);
        hipError_t err = hipGetLastError();
        if (err != hipSuccess) return err;
    }
    return hipSuccess;
}

// ------------------------------------------------------------------- X, G --
// X[r][a] = sum_j T*min(w, t1_a), G[r][a] = sum_j T*[w > t1_a] over the
// samples of resample r.  One 256-thread block per (resample, tile of kAT
// timers); threads stride over samples, then a fixed-order reduction.
constexpr int kAT = 8;

__global__ void __launch_bounds__(256) xg_kernel(SampleSrc src, Tables tb, double *X, double *G,
                                                 int *status)
{
    const int natiles = (tb.K1 + kAT - 1) / kAT;
    const int64_t r = blockIdx.x / natiles;
    const int a0 = (int)(blockIdx.x % natiles) * kAT;
    double t1v[kAT], xs[kAT], gs[kAT];
#pragma unroll
    for (int q = 0; q < kAT; ++q) {
        t1v[q] = (a0 + q < tb.K1) ? tb.t1[a0 + q] : 0.0;
        xs[q] = 0.0;
        gs[q] = 0.0;
    }
    const int64_t row_off = r * src.m;
    for (int64_t j = threadIdx.x; j < src.m; j += blockDim.x) {
        Sample s = fetch_sample(src, row_off, j, status);
#pragma unroll
        for (int q = 0; q < kAT; ++q) {
            xs[q] = fma(s.T, fmin(s.w, t1v[q]), xs[q]);
            gs[q] += (s.w > t1v[q]) ? s.T : 0.0;
        }
    }
    __shared__ double red[4][2 * kAT];
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
#pragma unroll
    for (int q = 0; q < kAT; ++q) {
        double x = wave_sum(xs[q]);
        double g = wave_sum(gs[q]);
        if (lane == 0) {
            red[wave][q] = x;
            red[wave][kAT + q] = g;
        }
    }
    __syncthreads();
    if (threadIdx.x < kAT && a0 + (int)threadIdx.x < tb.K1) {
        const int q = threadIdx.x;
        double x = ((red[0][q] + red[1][q]) + red[2][q]) + red[3][q];
        double g = ((red[0][kAT + q] + red[1][kAT + q]) + red[2][kAT + q]) + red[3][kAT + q];
        X[r * tb.K1 + a0 + q] = x;
        G[r * tb.K1 + a0 + q] = g;
    }
}

hipError_t launch_xg(const SampleSrc &src, int64_t R, const Tables &tb, double *X, double *G,
                     int *status, hipStream_t stream)
{
    const int natiles = (tb.K1 + kAT - 1) / kAT;
    hipLaunchKernelGGL(xg_kernel, dim3((unsigned)(R * natiles)), dim3(256), 0, stream, src, tb, X,
                       G, status);
    return hipGetLastError();
}

// ------------------------------------------------------------- grid kernel --
// ROWPAIR: K2 >= 64, so the 64 consecutive policies of a wave lie in at most
// two timer rows a0, a0+1.  The t1-dependent part of h, d = max(w,t1) - t1,
// is computed once per staged sample for both rows and each lane reads its
// row's copy from LDS.  Otherwise (K2 < 64) every lane computes d itself.
// Rounding note: min(fl(max(w,t1) - t1), fl(e - t1)) equals
// fl(min(max(w,t1), e) - t1) because rounding is monotone.
template <int LT, bool ROWPAIR>
__global__ void __launch_bounds__(kWave) grid_kernel(SampleSrc src, Tables tb, PriceDev pr,
                                                     GridPlan plan, const double *__restrict__ X,
                                                     const double *__restrict__ G,
                                                     double *__restrict__ cost_out,
                                                     ArgminCand *__restrict__ cand,
                                                     double *__restrict__ partials, int *status,
                                                     int64_t nlogical)
{
    __shared__ double2 wt[2][kChunk];     // (w, T) per staged sample
    __shared__ double2 dd[2][kChunk];     // (d for row a0, d for row a0+1)

    const int64_t logical = xcd_logical_block(blockIdx.x, nlogical);
    const int blk = (int)(logical % plan.nblk);
    int64_t rest = logical / plan.nblk;
    const int tile = (int)(rest % plan.ntiles);
    rest /= plan.ntiles;
    const int split = (int)(rest % plan.nsplit);
    const int64_t r = rest / plan.nsplit;

    const int lane = threadIdx.x;
    const int64_t P = (int64_t)tb.K1 * tb.K2;
    const int64_t f0 = (int64_t)blk * kWave;
    const int64_t f = f0 + lane;
    const bool valid = f < P;
    const int a = valid ? (int)(f / tb.K2) : (int)(f0 / tb.K2);
    const int k = valid ? (int)(f % tb.K2) : 0;
    const double t1 = tb.t1[a];
    const double e = valid ? t1 + tb.t2[k] : t1;   // deadline from suspension
    const double ep = e - t1;                       // host time before discard
    // rows staged for this wave
    const int a0 = (int)(f0 / tb.K2);
    const int a1r = (a0 + 1 < tb.K1) ? a0 + 1 : a0;
    const double t1A = tb.t1[a0], t1B = tb.t1[a1r];
    const int sel = (a != a0) ? 1 : 0;

    double a2[LT], acc[LT];
#pragma unroll
    for (int l = 0; l < LT; ++l) {
        a2[l] = tb.a2[tile * LT + l];
        acc[l] = 0.0;
    }
    double r3 = 0.0;

    const int64_t j0 = (int64_t)split * plan.split_len;
    int64_t j1 = j0 + plan.split_len;
    if (j1 > src.m) j1 = src.m;
    const int64_t nch = (j1 - j0 + kChunk - 1) / kChunk;
    const int64_t row_off = r * src.m;

    constexpr int kPer = kChunk / kWave;
    Sample pre[kPer];
    auto load_chunk = [&](int64_t c) {
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            int64_t j = j0 + c * kChunk + q * kWave + lane;
            if (j < j1) {
                pre[q] = fetch_sample(src, row_off, j, status);
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
            wt[b][s] = make_double2(pre[q].w, pre[q].T);
            if (ROWPAIR)
                dd[b][s] = make_double2(fmax(pre[q].w, t1A) - t1A, fmax(pre[q].w, t1B) - t1B);
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
        const double *drow = reinterpret_cast<const double *>(&dd[cur][0]) + sel;
#pragma unroll 4
        for (int j = 0; j < kChunk; ++j) {
            const double2 s = wt[cur][j];            // wave-uniform broadcast
            double d;
            if (ROWPAIR) d = drow[2 * j];             // this lane's timer row
            else d = fmax(s.x, t1) - t1;              // 0 when w <= t1
            const double h = s.y * fmin(d, ep);       // T * host seconds held
            const double gone = (s.x > e) ? 1.0 : 0.0;   // discarded before resume
            r3 = fma(gone, s.y, r3);
#pragma unroll
            for (int l = 0; l < LT; ++l) acc[l] = fma(a2[l], h, acc[l]);
        }
        if (c + 1 < nch) store_chunk(cur ^ 1);
        __syncthreads();
    }

    if (plan.nsplit == 1) {
        const double md = (double)src.m;
        const double x = valid ? X[r * tb.K1 + a] : 0.0;
        const double g = valid ? G[r * tb.K1 + a] : 0.0;
        const double base = pr.a1 * x + (pr.b2 * (g - r3) + pr.b3 * r3);
#pragma unroll
        for (int l = 0; l < LT; ++l) {
            const int lg = tile * LT + l;
            if (lg >= tb.L) break;
            const double c = (base + acc[l]) / md;
            if (cost_out != nullptr && valid) cost_out[(r * tb.L + lg) * P + f] = c;
            if (cand != nullptr) {
                double bc = valid ? c : INFINITY;
                int32_t bf = valid ? (int32_t)f : -1;
                wave_argmin(bc, bf);
                if (lane == 0) {
                    ArgminCand out;
                    out.cost = bc;
                    out.f = bf;
                    out.pad = 0;
                    cand[(r * plan.nblk + blk) * tb.L + lg] = out;
                }
            }
        }
    } else if (valid) {
        const int64_t base_row = (((int64_t)split * plan.R + r) * plan.ntiles + tile) * (LT + 1);
#pragma unroll
        for (int l = 0; l < LT; ++l) partials[(base_row + l) * P + f] = acc[l];
        partials[(base_row + LT) * P + f] = r3;
    }
}

template <int LT>
static hipError_t launch_grid_t(const SampleSrc &src, const Tables &tb, const PriceDev &pr,
                                const GridPlan &plan, const double *X, const double *G,
                                double *cost_out, ArgminCand *cand, double *partials,
                                int *status, hipStream_t stream)
{
    const int64_t nlogical = plan.R * plan.nsplit * plan.ntiles * plan.nblk;
    if (tb.K2 >= kWave)
        hipLaunchKernelGGL((grid_kernel<LT, true>), dim3((unsigned)nlogical), dim3(kWave), 0,
                           stream, src, tb, pr, plan, X, G, cost_out, cand, partials, status,
                           nlogical);
    else
        hipLaunchKernelGGL((grid_kernel<LT, false>), dim3((unsigned)nlogical), dim3(kWave), 0,
                           stream, src, tb, pr, plan, X, G, cost_out, cand, partials, status,
                           nlogical);
    return hipGetLastError();
}

hipError_t launch_grid(const SampleSrc &src, const Tables &tb, const PriceDev &pr,
                       const GridPlan &plan, const double *X, const double *G, double *cost_out,
                       ArgminCand *cand, double *partials, int *status, hipStream_t stream)
{
    switch (plan.LT) {
    case 4: return launch_grid_t<4>(src, tb, pr, plan, X, G, cost_out, cand, partials, status, stream);
    case 8: return launch_grid_t<8>(src, tb, pr, plan, X, G, cost_out, cand, partials, status, stream);
    case 16: return launch_grid_t<16>(src, tb, pr, plan, X, G, cost_out, cand, partials, status, stream);
    case 32: return launch_grid_t<32>(src, tb, pr, plan, X, G, cost_out, cand, partials, status, stream);
    default: return hipErrorInvalidValue;
    }
}

// ---------------------------------------------------- split reduce, finalize --
// One thread per (resample, load tile, policy): sums the split partials in
// split order and writes the final mean costs.
template <int LT>
__global__ void __launch_bounds__(256) reduce_partials_kernel(GridPlan plan, Tables tb,
                                                              PriceDev pr, double md,
                                                              const double *__restrict__ X,
                                                              const double *__restrict__ G,
                                                              const double *__restrict__ partials,
                                                              double *__restrict__ cost_out)
{
    const int64_t P = (int64_t)tb.K1 * tb.K2;
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (gid >= plan.R * plan.ntiles * P) return;
    const int64_t f = gid % P;
    const int tile = (int)((gid / P) % plan.ntiles);
    const int64_t r = gid / (P * plan.ntiles);
    const int a = (int)(f / tb.K2);
    double acc[LT + 1];
#pragma unroll
    for (int j = 0; j <= LT; ++j) acc[j] = 0.0;
    for (int s = 0; s < plan.nsplit; ++s) {
        const int64_t base_row = (((int64_t)s * plan.R + r) * plan.ntiles + tile) * (LT + 1);
#pragma unroll
        for (int j = 0; j <= LT; ++j) acc[j] += partials[(base_row + j) * P + f];
    }
    const double r3 = acc[LT];
    const double base = pr.a1 * X[r * tb.K1 + a] + (pr.b2 * (G[r * tb.K1 + a] - r3) + pr.b3 * r3);
#pragma unroll
    for (int l = 0; l < LT; ++l) {
        const int lg = tile * LT + l;
        if (lg < tb.L) cost_out[(r * tb.L + lg) * P + f] = (base + acc[l]) / md;
    }
}

hipError_t launch_reduce_partials(const GridPlan &plan, const Tables &tb, const PriceDev &pr,
                                  int64_t m, const double *X, const double *G,
                                  const double *partials, double *cost_out, hipStream_t stream)
{
    const int64_t P = (int64_t)tb.K1 * tb.K2;
    const int64_t threads = plan.R * plan.ntiles * P;
    const unsigned blocks = (unsigned)((threads + 255) / 256);
    const double md = (double)m;
    switch (plan.LT) {
    case 4: hipLaunchKernelGGL(reduce_partials_kernel<4>, dim3(blocks), dim3(256), 0, stream, plan, tb, pr, md, X, G, partials, cost_out); break;
    case 8: hipLaunchKernelGGL(reduce_partials_kernel<8>, dim3(blocks), dim3(256), 0, stream, plan, tb, pr, md, X, G, partials, cost_out); break;
    case 16: hipLaunchKernelGGL(reduce_partials_kernel<16>, dim3(blocks), dim3(256), 0, stream, plan, tb, pr, md, X, G, partials, cost_out); break;
    case 32: hipLaunchKernelGGL(reduce_partials_kernel<32>, dim3(blocks), dim3(256), 0, stream, plan, tb, pr, md, X, G, partials, cost_out); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// ------------------------------------------------------- selection kernels --
// Per (resample, load): best of the per-wave candidates.  One wave per row.
__global__ void __launch_bounds__(256) reduce_cands_kernel(const ArgminCand *__restrict__ cand,
                                                           int64_t rows, int nblk, int L,
                                                           int32_t *__restrict__ best,
                                                           double *__restrict__ best_cost)
{
    const int64_t row = (int64_t)blockIdx.x * 4 + threadIdx.x / kWave;
    const int lane = threadIdx.x % kWave;
    if (row >= rows) return;
    const int64_t r = row / L;
    const int l = (int)(row % L);
    double bc = INFINITY;
    int32_t bf = -1;
    for (int b = lane; b < nblk; b += kWave) {
        const ArgminCand c = cand[(r * nblk + b) * L + l];
        argmin_merge(bc, bf, c.cost, c.f);
    }
    wave_argmin(bc, bf);
    if (lane == 0) {
        best[row] = bf;
        best_cost[row] = bc;
    }
}

hipError_t launch_reduce_cands(const ArgminCand *cand, int64_t R, int nblk, int L, int32_t *best,
                               double *best_cost, hipStream_t stream)
{
    const int64_t rows = R * L;
    hipLaunchKernelGGL(reduce_cands_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, stream,
                       cand, rows, nblk, L, best, best_cost);
    return hipGetLastError();
}

// Per (batch, load) row of P costs: one 256-thread block per row.
__global__ void __launch_bounds__(256) select_kernel(const double *__restrict__ cost, int64_t P,
                                                     int K2, int last_inf,
                                                     int32_t *__restrict__ best,
                                                     double *__restrict__ best_cost,
                                                     int32_t *__restrict__ branch)
{
    const int64_t row = blockIdx.x;
    const double *c = cost + row * P;
    double bc = INFINITY;
    int32_t bf = -1;
    for (int64_t f = threadIdx.x; f < P; f += blockDim.x) argmin_merge(bc, bf, c[f], (int32_t)f);
    wave_argmin(bc, bf);
    __shared__ double sc[4];
    __shared__ int32_t sf[4];
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    if (lane == 0) {
        sc[wave] = bc;
        sf[wave] = bf;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int q = 1; q < 4; ++q) argmin_merge(bc, bf, sc[q], sf[q]);
        best[row] = bf;
        best_cost[row] = bc;
        if (branch != nullptr) branch[row] = (last_inf && (bf % K2) == K2 - 1) ? 0 : 1;
    }
}

hipError_t launch_select(const double *cost, int64_t batch, int L, int64_t P, int K2, int last_inf,
                         int32_t *best, double *best_cost, int32_t *branch, hipStream_t stream)
{
    const int64_t rows = batch * L;
    hipLaunchKernelGGL(select_kernel, dim3((unsigned)rows), dim3(256), 0, stream, cost, P, K2,
                       last_inf, best, best_cost, branch);
    return hipGetLastError();
}

}  // namespace kvr
