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
#include "kvr_device.h"

#include <math.h>

namespace kvr {

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

}  // namespace kvr
