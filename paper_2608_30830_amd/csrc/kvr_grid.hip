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
// acc[lambda] += a2(lambda) * h, after h is formed once per (sample, policy).
// The load-independent integer sums come from other kernels: X and G per
// (sample, t1) from xg_kernel, R3 per (resample, deadline) from the deadline
// bins of kvr_r3.hip; the epilogue combines them with the accumulators.
//
// Layout: one wave owns 64 consecutive policies (lane = one policy of one
// resample) and one tile of up to 32 loads.  The samples are streamed through
// LDS in chunks and read back as wave-uniform broadcasts, so each lane
// accumulates its own policy over the whole sample in a fixed order; no
// cross-lane reduction of costs is needed, and every policy of a call is
// summed in exactly the same order, which keeps policies with identical
// per-sample terms bit-identical (structural ties stay exact).
// No MFMA: nothing here is a dense contraction.
#include "kvr_device.h"

#include <math.h>

namespace kvr {

// ------------------------------------------------------------- grid kernel --
// Modes (chosen on the host, see GridPlan::mode):
//  kModePerLane  K2 < 64.  Groups of 64 policies of one resample; every lane
//                computes d = max(w,t1) - t1 itself.
//  kModeRows1    K2 >= 64, groups over the flattened (resample, policy) space
//                that never straddle a resample.  A group's 64 policies lie
//                in at most two (resample, t1-row) combinations; d is
//                computed once per staged sample for both and each lane reads
//                its combination's copy from LDS.
//  kModeRows2    As kModeRows1, but a group may straddle two resamples (the
//                policy count is not a multiple of 64): two sample streams are
//                staged, one per resample, with half-size chunks.
// Rounding note: min(fl(max(w,t1) - t1), fl(e - t1)) equals
// fl(min(max(w,t1), e) - t1) because rounding is monotone.
// Four resident waves per SIMD: the register budget is capped at 128 VGPRs
// (the accumulators and loads of LT = 32 fit without spilling).  One wave per
// block; small samples, where a wave per split leaves most SIMDs idle, take
// the blocks of several waves of kvr_small.hip instead.
template <int LT, int MODE>
__global__ void __launch_bounds__(kWave) __attribute__((amdgpu_waves_per_eu(4))) grid_kernel(SampleSrc src, Tables tb, PriceDev pr,
                                                     GridPlan plan, const double *__restrict__ X,
                                                     const double *__restrict__ G, R3Ws r3s,
                                                     double *__restrict__ cost_out,
                                                     ArgminCand *__restrict__ cand,
                                                     double *__restrict__ partials, int *status,
                                                     int64_t nlogical)
{
    constexpr bool kStaged = MODE != kModePerLane;
    constexpr bool kTwo = MODE == kModeRows2;
    constexpr int kCh = kTwo ? kChunk / 2 : kChunk;   // samples per staged chunk
    constexpr int kPer = kCh / kWave;                  // samples each lane stages per stream
    // per-lane d: (w, T) of each sample; staged d: (T, d) of each sample for
    // combination A and for B, so a lane reads one 16-byte record per sample
    __shared__ double2 wt[2][kStaged ? 1 : kCh];
    __shared__ double2 td[2][kStaged ? kCh : 1][2];

    const int64_t logical = xcd_logical_block(blockIdx.x, nlogical);
    const int tile = (int)(logical % plan.ntiles);
    int64_t rest = logical / plan.ntiles;
    const int split = (int)(rest % plan.nsplit);
    const int64_t grp = rest / plan.nsplit;

    const int lane = (int)threadIdx.x % kWave;
    const int64_t P = (int64_t)tb.K1 * tb.K2;
    const int64_t RP = plan.R * P;
    int64_t r, f;
    bool valid;
    int64_t FA = 0, FB = 0;
    if (MODE == kModePerLane) {
        r = grp / plan.nblk;
        const int64_t f0 = (grp % plan.nblk) * kWave;
        f = f0 + lane;
        valid = f < P;
        if (!valid) f = f0;
    } else {
        FA = grp * kWave;
        FB = (FA + kWave - 1 < RP) ? FA + kWave - 1 : RP - 1;
        int64_t F = FA + lane;
        valid = F < RP;
        if (!valid) F = FB;
        r = F / P;
        f = F % P;
    }
    const int a = (int)(f / tb.K2);
    const int k = (int)(f % tb.K2);
    const double t1 = tb.t1[a];
    const double e = t1 + tb.t2[k];   // deadline from suspension
    const double ep = e - t1;         // host time before discard
    // the (resample, t1-row) combinations of this group
    const int64_t rA = FA / P, rB = FB / P;
    const int aA = (int)((FA % P) / tb.K2), aB = (int)((FB % P) / tb.K2);
    const double t1A = tb.t1[aA], t1B = tb.t1[aB];
    // which staged combination; when the group straddles two resamples the
    // combinations are (rA, last t1 row) and (rB, first row), one per stream
    const int sel = (r == rA && a == aA) ? 0 : 1;
    const bool twoStreams = kTwo && rB != rA;

    double a2[LT], acc[LT];
#pragma unroll
    for (int l = 0; l < LT; ++l) {
        a2[l] = tb.a2[tile * LT + l];
        acc[l] = 0.0;
    }

    const int64_t j0 = (int64_t)split * plan.split_len;
    int64_t j1 = j0 + plan.split_len;
    if (j1 > src.m) j1 = src.m;
    const int64_t nch = (j1 - j0 + kCh - 1) / kCh;
    const int64_t offA = (kStaged ? rA : r) * src.m;   // index-row offsets of the streams
    const int64_t offB = rB * src.m;

    Sample preA[kPer], preB[kPer];
    auto load_chunk = [&](int64_t c) {
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            const int64_t j = j0 + c * kCh + q * kWave + lane;
            if (j < j1) {
                preA[q] = fetch_sample(src, offA, j, status);
                if (twoStreams) preB[q] = fetch_sample(src, offB, j, status);
                else preB[q] = preA[q];
            } else {  // padding: contributes exact zeros
                preA[q].w = 0.0;
                preA[q].T = 0.0;
                preB[q] = preA[q];
            }
        }
    };
    auto store_chunk = [&](int b) {
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            const int s = q * kWave + lane;
            if (kStaged) {
                td[b][s][0] = make_double2(preA[q].T, fmax(preA[q].w, t1A) - t1A);
                td[b][s][1] = make_double2(preB[q].T, fmax(preB[q].w, t1B) - t1B);
            } else {
                wt[b][s] = make_double2(preA[q].w, preA[q].T);
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
        for (int j = 0; j < kCh; ++j) {
            double T, d;
            if (kStaged) {                            // this lane's combination
                const double2 s = td[cur][j][sel];
                T = s.x;
                d = s.y;
            } else {
                const double2 s = wt[cur][j];
                T = s.y;
                d = fmax(s.x, t1) - t1;               // 0 when w <= t1
            }
            const double h = T * fmin(d, ep);         // T * host seconds held
#pragma unroll
            for (int l = 0; l < LT; ++l) acc[l] = fma(a2[l], h, acc[l]);
        }
        if (c + 1 < nch) store_chunk(cur ^ 1);
        __syncthreads();
    }

    if (partials == nullptr) {   // one split: the costs are finished here
        const double md = (double)src.m;
        const double x = valid ? X[r * tb.K1 + a] : 0.0;
        const double g = valid ? G[r * tb.K1 + a] : 0.0;
        const int32_t xb = r3s.lb[f];                 // recompute share of this deadline
        const double r3 = (valid && xb < r3s.nbins) ? (double)r3s.S[r * r3s.nbins + xb] : 0.0;
        const double base = pr.a1 * x + (pr.b2 * (g - r3) + pr.b3 * r3);
#pragma unroll
        for (int l = 0; l < LT; ++l) {
            const int lg = tile * LT + l;
            if (lg >= tb.L) break;
            const double c = (base + acc[l]) / md;
            if (cost_out != nullptr && valid) cost_out[(r * tb.L + lg) * P + f] = c;
            if (cand != nullptr) {
                // one candidate per (group, resample slot, load): slot 0 holds
                // the group's first resample, slot 1 the second one if any
                for (int slot = 0; slot < (twoStreams ? 2 : 1); ++slot) {
                    const bool mine = valid && (slot == 0 ? r == rA || !kStaged : r == rB);
                    double bc = mine ? c : INFINITY;
                    int32_t bf = mine ? (int32_t)f : -1;
                    wave_argmin(bc, bf);
                    if (lane == 0) {
                        ArgminCand out;
                        out.cost = bc;
                        out.f = bf;
                        out.pad = 0;
                        cand[(grp * 2 + slot) * tb.L + lg] = out;
                    }
                }
            }
        }
    } else if (valid) {   // split partials, finished by the reduction kernels
        const int64_t base_row = (((int64_t)split * plan.R + r) * plan.ntiles + tile) * LT;
#pragma unroll
        for (int l = 0; l < LT; ++l) partials[(base_row + l) * P + f] = acc[l];
    }
}

template <int LT, int MODE>
static hipError_t launch_grid_m(const SampleSrc &src, const Tables &tb, const PriceDev &pr,
                                const GridPlan &plan, const double *X, const double *G,
                                const R3Ws &r3, double *cost_out, ArgminCand *cand,
                                double *partials, int *status, hipStream_t stream)
{
    const int64_t nlogical = plan.ngroups * plan.nsplit * plan.ntiles;
    hipLaunchKernelGGL((grid_kernel<LT, MODE>), dim3((unsigned)nlogical), dim3(kWave), 0, stream,
                       src, tb, pr, plan, X, G, r3, cost_out, cand, partials, status, nlogical);
    return hipGetLastError();
}

template <int LT>
static hipError_t launch_grid_t(const SampleSrc &src, const Tables &tb, const PriceDev &pr,
                                const GridPlan &plan, const double *X, const double *G,
                                const R3Ws &r3, double *cost_out, ArgminCand *cand,
                                double *partials, int *status, hipStream_t stream)
{
    if (plan.wpb != 1) return hipErrorInvalidValue;
    switch (plan.mode) {
    case kModePerLane:
        return launch_grid_m<LT, kModePerLane>(src, tb, pr, plan, X, G, r3, cost_out, cand, partials, status, stream);
    case kModeRows1:
        return launch_grid_m<LT, kModeRows1>(src, tb, pr, plan, X, G, r3, cost_out, cand, partials, status, stream);
    case kModeRows2:
        return launch_grid_m<LT, kModeRows2>(src, tb, pr, plan, X, G, r3, cost_out, cand, partials, status, stream);
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_grid(const SampleSrc &src, const Tables &tb, const PriceDev &pr,
                       const GridPlan &plan, const double *X, const double *G, const R3Ws &r3,
                       double *cost_out, ArgminCand *cand, double *partials, int *status,
                       hipStream_t stream)
{
    switch (plan.LT) {
    case 4: return launch_grid_t<4>(src, tb, pr, plan, X, G, r3, cost_out, cand, partials, status, stream);
    case 8: return launch_grid_t<8>(src, tb, pr, plan, X, G, r3, cost_out, cand, partials, status, stream);
    case 16: return launch_grid_t<16>(src, tb, pr, plan, X, G, r3, cost_out, cand, partials, status, stream);
    case 32: return launch_grid_t<32>(src, tb, pr, plan, X, G, r3, cost_out, cand, partials, status, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace kvr
