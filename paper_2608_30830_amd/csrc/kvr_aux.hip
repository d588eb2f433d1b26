// Auxiliary kernels of the calibration replay for gfx950: status and table
// staging, the per-timer sums X and G, the reduction of sample splits, and the
// selection kernels (arg-min under the total order "smaller cost, then larger
// flat index").
#include "kvr_device.h"

#include <math.h>

namespace kvr {

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

__global__ void export_status_kernel(const int *status, int32_t *out)
{
    if (threadIdx.x == 0) out[0] = status[0] == 0 ? KVR_OK : KVR_E_DOMAIN;
}

hipError_t launch_export_status(const int *status, int32_t *out, hipStream_t stream)
{
    hipLaunchKernelGGL(export_status_kernel, dim3(1), dim3(64), 0, stream, status, out);
    return hipGetLastError();
}

// Clears the status word and a range of counters, and stores up to three host
// tables in one launch when they fit one payload together.
struct StagePlan {
    double *dst[3];
    int cnt[3];
    unsigned *zero;
    int nzero;
};

__global__ void stage_kernel(int *status, StagePlan sp, UploadPayload p)
{
    if (threadIdx.x == 0) status[0] = 0;
    for (int i = threadIdx.x; i < sp.nzero; i += blockDim.x) sp.zero[i] = 0u;
    int off = 0;
    for (int t = 0; t < 3; ++t) {
        for (int i = threadIdx.x; i < sp.cnt[t]; i += blockDim.x) sp.dst[t][i] = p.v[off + i];
        off += sp.cnt[t];
    }
}

hipError_t launch_stage(int *status, double *const dst[3], const double *const src[3],
                        const int64_t cnt[3], unsigned *zero, int nzero, hipStream_t stream)
{
    const bool one = cnt[0] + cnt[1] + cnt[2] <= kUploadMax;
    StagePlan sp;
    UploadPayload p;
    sp.zero = zero;
    sp.nzero = zero != nullptr ? nzero : 0;
    int off = 0;
    for (int t = 0; t < 3; ++t) {   // the tables ride along when they fit, else follow
        sp.dst[t] = dst[t];
        sp.cnt[t] = one ? (int)cnt[t] : 0;
        for (int64_t i = 0; i < sp.cnt[t]; ++i) p.v[off++] = src[t][i];
    }
    for (int i = off; i < kUploadMax; ++i) p.v[i] = 0.0;
    hipLaunchKernelGGL(stage_kernel, dim3(1), dim3(256), 0, stream, status, sp, p);
    hipError_t err = hipGetLastError();
    for (int t = 0; t < 3 && !one && err == hipSuccess; ++t)
        err = launch_upload(dst[t], src[t], cnt[t], stream);
    return err;
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
// samples of resample r.  One 256-thread block per (resample, group of ng
// tiles of kAT timers, sample part), ng = 1, 2, 4 or 8 (the smallest that
// covers the timers, at most 8): the block gathers each draw of its part
// once, in chunks of 256 staged in LDS, and thread (q, u) = (t % ng, t / ng)
// adds draws u, u + 256/ng, ... of every chunk for the kAT timers of tile q.
// A fixed-order tree over u follows.  With several parts the block writes a
// partial pair to xgp[part][r][a][2] and xg_reduce_kernel adds the parts in
// part order.
constexpr int kAT = 8;                  // timers per tile
constexpr int kAGMax = 8;               // tiles per block at most
constexpr int kXT = 256;                // threads per block = draws per chunk

static int xg_tiles_per_block(int K1)
{
    const int natiles = (K1 + kAT - 1) / kAT;
    int ng = 1;
    while (ng < natiles && ng < kAGMax) ng *= 2;
    return ng;
}

__global__ void __launch_bounds__(kXT) xg_kernel(SampleSrc src, Tables tb, int ng, int parts,
                                                 int64_t part_len, double *X, double *G,
                                                 double *xgp, const SampleRec *__restrict__ rec,
                                                 int *status)
{
    const int natiles = (tb.K1 + kAT - 1) / kAT;
    const int ngroups = (natiles + ng - 1) / ng;
    const int nu = kXT / ng;                         // threads per tile
    const int part = (int)(blockIdx.x % parts);
    const int64_t rest = blockIdx.x / parts;
    const int64_t r = rest / ngroups;
    const int tile0 = (int)(rest % ngroups) * ng;
    const int q = (int)threadIdx.x % ng, u = (int)threadIdx.x / ng;
    const int a0 = (tile0 + q) * kAT;                // first timer of this thread's tile
    double t1v[kAT], xs[kAT], gs[kAT];
#pragma unroll
    for (int k = 0; k < kAT; ++k) {
        t1v[k] = (a0 + k < tb.K1) ? tb.t1[a0 + k] : 0.0;
        xs[k] = 0.0;
        gs[k] = 0.0;
    }
    const int64_t row_off = r * src.m;
    const int64_t j0 = (int64_t)part * part_len;
    const int64_t j1 = (j0 + part_len < src.m) ? j0 + part_len : src.m;
    const int64_t nch = (j1 - j0 + kXT - 1) / kXT;

    __shared__ double2 stage[2][kXT];
    auto fetch = [&](int64_t c) {                  // this thread's draw of chunk c
        const int64_t j = j0 + c * kXT + threadIdx.x;
        Sample z;                                  // padding: adds exact zeros
        z.w = 0.0;
        z.T = 0.0;
        if (j >= j1) return z;
        if (rec == nullptr) return fetch_sample(src, row_off, j, status);
        // the cleaned record of the drawn sample: one 16-byte gather
        // (bad waits and contexts are flagged by the grid kernel's reads)
        int64_t i = j;
        if (src.idx) {
            int32_t ii = src.idx[row_off + j];
            if (ii < 0 || (int64_t)ii >= src.n) {
                flag_domain(status);
                ii = 0;
            }
            i = ii;
        }
        const SampleRec v = rec[i];
        z.w = v.w;
        z.T = (double)v.T;
        return z;
    };
    Sample pre = nch > 0 ? fetch(0) : Sample{0.0, 0.0};
    for (int64_t c = 0; c < nch; ++c) {
        // buffer c & 1 was last read in chunk c - 2; every thread finished
        // those reads before passing the barrier of chunk c - 1
        const int b = (int)(c & 1);
        stage[b][threadIdx.x] = make_double2(pre.w, pre.T);
        __syncthreads();
        if (c + 1 < nch) pre = fetch(c + 1);
        for (int v = 0; v < ng; ++v) {
            const double2 sm = stage[b][u + v * nu];
#pragma unroll
            for (int k = 0; k < kAT; ++k) {
                xs[k] = fma(sm.y, fmin(sm.x, t1v[k]), xs[k]);
                gs[k] += (sm.x > t1v[k]) ? sm.y : 0.0;
            }
        }
    }

    // fixed-order tree over the nu threads of each tile
    __shared__ double red[kXT][2 * kAT];
#pragma unroll
    for (int k = 0; k < kAT; ++k) {
        red[threadIdx.x][k] = xs[k];
        red[threadIdx.x][kAT + k] = gs[k];
    }
    __syncthreads();
    for (int stride = nu / 2; stride > 0; stride /= 2) {
        if (u < stride) {
#pragma unroll
            for (int k = 0; k < 2 * kAT; ++k) red[threadIdx.x][k] += red[threadIdx.x + stride * ng][k];
        }
        __syncthreads();
    }
    if (threadIdx.x < ng * 2 * kAT) {
        const int tq = (int)threadIdx.x / (2 * kAT), v = (int)threadIdx.x % (2 * kAT);
        const double acc = red[tq][v];               // row u = 0 of tile tq
        const int a = (tile0 + tq) * kAT + (v % kAT);
        if (a < tb.K1) {
            const bool isx = v < kAT;
            const int64_t ra = r * tb.K1 + a;
            if (parts == 1) {
                if (isx) X[ra] = acc;
                else G[ra] = acc;
            } else {
                const int64_t R = (int64_t)gridDim.x / parts / ngroups;
                xgp[2 * ((int64_t)part * R * tb.K1 + ra) + (isx ? 0 : 1)] = acc;
            }
        }
    }
}

// One thread per (resample, timer): adds the parts in part order.
__global__ void __launch_bounds__(256) xg_reduce_kernel(int parts, int64_t RK1,
                                                        const double *__restrict__ xgp,
                                                        double *__restrict__ X,
                                                        double *__restrict__ G)
{
    const int64_t ra = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (ra >= RK1) return;
    double x = 0.0, g = 0.0;
    for (int p = 0; p < parts; ++p) {
        x += xgp[2 * ((int64_t)p * RK1 + ra)];
        g += xgp[2 * ((int64_t)p * RK1 + ra) + 1];
    }
    X[ra] = x;
    G[ra] = g;
}

int xg_parts(int64_t R, int K1, int64_t m, int64_t *part_len)
{
    const int ng = xg_tiles_per_block(K1);
    const int64_t ngroups = ((K1 + kAT - 1) / kAT + ng - 1) / ng;
    int64_t parts = 1;
    if (R * ngroups < 1024) {
        parts = (1024 + R * ngroups - 1) / (R * ngroups);
        const int64_t most = (m + 4095) / 4096;  // at least 4,096 samples per part
        if (parts > most) parts = most;
        if (parts < 1) parts = 1;
    }
    *part_len = (m + parts - 1) / parts;
    return (int)((m + *part_len - 1) / *part_len);
}

hipError_t launch_xg(const SampleSrc &src, int64_t R, const Tables &tb, double *X, double *G,
                     double *xgp, const SampleRec *rec, int *status, hipStream_t stream)
{
    const int ng = xg_tiles_per_block(tb.K1);
    const int ngroups = ((tb.K1 + kAT - 1) / kAT + ng - 1) / ng;
    int64_t part_len = 0;
    const int parts = xg_parts(R, tb.K1, src.m, &part_len);
    hipLaunchKernelGGL(xg_kernel, dim3((unsigned)(R * ngroups * parts)), dim3(kXT), 0, stream, src,
                       tb, ng, parts, part_len, X, G, xgp, rec, status);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess || parts == 1) return err;
    const int64_t RK1 = R * tb.K1;
    hipLaunchKernelGGL(xg_reduce_kernel, dim3((unsigned)((RK1 + 255) / 256)), dim3(256), 0, stream,
                       parts, RK1, xgp, X, G);
    return hipGetLastError();
}

// ---------------------------------------------------- split reduce, finalize --
// Partials are laid out [split][resample][tile][value][policy] with the LT
// load accumulators as values (R3 comes from the deadline bins of
// kvr_r3.hip, X and G from xg_kernel).  Stage 1: one thread per
// element of split 0 sums it over the splits, in split order, in place.
__global__ void __launch_bounds__(256) reduce_splits_kernel(int64_t nsplit, int64_t slice,
                                                            double *__restrict__ partials)
{
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (gid >= slice) return;
    double s = partials[gid];
    int64_t q = 1;
    for (; q + 8 <= nsplit; q += 8) {   // eight loads in flight, added in split order
        double v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = partials[(q + u) * slice + gid];
#pragma unroll
        for (int u = 0; u < 8; ++u) s += v[u];
    }
    for (; q < nsplit; ++q) s += partials[q * slice + gid];
    partials[gid] = s;
}

// Stage 2: one thread per (resample, tile, policy) turns the sums into mean
// costs, with the same expression the fused grid kernel uses.
template <int LT>
__global__ void __launch_bounds__(256) finalize_kernel(GridPlan plan, Tables tb, PriceDev pr,
                                                       double md, const double *__restrict__ X,
                                                       const double *__restrict__ G, R3Ws r3s,
                                                       const double *__restrict__ sums,
                                                       double *__restrict__ cost_out)
{
    const int64_t P = (int64_t)tb.K1 * tb.K2;
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (gid >= plan.R * plan.ntiles * P) return;
    const int64_t f = gid % P;
    const int tile = (int)((gid / P) % plan.ntiles);
    const int64_t r = gid / (P * plan.ntiles);
    const int a = (int)(f / tb.K2);
    const int64_t base_row = (r * plan.ntiles + tile) * LT;
    const int32_t xb = r3s.lb[f];
    const double r3 = (xb < r3s.nbins) ? (double)r3s.S[r * r3s.nbins + xb] : 0.0;
    const double base = pr.a1 * X[r * tb.K1 + a] + (pr.b2 * (G[r * tb.K1 + a] - r3) + pr.b3 * r3);
#pragma unroll
    for (int l = 0; l < LT; ++l) {
        const int lg = tile * LT + l;
        if (lg < tb.L) cost_out[(r * tb.L + lg) * P + f] = (base + sums[(base_row + l) * P + f]) / md;
    }
}

hipError_t launch_reduce_partials(const GridPlan &plan, const Tables &tb, const PriceDev &pr,
                                  int64_t m, const double *X, const double *G, const R3Ws &r3,
                                  double *partials, double *cost_out, hipStream_t stream)
{
    const int64_t P = (int64_t)tb.K1 * tb.K2;
    const int64_t slice = plan.R * plan.ntiles * (int64_t)plan.LT * P;
    hipLaunchKernelGGL(reduce_splits_kernel, dim3((unsigned)((slice + 255) / 256)), dim3(256), 0,
                       stream, (int64_t)plan.nsplit, slice, partials);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    const int64_t threads = plan.R * plan.ntiles * P;
    const unsigned blocks = (unsigned)((threads + 255) / 256);
    const double md = (double)m;
    switch (plan.LT) {
    case 4: hipLaunchKernelGGL(finalize_kernel<4>, dim3(blocks), dim3(256), 0, stream, plan, tb, pr, md, X, G, r3, partials, cost_out); break;
    case 8: hipLaunchKernelGGL(finalize_kernel<8>, dim3(blocks), dim3(256), 0, stream, plan, tb, pr, md, X, G, r3, partials, cost_out); break;
    case 16: hipLaunchKernelGGL(finalize_kernel<16>, dim3(blocks), dim3(256), 0, stream, plan, tb, pr, md, X, G, r3, partials, cost_out); break;
    case 32: hipLaunchKernelGGL(finalize_kernel<32>, dim3(blocks), dim3(256), 0, stream, plan, tb, pr, md, X, G, r3, partials, cost_out); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// ------------------------------------------------------- selection kernels --
// Per (resample, load): best of the per-wave candidates.  One wave per row.
// The groups holding resample r's policies are r*nblk .. (r+1)*nblk-1 (one
// resample per group), or, for groups over the flattened (resample, policy)
// space, those covering flat indices r*P .. r*P + P - 1, where r sits in slot
// 0 if it is the group's first resample and in slot 1 otherwise.
__global__ void __launch_bounds__(256) reduce_cands_kernel(const ArgminCand *__restrict__ cand,
                                                           int64_t rows, int per_lane, int nblk,
                                                           int64_t P, int L,
                                                           int32_t *__restrict__ best,
                                                           double *__restrict__ best_cost)
{
    const int64_t row = (int64_t)blockIdx.x * 4 + threadIdx.x / kWave;
    const int lane = threadIdx.x % kWave;
    if (row >= rows) return;
    const int64_t r = row / L;
    const int l = (int)(row % L);
    int64_t g0, g1;
    if (per_lane) {
        g0 = r * nblk;
        g1 = g0 + nblk - 1;
    } else {
        g0 = (r * P) / kWave;
        g1 = (r * P + P - 1) / kWave;
    }
    double bc = INFINITY;
    int32_t bf = -1;
    for (int64_t g = g0 + lane; g <= g1; g += kWave) {
        const int slot = (per_lane || (g * kWave) / P == r) ? 0 : 1;
        const ArgminCand c = cand[(g * 2 + slot) * L + l];
        argmin_merge(bc, bf, c.cost, c.f);
    }
    wave_argmin(bc, bf);
    if (lane == 0) {
        best[row] = bf;
        best_cost[row] = bc;
    }
}

hipError_t launch_reduce_cands(const ArgminCand *cand, const GridPlan &plan, int64_t P, int L,
                               int32_t *best, double *best_cost, hipStream_t stream)
{
    const int64_t rows = plan.R * L;
    hipLaunchKernelGGL(reduce_cands_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, stream,
                       cand, rows, plan.mode == kModePerLane ? 1 : 0, plan.nblk, P, L, best,
                       best_cost);
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
