// Tail of the regime-aware controller (Section 3.4) and the crossover
// statistic of Section 4.3 / Figure 4(d).
//
// The two host branches are replayed by the admission-replay kernels (one
// lane per (sequence, branch)); what remains is integer bookkeeping: the
// share of waits at or below t* = beta_3 / alpha_1, the token total, and the
// per-branch sums of restored tokens and admissions.  All of it is exact
// integer arithmetic, so atomics and reduction order cannot change a result;
// the two totals b2*R + b3*(Ttot - R) are formed once, without contraction.
#include "kvr_device.h"

namespace kvr {

constexpr int kCountThreads = 256;
constexpr int kCountMaxBlocks = 2048;
constexpr int kCountUnroll = 4;

struct CountWs {
    unsigned long long n_short;
    unsigned long long tokens;
};

__global__ void zero_counts_kernel(CountWs *c)
{
    if (threadIdx.x == 0) {
        c->n_short = 0;
        c->tokens = 0;
    }
}

// counts.n_short += #(w <= t_star); counts.tokens += sum of context tokens
// (one per request without contexts).  Waits must be finite and >= 0.  Each
// thread fetches kCountUnroll elements before using them; each block adds its
// totals with one integer atomic per counter.
__global__ void __launch_bounds__(kCountThreads) short_count_kernel(
    const double *__restrict__ wait, const int32_t *__restrict__ ctx, int64_t N, double t_star,
    CountWs *counts, int *status)
{
    int64_t n_short = 0, tokens = 0;
    bool bad = false;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i0 < N;
         i0 += kCountUnroll * stride) {
        double w[kCountUnroll];
        int32_t t[kCountUnroll];
#pragma unroll
        for (int u = 0; u < kCountUnroll; ++u) {
            const int64_t i = i0 + u * stride;
            const bool in = i < N;
            w[u] = in ? wait[i] : 0.0;
            t[u] = in ? (ctx ? ctx[i] : 1) : 0;
        }
#pragma unroll
        for (int u = 0; u < kCountUnroll; ++u) {
            const bool in = i0 + u * stride < N;
            const uint64_t bits = (uint64_t)__double_as_longlong(w[u]);
            bad |= !(bits < 0x7ff0000000000000ull || bits == 0x8000000000000000ull);
            n_short += (in && w[u] <= t_star) ? 1 : 0;
            tokens += t[u];
        }
    }
    if (bad) flag_domain(status);
    n_short = wave_sum(n_short);
    tokens = wave_sum(tokens);
    __shared__ int64_t part[2][kCountThreads / kWave];
    const int lane = threadIdx.x % kWave, wv = threadIdx.x / kWave;
    if (lane == 0) {
        part[0][wv] = n_short;
        part[1][wv] = tokens;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        int64_t a = 0, b = 0;
        for (int q = 0; q < kCountThreads / kWave; ++q) {
            a += part[0][q];
            b += part[1][q];
        }
        atomicAdd(&counts->n_short, (unsigned long long)a);
        atomicAdd(&counts->tokens, (unsigned long long)b);
    }
}

__global__ void fraction_kernel(const CountWs *counts, int64_t N, int64_t *count,
                                double *fraction)
{
    if (threadIdx.x != 0) return;
    const int64_t c = (int64_t)counts->n_short;
    count[0] = c;
    if (fraction) fraction[0] = (double)c / (double)N;
}

// One block: sums of the replay's per-row counts [reps][2] (index 0 the
// timer branch, 1 host-retain), then the totals and the frozen branch.
__global__ void __launch_bounds__(256) controller_final_kernel(
    const int64_t *__restrict__ restored, const int64_t *__restrict__ admitted, int64_t reps,
    int64_t n_requests, const CountWs *counts, double t2, double t_star, double b2, double b3,
    kvr_controller_out *out)
{
    __shared__ int64_t red[4][256];
    int64_t s[4] = {0, 0, 0, 0};
    for (int64_t r = threadIdx.x; r < reps; r += blockDim.x) {
        s[0] += restored[2 * r];
        s[1] += restored[2 * r + 1];
        s[2] += admitted[2 * r];
        s[3] += admitted[2 * r + 1];
    }
    for (int k = 0; k < 4; ++k) red[k][threadIdx.x] = s[k];
    __syncthreads();
    for (int half = 128; half > 0; half >>= 1) {
        if ((int)threadIdx.x < half)
            for (int k = 0; k < 4; ++k) red[k][threadIdx.x] += red[k][threadIdx.x + half];
        __syncthreads();
    }
    if (threadIdx.x != 0) return;
    const int64_t total = (int64_t)counts->tokens;
    const int64_t n_short = (int64_t)counts->n_short;
    double cost[2];
    for (int k = 0; k < 2; ++k) {
#pragma clang fp contract(off)
        cost[k] = b2 * (double)red[k][0] + b3 * (double)(total - red[k][0]);
    }
    out->branch = (cost[0] < cost[1]) ? KVR_EXPIRE : KVR_RETAIN;
    out->restored_tokens[0] = red[0][0];
    out->restored_tokens[1] = red[1][0];
    out->admitted[0] = red[2][0];
    out->admitted[1] = red[3][0];
    out->total_tokens = total;
    out->n_short = n_short;
    out->n_requests = n_requests;
    out->t2_s = t2;
    out->total_cost[0] = cost[0];
    out->total_cost[1] = cost[1];
    out->cost_per_request[0] = cost[0] / (double)n_requests;
    out->cost_per_request[1] = cost[1] / (double)n_requests;
    out->t_star_s = t_star;
    out->p_short = (double)n_short / (double)n_requests;
}

size_t count_ws_bytes() { return 256; }

hipError_t launch_short_count(const double *wait, const int32_t *ctx, int64_t N, double t_star,
                              void *count_ws, int *status, hipStream_t stream)
{
    CountWs *c = static_cast<CountWs *>(count_ws);
    hipLaunchKernelGGL(zero_counts_kernel, dim3(1), dim3(64), 0, stream, c);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    int64_t blocks = (N + kCountThreads * 16 - 1) / (kCountThreads * 16);
    if (blocks > kCountMaxBlocks) blocks = kCountMaxBlocks;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(short_count_kernel, dim3((unsigned)blocks), dim3(kCountThreads), 0, stream,
                       wait, ctx, N, t_star, c, status);
    return hipGetLastError();
}

hipError_t launch_fraction(const void *count_ws, int64_t N, int64_t *count, double *fraction,
                           hipStream_t stream)
{
    hipLaunchKernelGGL(fraction_kernel, dim3(1), dim3(64), 0, stream,
                       static_cast<const CountWs *>(count_ws), N, count, fraction);
    return hipGetLastError();
}

hipError_t launch_controller_final(const int64_t *restored, const int64_t *admitted,
                                   int64_t reps, int64_t n_requests, const void *count_ws,
                                   double t2, double t_star, double b2, double b3,
                                   kvr_controller_out *out, hipStream_t stream)
{
    hipLaunchKernelGGL(controller_final_kernel, dim3(1), dim3(256), 0, stream, restored, admitted,
                       reps, n_requests, static_cast<const CountWs *>(count_ws), t2, t_star, b2,
                       b3, out);
    return hipGetLastError();
}

}  // namespace kvr
