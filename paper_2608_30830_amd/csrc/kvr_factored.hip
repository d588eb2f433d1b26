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
// Once per call: the base waits are radix-sorted; each t1 and each deadline
// gets its count of waits at or below it (a sorted position, a query), and
// the distinct query positions are numbered in order (slots).  Per batch of
// resamples: factored_prefix_kernel (one block per resample, four per CU: the
// draws' multiplicities per base sample in LDS, then, from LDS, a fixed-order
// scan of the weights c_k T_k (exact) and c_k T_k w_k over the positions that
// records N and S only at the query positions), factored_policy_kernel (one
// block per (resample, tile of 32 or 16 loads): every policy from its two slots,
// fused arg-min on the numerators m*C).
#include "kvr_device.h"
#include "kvr_dpp.h"
#include "kvr_factored.h"

namespace kvr {

constexpr int kFThreads = 1024;
constexpr int kFPThreads = 256;         // prefix kernel: four blocks (resamples) per CU
constexpr int kFLdsWords = 8192;        // 32 KiB of LDS counters per block
constexpr int kFBits = 4;               // bits of a narrow multiplicity counter
constexpr int kFPerWord = 32 / kFBits;  // narrow counters per LDS word
constexpr uint32_t kFMask = (1u << kFBits) - 1u;
constexpr int kFScanPer = 8;            // consecutive positions per thread in the scan
constexpr int kFUnroll = 8;             // draws per thread and step, fetched together
constexpr int kFLoads = 32;             // loads per policy-kernel block (16 when L <= 16)
constexpr int kFPolThreads = 256;
// Policies per thread and step in the policy kernel: 4 with 32-load tiles (two
// policies' dependent gathers more in flight, at the same three waves per
// SIMD), 2 with 16-load tiles (where 4 would cost a wave).
template <int FL> constexpr int kFPU = FL == 16 ? 2 : 4;
// Draws per resample up to which every N sum (m times a context size below
// 2^31) is an integer below 2^53, exact in double.
constexpr int64_t kFExactDoubleDraws = int64_t(1) << 22;

// One step of a wave arg-min by DPP: the (cost, index) pair CTRL names is
// merged into this lane's under the library's total order; a lane the
// control gives no source (or masks off) reads the identity (+inf, -1).
template <int CTRL, int ROWM>
__device__ __forceinline__ void dpp_argmin_step(double &c, int32_t &f)
{
    const double oc = dpp_move<CTRL, ROWM>(c, 0x7ff0000000000000ull);
    const int32_t of = dpp_move<CTRL, ROWM>(f, 0xffffffffull);
    argmin_merge(c, f, oc, of);
}

// Arg-min of (c, f) over the 64 lanes of a wave, left in lane 63: the steps
// of wave_incl_scan with the merge for the sum (the total order makes the
// result independent of the merge order).
__device__ __forceinline__ void wave_argmin_dpp(double &c, int32_t &f)
{
    dpp_argmin_step<kDppRowShr1, 0xf>(c, f);
    dpp_argmin_step<kDppRowShr2, 0xf>(c, f);
    dpp_argmin_step<kDppRowShr4, 0xf>(c, f);
    dpp_argmin_step<kDppRowShr8, 0xf>(c, f);
    dpp_argmin_step<kDppRowBcast15, 0xa>(c, f);
    dpp_argmin_step<kDppRowBcast31, 0xc>(c, f);
}

// Per sorted position k: the sorted wait and the context size there (below
// 1 counts as 1; the sort has flagged it); per base sample: its
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

__global__ void __launch_bounds__(256) factored_fill_kernel(uint32_t *__restrict__ qbits,
                                                            int64_t nwords)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < nwords) qbits[i] = 0u;
}

// Marks every query position: bit k of the position bitmask.
__global__ void __launch_bounds__(256) factored_mark_kernel(const int32_t *__restrict__ u1,
                                                            const int32_t *__restrict__ ue,
                                                            int32_t K1, int64_t P,
                                                            uint32_t *__restrict__ qbits)
{
    const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int64_t k = -1;
    if (g < K1) k = u1[g];
    else if (g - K1 < P) k = ue[g - K1];
    if (k >= 0) atomicOr(&qbits[k >> 5], 1u << (k & 31));
}

// One block: qbase[w] = the marked positions in words 0 .. w-1 (an exclusive
// scan of the words' bit counts; each thread a run of consecutive words, the
// runs across the block in order).
__global__ void __launch_bounds__(kFThreads) factored_slot_kernel(const uint32_t *__restrict__ qbits,
                                                                  int32_t *__restrict__ qbase,
                                                                  int64_t nwords)
{
    constexpr int nw = kFThreads / kWave;
    __shared__ int32_t wsum[nw];
    const int lane = threadIdx.x % kWave, wv = threadIdx.x / kWave;
    const int64_t per = (nwords + kFThreads - 1) / kFThreads;
    const int64_t w0 = (int64_t)threadIdx.x * per;
    const int64_t w1 = (w0 + per < nwords) ? w0 + per : nwords;
    int32_t cnt = 0;
    for (int64_t w = w0; w < w1; ++w) cnt += __popc(qbits[w]);
    int32_t x = cnt;   // inclusive scan of the run totals within the wave
    for (int off = 1; off < kWave; off <<= 1) {
        const int32_t y = __shfl_up(x, off, kWave);
        if (lane >= off) x += y;
    }
    if (lane == kWave - 1) wsum[wv] = x;
    __syncthreads();
    int32_t next = x - cnt;
    for (int q = 0; q < wv; ++q) next += wsum[q];
    for (int64_t w = w0; w < w1; ++w) {
        qbase[w] = next;
        next += __popc(qbits[w]);
    }
}

// Slot of a marked position k: the marks below it.
__device__ __forceinline__ int32_t slot_of(const uint32_t *__restrict__ qbits,
                                           const int32_t *__restrict__ qbase, int64_t k)
{
    const uint32_t below = (1u << (k & 31)) - 1u;
    return qbase[k >> 5] + __popc(qbits[k >> 5] & below);
}

// Items 0..K1-1 and K1..K1+P-1: u1[a] and ue[f] from sorted positions to
// slots; items K1+P .. K1+P+n: the slot of each sorted position 0..n, -1 if
// it is no query position.
__global__ void __launch_bounds__(256) factored_remap_kernel(int32_t *__restrict__ u1,
                                                             int32_t *__restrict__ ue, int32_t K1,
                                                             int64_t P, int64_t n,
                                                             const uint32_t *__restrict__ qbits,
                                                             const int32_t *__restrict__ qbase,
                                                             int32_t *__restrict__ qslot)
{
    const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (g < K1) {
        u1[g] = slot_of(qbits, qbase, u1[g]);
    } else if (g - K1 < P) {
        ue[g - K1] = slot_of(qbits, qbase, ue[g - K1]);
    } else if (g - K1 - P <= n) {
        const int64_t k = g - K1 - P;
        qslot[k] = ((qbits[k >> 5] >> (k & 31)) & 1u) ? slot_of(qbits, qbase, k) : -1;
    }
}

// One block per resample of the batch.  Per pass over a range of sorted
// positions: the number of the resample's draws of each position, counted in
// LDS, then a scan over the range in a fixed order (each thread its
// kFScanPer consecutive positions, the thread totals across the block: the
// lanes of a wave in wave_incl_scan's tree, the waves in order, then the
// earlier passes), which records
// at every query position k N(k) = sum_{j < k} c_j T_j (exact, then rounded
// to double as the closed form uses it) and S(k) = sum_{j < k} c_j T_j w_j
// (reproducible) in the query row, one 16-byte record per slot so that a
// policy's two lookups are two loads.  Position n (every wait) closes the
// row; tot[rb] = N(n).
//
// Counters: kFBits-bit fields of 32-bit LDS words, kFLdsWords * kFPerWord
// positions per pass (32 KiB, so that four blocks share a CU and one's
// barriers and loads overlap the others').  When that covers every position
// the draws are counted by base sample instead (no rank gather per draw) and
// the scan reads each position's count through the sort order.  A field that
// passes its maximum carries into (or out of) its word, and that only ever
// lowers the decoded total (a carry turns 2^kFBits counts into 1), so
// comparing the decoded total with the number of draws in the range (counted
// exactly) detects it; the resample then restarts with 32-bit counters by
// sorted position, kFLdsWords positions per pass.  A bootstrap row's
// multiplicities are Poisson(1)-like, so 4-bit fields almost never wrap.
// NT carries the N sums: double when every sum is an integer below 2^53 (the
// host picks it for m <= 2^22, a context size being below 2^31), where it is
// exact in any order and costs fewer instructions than 64-bit integers;
// unsigned 64-bit otherwise.
template <typename NT>
__global__ void __launch_bounds__(kFPThreads) factored_prefix_kernel(
    const int32_t *__restrict__ idx, int64_t n, int64_t m, int64_t r0,
    const int32_t *__restrict__ rank, const int32_t *__restrict__ perm,
    const int32_t *__restrict__ Ts,
    const double *__restrict__ sw, const int32_t *__restrict__ qslot, int64_t nqs,
    double2 *__restrict__ TQ, unsigned long long *__restrict__ tot, int *status)
{
    constexpr int nw = kFPThreads / kWave;
    constexpr int kTile = kFPThreads * kFScanPer;
    __shared__ uint32_t lh[kFLdsWords];
    __shared__ NT wn[nw];
    __shared__ double wsd[nw];
    __shared__ long long wchk[nw];
    const int64_t rb = blockIdx.x;
    const int64_t r = r0 + rb;
    double2 *qrow = TQ + rb * nqs;
    const int lane = threadIdx.x % kWave, wv = threadIdx.x / kWave;
    const int64_t B = blockDim.x;
    NT carry_n = 0;   // totals of the earlier positions (same in every thread)
    double carry_s = 0.0;
    for (int wide = 0; wide < 2; ++wide) {
        const int64_t PP = wide ? kFLdsWords : kFPerWord * (int64_t)kFLdsWords;   // positions per pass
        bool overflow = false;
        carry_n = 0;
        carry_s = 0.0;
        for (int64_t k0 = 0; k0 < n && !overflow; k0 += PP) {
            const int64_t nk = (n - k0 < PP) ? n - k0 : PP;
            const int64_t nwords = wide ? nk : (nk + kFPerWord - 1) / kFPerWord;
            // narrow counters over every position at once (n <= PP): count by
            // base sample instead of sorted position, so a draw needs no rank
            // gather; the scan then finds each position's count through perm
            const bool byidx = !wide && nk == n;
            for (int64_t x = threadIdx.x; x < nwords; x += B) lh[x] = 0u;
            __syncthreads();
            long long inr = 0;                              // draws counted in this range
            for (int64_t j = threadIdx.x; j < m; j += kFUnroll * B) {
                // the kFUnroll draws are loaded unconditionally (a position past
                // the row re-reads its last draw and is dropped) and checked with
                // selects and one branch for all, so the index loads, and then
                // the rank gathers, are in flight together
                int32_t ii[kFUnroll];
                bool live[kFUnroll];
#pragma unroll
                for (int u = 0; u < kFUnroll; ++u) {
                    live[u] = j + u * B < m;
                    ii[u] = idx[r * m + (live[u] ? j + u * B : m - 1)];
                }
                bool bad = false;
#pragma unroll
                for (int u = 0; u < kFUnroll; ++u) {
                    const bool out = ii[u] < 0 || (int64_t)ii[u] >= n;
                    bad = bad || (live[u] && out);
                    ii[u] = out ? 0 : ii[u];                // a bad draw counts as sample 0
                }
                if (bad) flag_domain(status);
                int64_t kk[kFUnroll];
#pragma unroll
                for (int u = 0; u < kFUnroll; ++u) {
                    kk[u] = byidx ? (int64_t)ii[u] : (int64_t)rank[ii[u]] - k0;
                    if (!live[u]) kk[u] = -1;                // past the row: no draw
                }
#pragma unroll
                for (int u = 0; u < kFUnroll; ++u) {
                    if (kk[u] >= 0 && kk[u] < nk) {
                        ++inr;
                        if (wide) atomicAdd(&lh[kk[u]], 1u);
                        else atomicAdd(&lh[kk[u] / kFPerWord], 1u << (kFBits * (int)(kk[u] % kFPerWord)));
                    }
                }
            }
            __syncthreads();
            if (!wide) {
                // decoded total minus the draws counted, over the whole block
                long long d = -inr;
                for (int64_t x = threadIdx.x; x < nwords; x += B) {
                    const uint32_t v = lh[x];
#pragma unroll
                    for (int h = 0; h < kFPerWord; ++h) d += (long long)((v >> (kFBits * h)) & kFMask);
                }
                d = wave_sum(d);
                if (lane == 0) wchk[wv] = d;
                __syncthreads();
                long long all = 0;
                for (int q = 0; q < nw; ++q) all += wchk[q];
                overflow = all != 0;                        // the same in every thread
                __syncthreads();
                if (overflow) break;
            }
            for (int64_t base = 0; base < nk; base += kTile) {
                const int64_t kl = base + (int64_t)threadIdx.x * kFScanPer;   // position in the pass
                NT cw[kFScanPer];
                double sv[kFScanPer];
                int32_t qs[kFScanPer];
                NT tn = 0;
                double ts = 0.0;
                // a full run of kFScanPer positions starts on a multiple of
                // kFScanPer (pass starts are multiples of 2^14): 16-byte loads
                // of Ts, qslot and perm (4 positions) and of sw (2) instead of
                // an element each
                int32_t tv[kFScanPer], qv[kFScanPer], pv[kFScanPer];
                double wv4[kFScanPer];
                if (kl + kFScanPer <= nk) {
                    static_assert(kFScanPer % 4 == 0, "the vector loads below read 4 positions");
#pragma unroll
                    for (int h = 0; h < kFScanPer; h += 4) {
                        const int4 t4 = *reinterpret_cast<const int4 *>(Ts + k0 + kl + h);
                        const int4 q4 = *reinterpret_cast<const int4 *>(qslot + k0 + kl + h);
                        const double2 w0 = reinterpret_cast<const double2 *>(sw + k0 + kl + h)[0];
                        const double2 w1 = reinterpret_cast<const double2 *>(sw + k0 + kl + h)[1];
                        tv[h] = t4.x; tv[h + 1] = t4.y; tv[h + 2] = t4.z; tv[h + 3] = t4.w;
                        qv[h] = q4.x; qv[h + 1] = q4.y; qv[h + 2] = q4.z; qv[h + 3] = q4.w;
                        wv4[h] = w0.x; wv4[h + 1] = w0.y; wv4[h + 2] = w1.x; wv4[h + 3] = w1.y;
                        if (byidx) {
                            const int4 p4 = *reinterpret_cast<const int4 *>(perm + k0 + kl + h);
                            pv[h] = p4.x; pv[h + 1] = p4.y; pv[h + 2] = p4.z; pv[h + 3] = p4.w;
                        }
                    }
                } else {
#pragma unroll
                    for (int q = 0; q < kFScanPer; ++q) {
                        const int64_t k = kl + q;
                        tv[q] = (k < nk) ? Ts[k0 + k] : 0;
                        qv[q] = (k < nk) ? qslot[k0 + k] : -1;
                        wv4[q] = (k < nk) ? sw[k0 + k] : 0.0;
                        if (byidx) pv[q] = (k < nk) ? perm[k0 + k] : 0;
                    }
                }
#pragma unroll
                for (int q = 0; q < kFScanPer; ++q) {
                    const int64_t k = kl + q;
                    const bool in = k < nk;
                    uint32_t c = 0u;
                    // the counter of position k, or of the base sample there
                    const int64_t ck = byidx ? (int64_t)((uint32_t)pv[q] < (uint32_t)n ? pv[q] : 0) : k;
                    if (in) c = wide ? lh[k] : (lh[ck / kFPerWord] >> (kFBits * (int)(ck % kFPerWord))) & kFMask;
                    const NT cwq = in ? (NT)c * (NT)tv[q] : (NT)0;   // exact
                    cw[q] = cwq;
                    sv[q] = (double)cwq * wv4[q];
                    qs[q] = in ? qv[q] : -1;
                    tn += cwq;
                    ts += sv[q];
                }
                // scan of the thread totals in the wave (DPP moves, a fixed tree)
                const NT xn = wave_incl_scan(tn), en = wave_lane_back(xn);
                const double xs = wave_incl_scan(ts), es = wave_lane_back(xs);
                if (lane == kWave - 1) {
                    wn[wv] = xn;
                    wsd[wv] = xs;
                }
                __syncthreads();
                NT pn = carry_n;
                double ps = carry_s;
                for (int q = 0; q < wv; ++q) {
                    pn += wn[q];
                    ps += wsd[q];
                }
                pn += en;
                ps += es;
                for (int q = 0; q < nw; ++q) {
                    carry_n += wn[q];
                    carry_s += wsd[q];
                }
#pragma unroll
                for (int q = 0; q < kFScanPer; ++q) {
                    if (qs[q] >= 0 && qs[q] < nqs) qrow[qs[q]] = make_double2((double)pn, ps);
                    pn += cw[q];
                    ps += sv[q];
                }
                __syncthreads();   // wn and wsd are rewritten by the next tile
            }
        }
        if (!overflow) break;
    }
    if (threadIdx.x == 0) {
        const int32_t q = qslot[n];
        if (q >= 0 && q < nqs) qrow[q] = make_double2((double)carry_n, carry_s);
        tot[rb] = (unsigned long long)carry_n;
    }
}

// One block per (resample of the batch, tile of FL loads): every policy's
// closed-form total m*C for the tile's loads, the optional cost output, and
// the arg-min per load under the library's total order (smaller first, then
// larger flat index).  Dividing by m is monotone, so the arg-min compares the
// totals and only the selected one is divided.
template <int FL>
__global__ void __launch_bounds__(kFPolThreads) factored_policy_kernel(
    const double2 *__restrict__ TQ, int64_t nqs,
    const unsigned long long *__restrict__ totN, int64_t m, int64_t r0, int ntl, Tables tb,
    PriceDev pr, const int32_t *__restrict__ u1, const int32_t *__restrict__ ue,
    int32_t *__restrict__ best, double *__restrict__ best_cost, double *__restrict__ cost_out)
{
    constexpr int nw = kFPolThreads / kWave;
    __shared__ double rc[nw][FL];
    __shared__ int32_t rf[nw][FL];
    const int64_t rb = blockIdx.x / ntl;
    const int tile = (int)(blockIdx.x % ntl);
    const int64_t r = r0 + rb;
    const double2 *qrow = TQ + rb * nqs;   // (N, S) at the query slots
    const int64_t P = (int64_t)tb.K1 * tb.K2;
    const int l0 = tile * FL;
    const int nl = (tb.L - l0 < FL) ? tb.L - l0 : FL;
    const double tot = (double)totN[rb];
    const double md = (double)m;
    double a2[FL], bc[FL];
    int32_t bf[FL];
#pragma unroll
    for (int l = 0; l < FL; ++l) {
        a2[l] = tb.a2[l0 + l];   // zero-padded to whole tiles
        bc[l] = INFINITY;
        bf[l] = -1;
    }
    // kFPU<FL> policies per thread and step: their slots, then their prefix
    // values, are fetched together before any is used.  P < 2^24, so policy
    // indices are split in 32-bit arithmetic.
    const uint32_t B = blockDim.x, K2 = (uint32_t)tb.K2, P32 = (uint32_t)P;
    for (uint32_t f0 = threadIdx.x; f0 < P32; f0 += kFPU<FL> * B) {
        int32_t p1[kFPU<FL>], pe[kFPU<FL>];
        double t1[kFPU<FL>], e[kFPU<FL>];
#pragma unroll
        for (int u = 0; u < kFPU<FL>; ++u) {
            const uint32_t f = (f0 + u * B < P32) ? f0 + u * B : f0;   // a repeat of f0 is skipped below
            const uint32_t a = f / K2, k = f - a * K2;
            t1[u] = tb.t1[a];
            e[u] = t1[u] + tb.t2[k];
            p1[u] = u1[a];
            pe[u] = ue[f];
        }
        double n1[kFPU<FL>], ne[kFPU<FL>], s1[kFPU<FL>], se[kFPU<FL>];
#pragma unroll
        for (int u = 0; u < kFPU<FL>; ++u) {   // one 16-byte record per slot
            const double2 q1 = qrow[p1[u]], qe = qrow[pe[u]];
            n1[u] = q1.x;
            s1[u] = q1.y;
            ne[u] = qe.x;
            se[u] = qe.y;
        }
#pragma unroll
        for (int u = 0; u < kFPU<FL>; ++u) {
            const uint32_t f = f0 + u * B;
            if (f >= P32) break;
            const double hbm = s1[u] + t1[u] * (tot - n1[u]);
            double hold = (se[u] - s1[u]) - t1[u] * (ne[u] - n1[u]);
            if (!isinf(e[u])) hold = hold + (e[u] - t1[u]) * (tot - ne[u]);
            const double fixed = pr.a1 * hbm + pr.b2 * (ne[u] - n1[u]) + pr.b3 * (tot - ne[u]);
            if (cost_out != nullptr) {   // unrolled, so that a2 stays in registers
#pragma unroll
                for (int l = 0; l < FL; ++l)
                    if (l < nl) cost_out[(r * tb.L + l0 + l) * P + f] = (fixed + a2[l] * hold) / md;
            }
            // every load of the tile (a2 is zero-padded past L; those lanes are
            // never stored); a thread visits its policies in increasing f, so
            // "not larger" keeps the larger index on a tie, as the total order
            // asks; the running minimum itself is a min (equal on a tie)
#pragma unroll
            for (int l = 0; l < FL; ++l) {
                const double tc = fixed + a2[l] * hold;
                const bool take = tc <= bc[l];
                bc[l] = fmin(bc[l], tc);
                bf[l] = take ? (int32_t)f : bf[l];
            }
        }
    }
    const int lane = threadIdx.x % kWave, wv = threadIdx.x / kWave;
#pragma unroll
    for (int l = 0; l < FL; ++l) {
        wave_argmin_dpp(bc[l], bf[l]);
        if (lane == kWave - 1) {
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

int64_t factored_query_slots(int64_t n, int64_t K1, int64_t P)
{
    // distinct query positions: at most one per t1 and deadline, at most n + 1
    return (K1 + P < n + 1) ? K1 + P : n + 1;
}

int64_t factored_batch(int64_t nqs, int64_t R)
{
    // at most 2 GiB of query rows per batch, and batches of equal size (a
    // short last batch would leave most of the chip idle)
    const int64_t per = nqs * 16 + 8;
    int64_t rb = ((int64_t)1 << 31) / per;
    if (rb < 1) rb = 1;
    if (rb >= R) return R;
    const int64_t nb = (R + rb - 1) / rb;
    return (R + nb - 1) / nb;
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
    const unsigned gq = (unsigned)((tb.K1 + P + 255) / 256);
    hipLaunchKernelGGL(factored_bounds_kernel, dim3(gq), dim3(256), 0, stream, ws.sw, n, tb, ws.u1,
                       ws.ue);
    const int64_t nwords = (n + 1 + 31) / 32;
    hipLaunchKernelGGL(factored_fill_kernel, dim3((unsigned)((nwords + 255) / 256)), dim3(256), 0,
                       stream, ws.qbits, nwords);
    hipLaunchKernelGGL(factored_mark_kernel, dim3(gq), dim3(256), 0, stream, ws.u1, ws.ue, tb.K1, P,
                       ws.qbits);
    hipLaunchKernelGGL(factored_slot_kernel, dim3(1), dim3(kFThreads), 0, stream, ws.qbits, ws.qbase,
                       nwords);
    hipLaunchKernelGGL(factored_remap_kernel, dim3((unsigned)((tb.K1 + P + n + 1 + 255) / 256)),
                       dim3(256), 0, stream, ws.u1, ws.ue, tb.K1, P, n, ws.qbits, ws.qbase,
                       ws.qslot);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    const int FL = tb.L <= 16 ? 16 : kFLoads;                 // loads per policy block
    const int ntl = (tb.L + FL - 1) / FL;
    for (int64_t r0 = 0; r0 < R; r0 += ws.Rb) {
        const int64_t rb = (R - r0 < ws.Rb) ? R - r0 : ws.Rb;
        if (m <= kFExactDoubleDraws)
            hipLaunchKernelGGL(factored_prefix_kernel<double>, dim3((unsigned)rb),
                               dim3(kFPThreads), 0, stream, src.idx, n, m, r0, ws.rank,
                               ws.sort.vals[cur], ws.Ts, ws.sw, ws.qslot, ws.nqs, ws.TQ, ws.tot,
                               status);
        else
            hipLaunchKernelGGL(factored_prefix_kernel<unsigned long long>, dim3((unsigned)rb),
                               dim3(kFPThreads), 0, stream, src.idx, n, m, r0, ws.rank,
                               ws.sort.vals[cur], ws.Ts, ws.sw, ws.qslot, ws.nqs, ws.TQ, ws.tot,
                               status);
        if (FL == 16)
            hipLaunchKernelGGL(factored_policy_kernel<16>, dim3((unsigned)(rb * ntl)),
                               dim3(kFPolThreads), 0, stream, ws.TQ, ws.nqs, ws.tot, m, r0,
                               ntl, tb, pr, ws.u1, ws.ue, best, best_cost, cost_out);
        else
            hipLaunchKernelGGL(factored_policy_kernel<kFLoads>, dim3((unsigned)(rb * ntl)),
                               dim3(kFPolThreads), 0, stream, ws.TQ, ws.nqs, ws.tot, m, r0,
                               ntl, tb, pr, ws.u1, ws.ue, best, best_cost, cost_out);
        if ((err = hipGetLastError()) != hipSuccess) return err;
    }
    return hipSuccess;
}

}  // namespace kvr
