// Device helpers shared by the library's kernels.
#pragma once

#include "kvr_internal.h"

namespace kvr {

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

}  // namespace kvr
