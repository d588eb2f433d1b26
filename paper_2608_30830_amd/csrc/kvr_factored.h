// Internal declarations of the multiplicity-count closed form
// (kvr_factored.hip); not part of the ABI.
#pragma once

#include "kvr_internal.h"

namespace kvr {

struct FactoredWs {
    SortWs sort;              // radix sort of the base waits
    int32_t *rank;            // [n] sorted position of each base sample
    int32_t *Ts;              // [n] context size (clamped to >= 1) at each sorted position
    double *sw;               // [n] sorted waits
    int32_t *u1;              // [K1] sorted waits <= t1, then that position's query slot
    int32_t *ue;              // [K1*K2] sorted waits <= t1 + t2, then its query slot
    int32_t *qslot;           // [n+1] query slot of each sorted position, -1 if none
    uint32_t *qbits;          // [(n+32)/32] bit k: sorted position k is a query position
    int32_t *qbase;           // [(n+32)/32] query positions below each word of qbits
    int64_t nqs;              // query slots per row (an upper bound on the distinct positions)
    double2 *TQ;              // [Rb][nqs] (N, S) at each query slot: prefixes of mult x T
                              // (N, rounded to double as the closed form uses it) and of mult x T x w
    unsigned long long *tot;  // [Rb] N over every position
    int64_t Rb;               // resamples per batch
};
int64_t factored_query_slots(int64_t n, int64_t K1, int64_t P);
int64_t factored_batch(int64_t nqs, int64_t R);
hipError_t launch_factored(const SampleSrc &src, int64_t R, const Tables &tb, const PriceDev &pr,
                           FactoredWs &ws, int32_t *best, double *best_cost, double *cost_out,
                           int *status, hipStream_t stream);

}  // namespace kvr
