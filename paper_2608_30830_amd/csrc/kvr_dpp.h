// Wave-wide scans for gfx950 by DPP moves: VALU operations that read another
// lane's register, in place of LDS shuffle rounds (ds_bpermute) and their
// lane selects.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kvr {

// DPP controls (GFX9 encoding): shift right by 1, 2, 4, 8 lanes within each
// row of 16; lane 15 of a row to the next row; lane 31 to rows 2 and 3; the
// whole wave right by one lane.
constexpr int kDppRowShr1 = 0x111;
constexpr int kDppRowShr2 = 0x112;
constexpr int kDppRowShr4 = 0x114;
constexpr int kDppRowShr8 = 0x118;
constexpr int kDppRowBcast15 = 0x142;
constexpr int kDppRowBcast31 = 0x143;
constexpr int kDppWaveShr1 = 0x138;

// A 32-bit value moved by DPP; a lane the control gives no source lane, or
// whose row the row mask leaves out, reads `old`.
template <int CTRL, int ROWM>
__device__ __forceinline__ uint32_t dpp_move32(uint32_t v, uint32_t old)
{
    return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)v, CTRL, ROWM, 0xf, false);
}

// The same for a 4- or 8-byte value (two halves), `old` given as its bits.
template <int CTRL, int ROWM, typename V>
__device__ __forceinline__ V dpp_move(V v, uint64_t old_bits)
{
    static_assert(sizeof(V) == 4 || sizeof(V) == 8, "DPP moves of 4- or 8-byte values");
    if constexpr (sizeof(V) == 4) {
        uint32_t u;
        __builtin_memcpy(&u, &v, 4);
        u = dpp_move32<CTRL, ROWM>(u, (uint32_t)old_bits);
        V r;
        __builtin_memcpy(&r, &u, 4);
        return r;
    } else {
        uint64_t u;
        __builtin_memcpy(&u, &v, 8);
        const uint32_t lo = dpp_move32<CTRL, ROWM>((uint32_t)u, (uint32_t)old_bits);
        const uint32_t hi = dpp_move32<CTRL, ROWM>((uint32_t)(u >> 32), (uint32_t)(old_bits >> 32));
        u = ((uint64_t)hi << 32) | lo;
        V r;
        __builtin_memcpy(&r, &u, 8);
        return r;
    }
}

// Inclusive sum over the 64 lanes of a wave: within each row of 16 the
// values 1, 2, 4 and 8 lanes back are added, then lane 15's sum into rows 1
// and 3 and lane 31's into rows 2 and 3.  A fixed tree: equal inputs give
// equal sums.  (For integer and floating types whose zero is all-zero bits.)
template <typename V>
__device__ __forceinline__ V wave_incl_scan(V x)
{
    x += dpp_move<kDppRowShr1, 0xf>(x, 0);
    x += dpp_move<kDppRowShr2, 0xf>(x, 0);
    x += dpp_move<kDppRowShr4, 0xf>(x, 0);
    x += dpp_move<kDppRowShr8, 0xf>(x, 0);
    x += dpp_move<kDppRowBcast15, 0xa>(x, 0);
    x += dpp_move<kDppRowBcast31, 0xc>(x, 0);
    return x;
}

// Sum over the 64 lanes in wave_incl_scan's tree, returned to every lane
// (lane 63's inclusive value, read as a scalar).
template <typename V>
__device__ __forceinline__ V wave_total(V x)
{
    static_assert(sizeof(V) == 4 || sizeof(V) == 8, "4- or 8-byte values");
    x = wave_incl_scan(x);
    if constexpr (sizeof(V) == 4) {
        uint32_t u;
        __builtin_memcpy(&u, &x, 4);
        u = (uint32_t)__builtin_amdgcn_readlane((int)u, 63);
        __builtin_memcpy(&x, &u, 4);
    } else {
        uint64_t u;
        __builtin_memcpy(&u, &x, 8);
        const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, 63);
        const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), 63);
        u = ((uint64_t)hi << 32) | lo;
        __builtin_memcpy(&x, &u, 8);
    }
    return x;
}

// The value one lane back (zero in lane 0): with an inclusive scan, the
// exclusive one.
template <typename V>
__device__ __forceinline__ V wave_lane_back(V x)
{
    return dpp_move<kDppWaveShr1, 0xf>(x, 0);
}

}  // namespace kvr
