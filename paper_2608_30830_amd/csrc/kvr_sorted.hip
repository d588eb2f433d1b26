// Sorted path for gfx950: stable LSD radix sort of the waits, prefix scans of
// T and T*w in sorted order, and the closed-form mean cost per policy.
//
// With the waits sorted and N(x) = sum_{w_i <= x} T_i, S(x) = sum_{w_i <= x} T_i w_i,
// integrating the per-request cost of Eq. 1 (HBM until t1, host until the
// deadline e = t1 + t2 at the Eq. 3 price, restore or recompute at resume)
// over the sample gives, with Ttot = N(inf):
//   n*C = a1*[S(t1) + t1*(Ttot - N(t1))]
//       + a2*[(S(e) - S(t1)) - t1*(N(e) - N(t1)) + (e - t1)*(Ttot - N(e))]
//       + b2*(N(e) - N(t1)) + b3*(Ttot - N(e));
// the (e - t1)*(Ttot - N(e)) term is absent for e = +inf.
//
// Sort: keys are the bits of w + 0.0 (waits are >= 0, so unsigned order of
// the bits is numeric order and -0.0 sorts as +0.0).  Eight 8-bit digit
// passes, each reduce-then-scan (tile histograms, one exclusive scan, a
// ranking scatter); no inter-workgroup waiting, so no forward-progress
// assumption.  Ranking inside a tile is stable: a wave ranks its keys with a
// ballot match on the digit, in input order.  The first pass reads the waits
// themselves (its histograms come straight from them, so no key array is
// written before it); from 2^22 keys each scatter also writes the next digit
// as one byte per key, which the next histogram reads instead of the keys.
//
// Scans: the closed form needs N and S only at t1, at each deadline and at
// the whole sample.  Without a requested order they are formed there, from
// the scan tiles' exclusive prefixes and the sums of every run of 64 sorted
// positions; with an order requested (or very many policies) the full
// inclusive prefix arrays are written and read.
#include "kvr_device.h"
#include "kvr_dpp.h"

#include <type_traits>

namespace kvr {

constexpr int kSortThreads = 256;
constexpr int kSortKPT = 8;                                   // keys per thread
constexpr int kSortTile = kSortThreads * kSortKPT;            // 2048 keys per tile
constexpr int kScanThreads = 256;
constexpr int kScanIPT = 8;
constexpr int kScanTile = kScanThreads * kScanIPT;

static inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
static inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Keys per thread of the multi-block sort: the largest tile (256 * kpt keys,
// kpt = 2, 4, 8 or 16) that still gives about one block per CU, since below
// that each pass is bound by the length of a block's chain (measured on
// MI355X: 65,536 keys 0.150 ms with kpt = 2 against 0.203 ms with 8; 2^20
// keys 0.31 ms with 8 against 0.41 ms with 2).  Longer tiles also give each
// digit longer runs of consecutive destinations: at 2^24 keys a scatter pass
// writes exactly its 24 algorithmic bytes per key with 4,096-key tiles (103 us)
// and 12-37 % more with 2,048-key tiles (129-134 us); at 2^22 keys the shorter
// tiles still win (23.4 against 29.4 us), having twice the blocks.
static int sort_kpt(int64_t n)
{
    return n >= (int64_t(1) << 23) ? 16 : n >= (int64_t(1) << 19) ? 8 : n >= (int64_t(1) << 18) ? 4 : 2;
}

size_t sort_ws_bytes(int64_t n)
{
    const int64_t nb = cdiv(n, kSortThreads * sort_kpt(n)), ns = cdiv(n, kScanTile);
    size_t b = 0;
    b += 2 * align256(sizeof(uint64_t) * n);
    b += 2 * align256(sizeof(int32_t) * n);
    b += align256(sizeof(uint32_t) * 256 * nb);
    b += align256(sizeof(uint32_t) * 256);
    b += align256(sizeof(int64_t) * n);
    b += align256(sizeof(double) * n);
    b += align256(sizeof(int64_t) * ns);
    b += align256(sizeof(double) * ns);
    return b;
}

void sort_ws_carve(void *base, int64_t n, SortWs &ws)
{
    char *p = static_cast<char *>(base);
    ws.kpt = sort_kpt(n);
    ws.nblocks = (int)cdiv(n, kSortThreads * ws.kpt);
    ws.nblocks_scan = (int)cdiv(n, kScanTile);
    auto take = [&](size_t bytes) {
        char *q = p;
        p += align256(bytes);
        return q;
    };
    ws.keys[0] = (uint64_t *)take(sizeof(uint64_t) * n);
    ws.keys[1] = (uint64_t *)take(sizeof(uint64_t) * n);
    ws.vals[0] = (int32_t *)take(sizeof(int32_t) * n);
    ws.vals[1] = (int32_t *)take(sizeof(int32_t) * n);
    ws.hist = (uint32_t *)take(sizeof(uint32_t) * 256 * ws.nblocks);
    ws.counts = (uint32_t *)take(sizeof(uint32_t) * 256);
    ws.Nsum = (int64_t *)take(sizeof(int64_t) * n);
    ws.Ssum = (double *)take(sizeof(double) * n);
    ws.blkN = (int64_t *)take(sizeof(int64_t) * ws.nblocks_scan);
    ws.blkS = (double *)take(sizeof(double) * ws.nblocks_scan);
}

// Sort tiles are numbered so that each XCD takes a contiguous range of them:
// neighbouring tiles share the cache lines of the digit-major histogram and of
// its scanned offsets, and then share them in one L2.
__device__ __forceinline__ int sort_tile(int nblocks)
{
    return (int)xcd_logical_block(blockIdx.x, nblocks);
}

// Key of a wait: its bits, with -0.0 as +0.0 (waits are >= 0, so the
// unsigned order of the bits is numeric order); a NaN, an infinity or a
// negative wait sets bad and becomes key 0.
__device__ __forceinline__ uint64_t wait_key(double x, bool &bad)
{
    uint64_t b = (uint64_t)__double_as_longlong(x);
    if (b == 0x8000000000000000ull) b = 0;
    if (b >= 0x7ff0000000000000ull) {
        bad = true;
        b = 0;
    }
    return b;
}

// Tile histograms of the first digit straight from the waits (domain-checked
// on the bits), so that the first scatter can read the waits and context
// sizes itself and no key array is written before it.  Tiles are those of the
// digit passes (256 * KPT keys); digit-major histogram hist[d * nblocks + tile].
template <int KPT>
__global__ void __launch_bounds__(kSortThreads) sort_first_hist_kernel(
    const double *__restrict__ w, int64_t n, uint32_t *__restrict__ hist, int nblocks,
    int *status)
{
    __shared__ uint32_t h[256];
    h[threadIdx.x] = 0;
    __syncthreads();
    const int tile = sort_tile(nblocks);
    const int64_t base = (int64_t)tile * (kSortThreads * KPT);
    double x[KPT];
#pragma unroll
    for (int q = 0; q < KPT; ++q) {   // every load in flight before counting
        const int64_t i = base + q * kSortThreads + threadIdx.x;
        x[q] = i < n ? w[i] : 0.0;
    }
    bool bad = false;
#pragma unroll
    for (int q = 0; q < KPT; ++q)
        if (base + q * kSortThreads + threadIdx.x < n) atomicAdd(&h[wait_key(x[q], bad) & 255u], 1u);
    if (bad) flag_domain(status);
    __syncthreads();
    hist[(int64_t)threadIdx.x * nblocks + tile] = h[threadIdx.x];
}

__device__ __forceinline__ uint32_t lanes_below(uint64_t mask)
{
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                     __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

// Lanes of the wave whose (valid) digit equals this lane's: a ballot per bit.
__device__ __forceinline__ uint64_t digit_peers(uint32_t d, bool valid)
{
    uint64_t peers = __ballot(valid);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
        const bool bit = (d >> b) & 1u;
        const uint64_t m = __ballot(bit);
        peers &= bit ? m : ~m;
    }
    return peers;
}

// Per-tile digit histogram (tiles of 256 * KPT keys), digit-major:
// hist[d * nblocks + tile].  The keys of a wave that share the first lane's
// digit add their count through that lane, the others one by one: when most
// keys hold one digit (the high bytes of waits spread over a few binades)
// this replaces up to 64 atomics on one LDS word by one.
template <int KPT>
__global__ void __launch_bounds__(kSortThreads) sort_hist_kernel(const uint64_t *__restrict__ keys,
                                                                 int64_t n, int shift,
                                                                 uint32_t *__restrict__ hist,
                                                                 int nblocks)
{
    __shared__ uint32_t h[256];
    h[threadIdx.x] = 0;
    __syncthreads();
    const int tile = sort_tile(nblocks);
    const int64_t base = (int64_t)tile * (kSortThreads * KPT);
    uint64_t key[KPT];
#pragma unroll
    for (int q = 0; q < KPT; ++q) {
        const int64_t i = base + q * kSortThreads + threadIdx.x;
        key[q] = i < n ? keys[i] : 0;
    }
    const int lane = threadIdx.x % kWave;
#pragma unroll
    for (int q = 0; q < KPT; ++q) {
        const bool valid = base + q * kSortThreads + threadIdx.x < n;
        const uint32_t d = (uint32_t)(key[q] >> shift) & 255u;
        const uint32_t d0 = __builtin_amdgcn_readfirstlane(d);
        const uint64_t same = __ballot(valid && d == d0);
        if (lane == 0 && same != 0) atomicAdd(&h[d0], (uint32_t)__popcll(same));
        else if (valid && d != d0) atomicAdd(&h[d], 1u);
    }
    __syncthreads();
    hist[(int64_t)threadIdx.x * nblocks + tile] = h[threadIdx.x];
}

// The same histogram from the digit bytes that the previous pass's scatter
// wrote beside the keys (dig[i] = this pass's digit of the key at i): one
// byte per key read instead of eight.  A tile's count does not depend on the
// order of its keys, so each thread reads KPT consecutive bytes in one load;
// bytes past n (up to the end of the last tile, inside the buffer) are not
// counted.
template <int KPT>
__global__ void __launch_bounds__(kSortThreads) sort_hist_bytes_kernel(
    const uint8_t *__restrict__ dig, int64_t n, uint32_t *__restrict__ hist, int nblocks)
{
    using Vec = typename std::conditional<
        KPT == 16, uint4,
        typename std::conditional<KPT == 8, uint2,
                                  typename std::conditional<KPT == 4, uint32_t, uint16_t>::type>::type>::type;
    static_assert(sizeof(Vec) == KPT, "one load of KPT bytes");
    __shared__ uint32_t h[256];
    h[threadIdx.x] = 0;
    __syncthreads();
    const int tile = sort_tile(nblocks);
    const int64_t i0 = (int64_t)tile * (kSortThreads * KPT) + (int64_t)threadIdx.x * KPT;
    const Vec v = *reinterpret_cast<const Vec *>(dig + i0);
    uint8_t b[KPT];
    __builtin_memcpy(b, &v, KPT);
    const int lane = threadIdx.x % kWave;
#pragma unroll
    for (int q = 0; q < KPT; ++q) {
        const bool valid = i0 + q < n;
        const uint32_t d = b[q];
        const uint32_t d0 = __builtin_amdgcn_readfirstlane(d);
        const uint64_t same = __ballot(valid && d == d0);
        if (lane == 0 && same != 0) atomicAdd(&h[d0], (uint32_t)__popcll(same));
        else if (valid && d != d0) atomicAdd(&h[d], 1u);
    }
    __syncthreads();
    hist[(int64_t)threadIdx.x * nblocks + tile] = h[threadIdx.x];
}

// Exclusive scan, within one block of 256 threads, of one value per thread;
// returns the prefix and writes the block total to *total (all threads).
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t *total)
{
    __shared__ uint32_t wsum[4];
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const uint32_t x = wave_incl_scan(v);
    if (lane == kWave - 1) wsum[wave] = x;
    __syncthreads();
    uint32_t before = 0;
    for (int q = 0; q < wave; ++q) before += wsum[q];
    *total = wsum[0] + wsum[1] + wsum[2] + wsum[3];
    __syncthreads();
    return before + x - v;
}

// Exclusive scan over the 1,024 threads of a block of one value per thread
// (a fixed order: wave_incl_scan's tree within each wave, then the wave totals
// in order); *total receives the block's sum.
template <typename V>
__device__ __forceinline__ V block1024_exclusive_scan(V v, V *total)
{
    __shared__ V wsum[1024 / kWave];
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const V x = wave_incl_scan(v);
    const V ex = wave_lane_back(x);
    if (lane == kWave - 1) wsum[wave] = x;
    __syncthreads();
    V before = 0, all = 0;
    for (int q = 0; q < 1024 / kWave; ++q) {
        if (q < wave) before += wsum[q];
        all += wsum[q];
    }
    *total = all;
    __syncthreads();
    return before + ex;
}

// One block of 1,024 threads per digit: exclusive scan of that digit's
// per-tile counts over the tiles (in place) and the digit's total.  Each
// thread takes a run of consecutive tiles, so the row is scanned in one round.
constexpr int kRunRegs = 8;   // runs up to this length stay in registers (8,192 tiles)

__global__ void __launch_bounds__(1024) digit_scan_kernel(uint32_t *__restrict__ hist, int nblocks,
                                                          uint32_t *__restrict__ totals)
{
    uint32_t *row = hist + (int64_t)blockIdx.x * nblocks;
    const int per = (nblocks + 1023) / 1024;
    const int64_t t0 = (int64_t)threadIdx.x * per;
    int64_t t1 = t0 + per;
    if (t1 > nblocks) t1 = nblocks;
    uint32_t all;
    if (per <= kRunRegs) {   // uniform: the row passes through LDS with coalesced accesses
        __shared__ uint32_t lrow[1024 * kRunRegs];
        for (int t = threadIdx.x; t < nblocks; t += 1024) lrow[t] = row[t];
        __syncthreads();
        uint32_t c[kRunRegs];
        uint32_t sum = 0;
#pragma unroll
        for (int i = 0; i < kRunRegs; ++i) {
            c[i] = (t0 + i < t1) ? lrow[t0 + i] : 0u;
            sum += c[i];
        }
        uint32_t run = block1024_exclusive_scan(sum, &all);
#pragma unroll
        for (int i = 0; i < kRunRegs; ++i) {
            if (t0 + i < t1) lrow[t0 + i] = run;
            run += c[i];
        }
        __syncthreads();
        for (int t = threadIdx.x; t < nblocks; t += 1024) row[t] = lrow[t];
    } else {
        uint32_t sum = 0;
        for (int64_t t = t0; t < t1; ++t) sum += row[t];
        uint32_t run = block1024_exclusive_scan(sum, &all);
        for (int64_t t = t0; t < t1; ++t) {
            const uint32_t c = row[t];
            row[t] = run;
            run += c;
        }
    }
    if (threadIdx.x == 0) totals[blockIdx.x] = all;
}

// Stable ranking scatter of one digit pass.  The destination of a key is
// (keys with a smaller digit) + (keys with its digit in earlier tiles, from
// digit_scan_kernel) + (keys with its digit earlier in this tile).  The tile
// is first reordered by digit in LDS, then written out in that order, so
// consecutive threads store consecutive addresses within each digit's run.
template <int KPT, bool FIRST>
__global__ void __launch_bounds__(kSortThreads) sort_scatter_kernel(
    const uint64_t *__restrict__ keys_in, const int32_t *__restrict__ vals_in,
    const double *__restrict__ w, const int32_t *__restrict__ T, int payload_T, int64_t n,
    int shift, const uint32_t *__restrict__ offs, const uint32_t *__restrict__ totals, int nblocks,
    uint64_t *__restrict__ keys_out, int32_t *__restrict__ vals_out, uint8_t *__restrict__ dig_out,
    int *status)
{
    // 16-bit counters and 32-bit bases keep a block at 27.5 KiB of LDS at
    // 2,048-key tiles (five resident blocks per CU) and at 51.5 KiB at 4,096
    // (three; with a separate offset table, 53.5 KiB, two): a wave holds at
    // most 64 * KPT keys, a tile at most 4,096, and a destination fits 32 bits
    // (n < 2^31).  wcnt holds the waves' digit counts, then, in place, each
    // wave's first tile position within its digit (wofs)
    __shared__ uint16_t wcnt[4][256];
    auto &wofs = wcnt;
    __shared__ int32_t gbase[256];                   // destination of digit d's first tile key
    constexpr int kTile = kSortThreads * KPT, kWaveK = kWave * KPT;
    __shared__ uint64_t lkey[kTile];
    __shared__ int32_t lval[kTile];
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const int tile = sort_tile(nblocks);
    // this tile's offset within digit threadIdx.x, loaded early (its latency
    // overlaps the ranking below)
    const uint32_t my_off = offs[(int64_t)threadIdx.x * nblocks + tile];
#pragma unroll
    for (int q = 0; q < 4; ++q) wcnt[q][threadIdx.x] = 0;
    uint32_t dbase;
    {
        uint32_t all;
        dbase = block_exclusive_scan(totals[threadIdx.x], &all);
    }
    __syncthreads();

    const int64_t base = (int64_t)tile * kTile + (int64_t)wave * kWaveK;
    uint64_t key[KPT];
    int32_t val[KPT];
    uint32_t local[KPT];
    if (FIRST) {   // keys from the waits, payload the context size (payload_T) or the base index
        double x[KPT];
        int32_t t[KPT];
#pragma unroll
        for (int j = 0; j < KPT; ++j) {   // every load of the wave in flight before ranking
            const int64_t i = base + j * kWave + lane;
            x[j] = i < n ? w[i] : 0.0;
            t[j] = i < n ? T[i] : 1;
        }
        bool bad = false;
#pragma unroll
        for (int j = 0; j < KPT; ++j) {
            key[j] = wait_key(x[j], bad);
            if (t[j] < 1) {
                bad = true;
                t[j] = 1;
            }
            val[j] = payload_T ? t[j] : (int32_t)(base + j * kWave + lane);
        }
        if (bad) flag_domain(status);
    } else {
#pragma unroll
        for (int j = 0; j < KPT; ++j) {   // every load of the wave in flight before ranking
            const int64_t i = base + j * kWave + lane;
            key[j] = i < n ? keys_in[i] : 0;
            val[j] = i < n ? vals_in[i] : 0;
        }
    }
#pragma unroll
    for (int j = 0; j < KPT; ++j) {
        const bool valid = base + j * kWave + lane < n;
        const uint32_t d = (uint32_t)(key[j] >> shift) & 255u;
        const uint64_t peers = digit_peers(d, valid);
        const uint32_t rank = lanes_below(peers);
        const uint32_t before = wcnt[wave][d];
        local[j] = before + rank;
        __builtin_amdgcn_wave_barrier();
        if (valid && rank == 0) wcnt[wave][d] = (uint16_t)(before + (uint32_t)__popcll(peers));
        __builtin_amdgcn_wave_barrier();
    }
    __syncthreads();
    {
        const int d = threadIdx.x;
        uint32_t cnt[4], run = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            cnt[q] = wcnt[q][d];
            run += cnt[q];
        }
        uint32_t all;
        const uint32_t tstart = block_exclusive_scan(run, &all);   // run = this tile's count of digit d
        // wofs holds tile positions: digit d's run starts at tstart
        uint32_t at = tstart;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            wofs[q][d] = (uint16_t)at;
            at += cnt[q];
        }
        gbase[d] = (int32_t)((int64_t)dbase + my_off - tstart);
    }
    __syncthreads();
    // tile positions are dense: the valid keys of the tile fill [0, nvalid)
#pragma unroll
    for (int j = 0; j < KPT; ++j) {
        const int64_t i = base + j * kWave + lane;
        if (i < n) {
            const uint32_t d = (uint32_t)(key[j] >> shift) & 255u;
            const uint32_t pos = wofs[wave][d] + local[j];
            if (pos < (uint32_t)kTile) {           // always true; never write outside
                lkey[pos] = key[j];
                lval[pos] = val[j];
            }
        }
    }
    __syncthreads();
    const int64_t tile0 = (int64_t)tile * kTile;
    const int64_t left = n - tile0;
    const int nvalid = left < kTile ? (int)left : kTile;
#pragma unroll
    for (int q = 0; q < KPT; ++q) {
        const int pos = q * kSortThreads + (int)threadIdx.x;
        if (pos < nvalid) {
            const uint64_t k = lkey[pos];
            const int64_t dest = (int64_t)gbase[(k >> shift) & 255u] + pos;
            if (dest >= 0 && dest < n) {  // always true when the histograms agree
                keys_out[dest] = k;
                vals_out[dest] = lval[pos];
                if (dig_out != nullptr) dig_out[dest] = (uint8_t)(k >> (shift + 8));   // uniform
            }
        }
    }
}

// n <= kSortTile: the whole sorted path's sort (and, with Nsum, its prefix
// arrays) in one block, so a small sample costs two launches instead of
// thirty.  Keys and payload stay in LDS for the eight digit passes, ranked as
// in sort_scatter_kernel with the tile as the whole array (a stable counting
// sort per digit); then the sorted keys and payload are stored, and, with
// Nsum, the inclusive prefix arrays of T and T*w in a fixed order (each thread
// its kOneKPT consecutive positions, the thread totals across the block).
// Sixteen waves of two keys per lane: each wave's ranking is a chain of two
// dependent LDS updates per pass instead of eight, and the sixteen chains
// overlap (four waves of eight keys took 29 us for 1,000 keys on MI355X).
constexpr int kOneThreads = 1024;
constexpr int kOneKPT = kSortTile / kOneThreads;   // keys per thread
constexpr int kOneWaves = kOneThreads / kWave;
constexpr int kOneWaveKeys = kWave * kOneKPT;      // consecutive keys of one wave

__global__ void __launch_bounds__(kOneThreads) sort_small_kernel(
    const double *__restrict__ w, const int32_t *__restrict__ T, int64_t n,
    uint64_t *__restrict__ keys_out, int32_t *__restrict__ vals_out, int64_t *__restrict__ Nsum,
    double *__restrict__ Ssum, int32_t *__restrict__ perm_out, int *status)
{
    __shared__ uint64_t lk[2][kSortTile];
    __shared__ int32_t lv[2][kSortTile];
    // per-wave digit counts, then their wave prefixes; two sets, so that the
    // next pass's set is cleared while this pass uses the other
    __shared__ uint16_t wcnt[2][kOneWaves][256];
    __shared__ uint32_t lexcl[256];             // digit's start within its group of 64 digits
    __shared__ uint32_t dsum[256 / kWave];       // keys in each group of 64 digits
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const int nn = (int)n;   // at most kSortTile
    for (int i = threadIdx.x; i < nn; i += kOneThreads) {
        uint64_t b = (uint64_t)__double_as_longlong(w[i]);
        if (b == 0x8000000000000000ull) b = 0;  // -0.0 sorts as +0.0
        if (b >= 0x7ff0000000000000ull) {        // NaN, inf or negative
            flag_domain(status);
            b = 0;
        }
        if (T[i] < 1) flag_domain(status);
        lk[0][i] = b;
        lv[0][i] = i;
    }
    for (int q = threadIdx.x; q < kOneWaves * 256; q += kOneThreads) (&wcnt[0][0][0])[q] = 0;
    __syncthreads();
    int cur = 0;
    for (int pass = 0; pass < 8; ++pass) {
        const int shift = 8 * pass, wb = pass & 1;
        // the other set was last read before the previous pass's final barrier
        for (int q = threadIdx.x; q < kOneWaves * 256; q += kOneThreads) (&wcnt[wb ^ 1][0][0])[q] = 0;
        uint64_t key[kOneKPT];
        int32_t val[kOneKPT];
        uint32_t local[kOneKPT];
#pragma unroll
        for (int j = 0; j < kOneKPT; ++j) {
            const int i = wave * kOneWaveKeys + j * kWave + lane;
            const bool valid = i < nn;
            key[j] = valid ? lk[cur][i] : 0;
            val[j] = valid ? lv[cur][i] : 0;
            const uint32_t d = (uint32_t)(key[j] >> shift) & 255u;
            const uint64_t peers = digit_peers(d, valid);
            const uint32_t rank = lanes_below(peers);
            const uint32_t before = wcnt[wb][wave][d];
            local[j] = before + rank;
            __builtin_amdgcn_wave_barrier();
            if (valid && rank == 0) wcnt[wb][wave][d] = (uint16_t)(before + (uint32_t)__popcll(peers));
            __builtin_amdgcn_wave_barrier();
        }
        __syncthreads();
        // digit d (threads below 256): the waves' counts in wave order become
        // each wave's offset within the digit; the digit totals are scanned
        // within each group of 64 digits (one wave), the groups' totals kept
        if ((int)threadIdx.x < 256) {
            const int d = threadIdx.x;
            uint32_t c[kOneWaves], tot = 0;
#pragma unroll
            for (int q = 0; q < kOneWaves; ++q) c[q] = wcnt[wb][q][d];   // all loads in flight
#pragma unroll
            for (int q = 0; q < kOneWaves; ++q) {
                wcnt[wb][q][d] = (uint16_t)tot;
                tot += c[q];
            }
            const uint32_t incl = wave_incl_scan(tot);
            lexcl[d] = incl - tot;
            if (lane == kWave - 1) dsum[wave] = incl;
        }
        __syncthreads();
#pragma unroll
        for (int j = 0; j < kOneKPT; ++j) {
            const int i = wave * kOneWaveKeys + j * kWave + lane;
            if (i < nn) {
                const uint32_t d = (uint32_t)(key[j] >> shift) & 255u;
                uint32_t pos = lexcl[d] + wcnt[wb][wave][d] + local[j];
                for (uint32_t g = 0; g < d / kWave; ++g) pos += dsum[g];
                if (pos < (uint32_t)nn) {                 // always true; never write outside
                    lk[cur ^ 1][pos] = key[j];
                    lv[cur ^ 1][pos] = val[j];
                }
            }
        }
        __syncthreads();
        cur ^= 1;
    }
    for (int i = threadIdx.x; i < nn; i += kOneThreads) {
        keys_out[i] = lk[cur][i];
        vals_out[i] = lv[cur][i];
    }
    if (Nsum == nullptr) return;   // uniform: the sort alone
    const int k0 = (int)threadIdx.x * kOneKPT;
    int64_t tn[kOneKPT];
    double ts[kOneKPT];
    int64_t sn = 0;
    double ss = 0.0;
#pragma unroll
    for (int q = 0; q < kOneKPT; ++q) {
        const int k = k0 + q;
        if (k < nn) {
            const int32_t pj = lv[cur][k];
            const int32_t p = (pj >= 0 && pj < nn) ? pj : 0;   // a permutation of [0, n)
            const int32_t t = T[p] < 1 ? 1 : T[p];
            sn += t;
            ss += (double)t * __longlong_as_double((long long)lk[cur][k]);
            if (perm_out != nullptr) perm_out[k] = p;
        }
        tn[q] = sn;
        ts[q] = ss;
    }
    // scan of the thread totals in the wave: inclusive, then exclusive
    const int64_t xn = wave_incl_scan(sn), en = wave_lane_back(xn);
    const double xs = wave_incl_scan(ss), es = wave_lane_back(xs);
    __shared__ int64_t wn[kOneWaves];
    __shared__ double wsm[kOneWaves];
    if (lane == kWave - 1) {
        wn[wave] = xn;
        wsm[wave] = xs;
    }
    __syncthreads();
    int64_t pn = 0;
    double ps = 0.0;
    for (int q = 0; q < wave; ++q) {
        pn += wn[q];
        ps += wsm[q];
    }
    pn += en;
    ps += es;
#pragma unroll
    for (int q = 0; q < kOneKPT; ++q) {
        const int k = k0 + q;
        if (k < nn) {
            Nsum[k] = pn + tn[q];
            Ssum[k] = ps + ts[q];
        }
    }
}

// Per scan tile: sums of T and T*w over the sorted order.  GATHER: the sort's
// payload is the base index (perm) and the context sizes are gathered through
// it once, into Tsorted; otherwise the payload already is the context size in
// sorted order (Tsorted) and is only read.  CHUNKS: the sums of every run of 64
// sorted positions are also written (chunkN, chunkS; run c of tile b is
// c = 32 b + 4 q + wave, the positions of row q that a wave holds), so that N
// and S at a few query positions can be formed without the full prefix arrays.
template <bool GATHER, bool CHUNKS>
__global__ void __launch_bounds__(kScanThreads) scan_reduce_kernel(
    const uint64_t *__restrict__ skeys, const int32_t *__restrict__ perm,
    const int32_t *__restrict__ T, int64_t n, int64_t *__restrict__ blkN,
    double *__restrict__ blkS, int32_t *__restrict__ Tsorted, int64_t *__restrict__ chunkN,
    double *__restrict__ chunkS)
{
    // striped over the tile (element q*256 + t of it), so that every load and
    // store of a wave covers consecutive positions; the tile's total is summed
    // in this fixed order
    const int64_t base = (int64_t)blockIdx.x * kScanTile + threadIdx.x;
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    int64_t sn = 0;
    double ss = 0.0;
#pragma unroll
    for (int q = 0; q < kScanIPT; ++q) {
        const int64_t j = base + (int64_t)q * kScanThreads;
        int64_t en = 0;
        double es = 0.0;
        if (j < n) {
            int32_t t;
            if (GATHER) {
                const int32_t pj = perm[j];
                const int32_t pi = (pj >= 0 && pj < n) ? pj : 0;  // perm is a permutation of [0, n)
                t = T[pi] < 1 ? 1 : T[pi];
                Tsorted[j] = t;   // the gather is done once; the final pass streams it
            } else {
                t = Tsorted[j];   // clamped to >= 1 when the keys were prepared
            }
            en = t;
            es = (double)t * __longlong_as_double((long long)skeys[j]);
        }
        if (CHUNKS) {   // this wave's 64 positions of row q (their sum in lane 63), then into the wave's total
            en = wave_incl_scan(en);
            es = wave_incl_scan(es);
            const int64_t c = ((int64_t)blockIdx.x * kScanIPT + q) * (kScanThreads / kWave) + wave;
            if (lane == kWave - 1 && c * kWave < n) {
                chunkN[c] = en;
                chunkS[c] = es;
            }
        }
        sn += en;
        ss += es;
    }
    // fixed-order tree: wave_incl_scan's within each wave (done per chunk
    // with CHUNKS), the total in lane 63, then the four waves in order
    if (!CHUNKS) {
        sn = wave_incl_scan(sn);
        ss = wave_incl_scan(ss);
    }
    __shared__ int64_t rn[kScanThreads / kWave];
    __shared__ double rs[kScanThreads / kWave];
    if (lane == kWave - 1) {
        rn[wave] = sn;
        rs[wave] = ss;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        int64_t a = 0;
        double b = 0.0;
        for (int q = 0; q < kScanThreads / kWave; ++q) {
            a += rn[q];
            b += rs[q];
        }
        blkN[blockIdx.x] = a;
        blkS[blockIdx.x] = b;
    }
}

// Exclusive scan of the tile sums in place, one block of 1,024 threads, each
// thread a run of consecutive tiles added in order, then the run totals across
// the block in a fixed order (reproducible).
__global__ void __launch_bounds__(1024) scan_blocks_kernel(int64_t *blkN, double *blkS, int nb)
{
    const int per = (nb + 1023) / 1024;
    const int64_t t0 = (int64_t)threadIdx.x * per;
    int64_t t1 = t0 + per;
    if (t1 > nb) t1 = nb;
    int64_t alln;
    double alls;
    if (per <= kRunRegs) {   // uniform
        int64_t cn[kRunRegs];
        double cs[kRunRegs];
        int64_t sn = 0;
        double ss = 0.0;
#pragma unroll
        for (int i = 0; i < kRunRegs; ++i) {
            const bool in = t0 + i < t1;
            cn[i] = in ? blkN[t0 + i] : 0;
            cs[i] = in ? blkS[t0 + i] : 0.0;
            sn += cn[i];
            ss += cs[i];
        }
        int64_t pn = block1024_exclusive_scan(sn, &alln);
        double ps = block1024_exclusive_scan(ss, &alls);
#pragma unroll
        for (int i = 0; i < kRunRegs; ++i) {
            if (t0 + i < t1) {
                blkN[t0 + i] = pn;
                blkS[t0 + i] = ps;
            }
            pn += cn[i];
            ps += cs[i];
        }
        return;
    }
    int64_t sn = 0;
    double ss = 0.0;
    for (int64_t t = t0; t < t1; ++t) {
        sn += blkN[t];
        ss += blkS[t];
    }
    int64_t pn = block1024_exclusive_scan(sn, &alln);
    double ps = block1024_exclusive_scan(ss, &alls);
    for (int64_t t = t0; t < t1; ++t) {
        const int64_t cn = blkN[t];
        const double cs = blkS[t];
        blkN[t] = pn;
        blkS[t] = ps;
        pn += cn;
        ps += cs;
    }
}

// Inclusive prefix within each tile plus the tile's offset, over the context
// sizes in sorted order that scan_reduce_kernel gathered; also emits perm.
__global__ void __launch_bounds__(kScanThreads) scan_final_kernel(
    const uint64_t *__restrict__ skeys, const int32_t *__restrict__ perm,
    const int32_t *__restrict__ Tsorted, int64_t n, const int64_t *__restrict__ blkN,
    const double *__restrict__ blkS, int64_t *__restrict__ Nsum, double *__restrict__ Ssum,
    int32_t *__restrict__ perm_out)
{
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanIPT;
    int64_t tn[kScanIPT];
    double ts[kScanIPT];
    int64_t sn = 0;
    double ss = 0.0;
    // a thread's kScanIPT positions are adjacent and start on a multiple of 8
    // elements, so a full run is read with 16-byte loads (the workspace
    // arrays are 256-byte aligned)
    const bool full = base + kScanIPT <= n;
    int32_t tv[kScanIPT];
    uint64_t kv[kScanIPT];
    if (full) {
        static_assert(kScanIPT == 8, "vector loads below assume 8 positions per thread");
        const int4 *tp = reinterpret_cast<const int4 *>(Tsorted + base);
        const ulonglong2 *kp = reinterpret_cast<const ulonglong2 *>(skeys + base);
        const int4 t0 = tp[0], t1 = tp[1];
        const ulonglong2 k0 = kp[0], k1 = kp[1], k2 = kp[2], k3 = kp[3];
        tv[0] = t0.x; tv[1] = t0.y; tv[2] = t0.z; tv[3] = t0.w;
        tv[4] = t1.x; tv[5] = t1.y; tv[6] = t1.z; tv[7] = t1.w;
        kv[0] = k0.x; kv[1] = k0.y; kv[2] = k1.x; kv[3] = k1.y;
        kv[4] = k2.x; kv[5] = k2.y; kv[6] = k3.x; kv[7] = k3.y;
    } else {
#pragma unroll
        for (int q = 0; q < kScanIPT; ++q) {
            const int64_t j = base + q;
            tv[q] = (j < n) ? Tsorted[j] : 0;
            kv[q] = (j < n) ? skeys[j] : 0;
        }
    }
#pragma unroll
    for (int q = 0; q < kScanIPT; ++q) {
        const int64_t j = base + q;
        if (j < n) {
            sn += tv[q];
            ss += (double)tv[q] * __longlong_as_double((long long)kv[q]);
            if (perm_out != nullptr) {
                const int32_t pj = perm[j];
                perm_out[j] = (pj >= 0 && pj < n) ? pj : 0;  // perm is a permutation of [0, n)
            }
        }
        tn[q] = sn;
        ts[q] = ss;
    }
    // exclusive scan of the per-thread totals across the block
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const int64_t xn = wave_incl_scan(sn), en = wave_lane_back(xn);
    const double xs = wave_incl_scan(ss), es = wave_lane_back(xs);
    __shared__ int64_t wn[4];
    __shared__ double wsm[4];
    if (lane == kWave - 1) {
        wn[wave] = xn;
        wsm[wave] = xs;
    }
    __syncthreads();
    int64_t pn = blkN[blockIdx.x];
    double ps = blkS[blockIdx.x];
    for (int q = 0; q < wave; ++q) {
        pn += wn[q];
        ps += wsm[q];
    }
    pn += en;
    ps += es;
    if (full) {
        longlong2 *np = reinterpret_cast<longlong2 *>(Nsum + base);
        double2 *sp = reinterpret_cast<double2 *>(Ssum + base);
#pragma unroll
        for (int h = 0; h < kScanIPT / 2; ++h) {
            np[h] = make_longlong2(pn + tn[2 * h], pn + tn[2 * h + 1]);
            sp[h] = make_double2(ps + ts[2 * h], ps + ts[2 * h + 1]);
        }
    } else {
#pragma unroll
        for (int q = 0; q < kScanIPT; ++q) {
            const int64_t j = base + q;
            if (j < n) {
                Nsum[j] = pn + tn[q];
                Ssum[j] = ps + ts[q];
            }
        }
    }
}

// Number of sorted waits <= x.
__device__ __forceinline__ int64_t upper_bound_keys(const uint64_t *__restrict__ skeys, int64_t n,
                                                    double x)
{
    int64_t lo = 0, hi = n;
    while (lo < hi) {
        const int64_t mid = lo + (hi - lo) / 2;
        if (__longlong_as_double((long long)skeys[mid]) <= x) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

// Number of sorted waits <= x found by one wave in steps of a 64-ary search:
// the lanes compare 64 evenly spaced keys of the open range [lo, hi) (keys
// before lo are <= x, keys from hi on are > x; sorted keys make the lanes
// with key <= x a prefix), which shrinks 65-fold per step; the last <= 64
// keys are compared directly.  Every lane returns the count.
__device__ __forceinline__ int64_t wave_upper_bound(const uint64_t *__restrict__ skeys, int64_t n,
                                                    double x)
{
    const int lane = threadIdx.x % kWave;
    int64_t lo = 0, hi = n;
    while (hi - lo > kWave) {
        const int64_t len = hi - lo;
        const int64_t pos = lo + ((int64_t)(lane + 1) * len) / (kWave + 1);   // strictly increasing
        const bool le = __longlong_as_double((long long)skeys[pos]) <= x;
        const int k = __popcll(__ballot(le));
        const int64_t below = __shfl(pos, k > 0 ? k - 1 : 0, kWave);
        const int64_t above = __shfl(pos, k < kWave ? k : kWave - 1, kWave);
        if (k > 0) lo = below + 1;
        if (k < kWave) hi = above;
    }
    const int64_t pos = lo + lane;
    const bool le = pos < hi && __longlong_as_double((long long)skeys[pos]) <= x;
    return lo + __popcll(__ballot(le));
}

// The closed form of policy f for every load, from its two positions (counts of
// sorted waits <= t1 and <= e); loads l0, l0 + lstep, ... are written.
__device__ __forceinline__ void closed_form_values(int64_t tot, int64_t n1, int64_t ne, double s1,
                                                   double se, int64_t n, const Tables &tb,
                                                   const PriceDev &pr, int64_t f, double t1,
                                                   double e, int l0, int lstep,
                                                   double *__restrict__ cost)
{
    const int64_t P = (int64_t)tb.K1 * tb.K2;
    const double hbm = s1 + t1 * (double)(tot - n1);
    double hold = (se - s1) - t1 * (double)(ne - n1);
    if (!isinf(e)) hold += (e - t1) * (double)(tot - ne);
    const double fixed = pr.a1 * hbm + pr.b2 * (double)(ne - n1) + pr.b3 * (double)(tot - ne);
    const double nd = (double)n;
    for (int l = l0; l < tb.L; l += lstep) cost[(int64_t)l * P + f] = (fixed + tb.a2[l] * hold) / nd;
}

// The same from the inclusive prefix arrays.
__device__ __forceinline__ void closed_form_policy(const int64_t *__restrict__ Nsum,
                                                   const double *__restrict__ Ssum, int64_t n,
                                                   const Tables &tb, const PriceDev &pr, int64_t f,
                                                   double t1, double e, int64_t p1, int64_t pe,
                                                   int l0, int lstep, double *__restrict__ cost)
{
    const int64_t tot = Nsum[n - 1];
    const int64_t n1 = p1 ? Nsum[p1 - 1] : 0, ne = pe ? Nsum[pe - 1] : 0;
    const double s1 = p1 ? Ssum[p1 - 1] : 0.0, se = pe ? Ssum[pe - 1] : 0.0;
    closed_form_values(tot, n1, ne, s1, se, n, tb, pr, f, t1, e, l0, lstep, cost);
}

// N and S over the sorted positions [0, p), by one wave: the tile's exclusive
// prefix, the 64-position chunk sums of the tile before p and the positions of
// p's own chunk, each group added across the lanes in wave_total's fixed tree;
// every lane returns the same values, and equal p give equal values.
__device__ __forceinline__ void wave_prefix_at(int64_t p, int nb, const int64_t *__restrict__ blkN,
                                               const double *__restrict__ blkS,
                                               const int64_t *__restrict__ chunkN,
                                               const double *__restrict__ chunkS,
                                               const uint64_t *__restrict__ skeys,
                                               const int32_t *__restrict__ Tsorted, int64_t &N,
                                               double &S)
{
    const int lane = threadIdx.x % kWave;
    int64_t tile = p / kScanTile;
    if (tile > nb - 1) tile = nb - 1;
    const int64_t off = p - tile * kScanTile;     // 0 .. kScanTile
    const int nc = (int)(off / kWave), rem = (int)(off % kWave);
    int64_t cn = 0, en = 0;
    double cs = 0.0, es = 0.0;
    if (lane < nc) {
        const int64_t c = tile * (kScanTile / kWave) + lane;
        cn = chunkN[c];
        cs = chunkS[c];
    }
    if (lane < rem) {
        const int64_t j = tile * kScanTile + (int64_t)nc * kWave + lane;
        const int32_t t = Tsorted[j];
        en = t;
        es = (double)t * __longlong_as_double((long long)skeys[j]);
    }
    cn = wave_total(cn);
    cs = wave_total(cs);
    en = wave_total(en);
    es = wave_total(es);
    N = blkN[tile] + cn + en;
    S = (blkS[tile] + cs) + es;
}

// One thread per policy (a, k): closed form for every load (many policies).
__global__ void __launch_bounds__(256) closed_form_kernel(const uint64_t *__restrict__ skeys,
                                                          const int64_t *__restrict__ Nsum,
                                                          const double *__restrict__ Ssum, int64_t n,
                                                          Tables tb, PriceDev pr,
                                                          double *__restrict__ cost)
{
    const int64_t P = (int64_t)tb.K1 * tb.K2;
    const int64_t f = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (f >= P) return;
    const int a = (int)(f / tb.K2), k = (int)(f % tb.K2);
    const double t1 = tb.t1[a];
    const double e = t1 + tb.t2[k];
    closed_form_policy(Nsum, Ssum, n, tb, pr, f, t1, e, upper_bound_keys(skeys, n, t1),
                       upper_bound_keys(skeys, n, e), 0, 1, cost);
}

// One wave per policy (few policies): the two positions by 64-ary searches,
// whose few dependent steps replace a binary search's ~log2(n), then the
// lanes share the loads.
__global__ void __launch_bounds__(256) closed_form_wave_kernel(const uint64_t *__restrict__ skeys,
                                                               const int64_t *__restrict__ Nsum,
                                                               const double *__restrict__ Ssum,
                                                               int64_t n, Tables tb, PriceDev pr,
                                                               double *__restrict__ cost)
{
    const int64_t P = (int64_t)tb.K1 * tb.K2;
    const int64_t f = (int64_t)blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave;
    if (f >= P) return;   // uniform per wave
    const int a = (int)(f / tb.K2), k = (int)(f % tb.K2);
    const double t1 = tb.t1[a];
    const double e = t1 + tb.t2[k];
    const int64_t p1 = wave_upper_bound(skeys, n, t1);
    const int64_t pe = wave_upper_bound(skeys, n, e);
    closed_form_policy(Nsum, Ssum, n, tb, pr, f, t1, e, p1, pe, (int)(threadIdx.x % kWave), kWave,
                       cost);
}

// One wave per policy, N and S at the query positions only (no prefix arrays):
// the two positions by 64-ary searches, then wave_prefix_at for t1, the
// deadline and the whole sample.
__global__ void __launch_bounds__(256) closed_form_query_kernel(
    const uint64_t *__restrict__ skeys, const int32_t *__restrict__ Tsorted, int64_t n, int nb,
    const int64_t *__restrict__ blkN, const double *__restrict__ blkS,
    const int64_t *__restrict__ chunkN, const double *__restrict__ chunkS, Tables tb, PriceDev pr,
    double *__restrict__ cost)
{
    const int64_t P = (int64_t)tb.K1 * tb.K2;
    const int64_t f = (int64_t)blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave;
    if (f >= P) return;   // uniform per wave
    const int a = (int)(f / tb.K2), k = (int)(f % tb.K2);
    const double t1 = tb.t1[a];
    const double e = t1 + tb.t2[k];
    const int64_t p1 = wave_upper_bound(skeys, n, t1);
    const int64_t pe = wave_upper_bound(skeys, n, e);
    int64_t tot, n1, ne;
    double sall, s1, se;
    wave_prefix_at(n, nb, blkN, blkS, chunkN, chunkS, skeys, Tsorted, tot, sall);
    wave_prefix_at(p1, nb, blkN, blkS, chunkN, chunkS, skeys, Tsorted, n1, s1);
    wave_prefix_at(pe, nb, blkN, blkS, chunkN, chunkS, skeys, Tsorted, ne, se);
    closed_form_values(tot, n1, ne, s1, se, n, tb, pr, f, t1, e, (int)(threadIdx.x % kWave), kWave,
                       cost);
}

// Policies up to which a wave per policy pays (its searches are short chains
// of dependent loads; many policies already fill the chip with one thread each).
constexpr int64_t kWavePolicies = 16384;

static hipError_t launch_closed_form(const uint64_t *skeys, const SortWs &ws, int64_t n,
                                     const Tables &tb, const PriceDev &pr, double *cost_out,
                                     hipStream_t stream)
{
    const int64_t P = (int64_t)tb.K1 * tb.K2;
    if (P <= kWavePolicies)
        hipLaunchKernelGGL(closed_form_wave_kernel, dim3((unsigned)cdiv(P, 256 / kWave)), dim3(256),
                           0, stream, skeys, ws.Nsum, ws.Ssum, n, tb, pr, cost_out);
    else
        hipLaunchKernelGGL(closed_form_kernel, dim3((unsigned)cdiv(P, 256)), dim3(256), 0, stream,
                           skeys, ws.Nsum, ws.Ssum, n, tb, pr, cost_out);
    return hipGetLastError();
}

// Unused dynamic LDS that holds the 4,096-key scatter at two blocks per CU
// from 2^24 keys: three blocks per CU (52 KiB each) measured faster at 2^23
// (0.585 against 0.634 ms per call on MI355X) but slower at 2^24 (1.287
// against 1.256 ms, the same box).
constexpr int64_t kDigitBytesFrom = int64_t(1) << 22;

static size_t scatter_lds_pad(int kpt, int64_t n)
{
    return (kpt == 16 && n >= (int64_t(1) << 24)) ? 4096 : 0;
}

template <int KPT>
static hipError_t launch_digit_passes(const double *w, const int32_t *T, int64_t n, SortWs &ws,
                                      int payload_T, int *status, hipStream_t stream)
{
    // From 2^22 keys each scatter also writes the next pass's digit bytes, to
    // the prefix-sum buffer (unused until the sort is done; 8 n bytes hold the
    // bytes of whole tiles, n > kSortTile), and the histograms read those.
    // Measured on MI355X: at 2^24 a pass's histogram 31.8 -> 13.0 us, its
    // scatter 99.3 -> 107.7 us, the call 1.227 -> 1.160 ms; at 2^20 the
    // scatter's extra stores cost more than the histogram saves (12.8 -> 15.3
    // against 4.9 -> 4.2 us).
    uint8_t *const dig = n >= kDigitBytesFrom ? reinterpret_cast<uint8_t *>(ws.Nsum) : nullptr;
    if ((int64_t)ws.nblocks * kSortThreads * KPT > 8 * n) return hipErrorInvalidValue;
    const size_t pad = scatter_lds_pad(KPT, n);
    hipError_t err = hipSuccess;
    // pass p reads buffer (p & 1) and writes the other; the first reads the
    // waits and context sizes and writes buffer 1, so the eighth writes buffer 0
    for (int pass = 0; pass < 8 && err == hipSuccess; ++pass) {
        const int shift = 8 * pass, in = pass & 1, out = in ^ 1;
        if (pass == 0)
            hipLaunchKernelGGL(sort_first_hist_kernel<KPT>, dim3(ws.nblocks), dim3(kSortThreads),
                               0, stream, w, n, ws.hist, ws.nblocks, status);
        else if (dig != nullptr)
            hipLaunchKernelGGL(sort_hist_bytes_kernel<KPT>, dim3(ws.nblocks), dim3(kSortThreads),
                               0, stream, dig, n, ws.hist, ws.nblocks);
        else
            hipLaunchKernelGGL(sort_hist_kernel<KPT>, dim3(ws.nblocks), dim3(kSortThreads), 0,
                               stream, ws.keys[in], n, shift, ws.hist, ws.nblocks);
        hipLaunchKernelGGL(digit_scan_kernel, dim3(256), dim3(1024), 0, stream, ws.hist,
                           ws.nblocks, ws.counts);
        uint8_t *const dnext = pass < 7 ? dig : nullptr;
        if (pass == 0)
            hipLaunchKernelGGL((sort_scatter_kernel<KPT, true>), dim3(ws.nblocks),
                               dim3(kSortThreads), pad, stream, nullptr, nullptr, w, T, payload_T,
                               n, shift, ws.hist, ws.counts, ws.nblocks, ws.keys[out],
                               ws.vals[out], dnext, status);
        else
            hipLaunchKernelGGL((sort_scatter_kernel<KPT, false>), dim3(ws.nblocks),
                               dim3(kSortThreads), pad, stream, ws.keys[in], ws.vals[in], nullptr,
                               nullptr, 0, n, shift, ws.hist, ws.counts, ws.nblocks, ws.keys[out],
                               ws.vals[out], dnext, status);
        err = hipGetLastError();
    }
    return err;
}

// Eight passes leave the result in buffer 0.
static hipError_t launch_sort(const double *w, const int32_t *T, int64_t n, SortWs &ws,
                              int payload_T, int *status, hipStream_t stream)
{
    switch (ws.kpt) {
    case 16: return launch_digit_passes<16>(w, T, n, ws, payload_T, status, stream);
    case 8: return launch_digit_passes<8>(w, T, n, ws, payload_T, status, stream);
    case 4: return launch_digit_passes<4>(w, T, n, ws, payload_T, status, stream);
    default: return launch_digit_passes<2>(w, T, n, ws, payload_T, status, stream);
    }
}

hipError_t launch_sort_keys(const double *w, const int32_t *T, int64_t n, SortWs &ws, int *cur_out,
                            int *status, hipStream_t stream)
{
    *cur_out = 0;
    if (n <= kSortTile) {   // one block
        hipLaunchKernelGGL(sort_small_kernel, dim3(1), dim3(kOneThreads), 0, stream, w, T, n,
                           ws.keys[0], ws.vals[0], nullptr, nullptr, nullptr, status);
        return hipGetLastError();
    }
    return launch_sort(w, T, n, ws, 0, status, stream);
}

hipError_t launch_sorted_path(const double *w, const int32_t *T, int64_t n, const Tables &tb,
                              const PriceDev &pr, SortWs &ws, double *cost_out,
                              int32_t *perm_out, int *status, hipStream_t stream)
{
    if (n <= kSortTile) {   // sort and prefix arrays in one block
        hipLaunchKernelGGL(sort_small_kernel, dim3(1), dim3(kOneThreads), 0, stream, w, T, n,
                           ws.keys[0], ws.vals[0], ws.Nsum, ws.Ssum, perm_out, status);
        const hipError_t err = hipGetLastError();
        if (err != hipSuccess) return err;
        return launch_closed_form(ws.keys[0], ws, n, tb, pr, cost_out, stream);
    }
    // without a requested order the payload is the context size itself, so the
    // scans read it in sorted order instead of gathering it through the order
    const bool want_perm = perm_out != nullptr;
    hipError_t err = launch_sort(w, T, n, ws, want_perm ? 0 : 1, status, stream);
    if (err != hipSuccess) return err;
    int32_t *Tsorted = want_perm ? ws.vals[1] : ws.vals[0];   // buffer 1 is free after the sort
    const int64_t P = (int64_t)tb.K1 * tb.K2;
    if (!want_perm && P <= kWavePolicies) {
        // N and S are needed at 2 P + 1 positions only: the tile sums, the
        // 64-position chunk sums (in the prefix arrays' space) and the tiles'
        // prefixes, then one wave per policy; no prefix arrays are written
        hipLaunchKernelGGL((scan_reduce_kernel<false, true>), dim3(ws.nblocks_scan),
                           dim3(kScanThreads), 0, stream, ws.keys[0], nullptr, T, n, ws.blkN,
                           ws.blkS, Tsorted, ws.Nsum, ws.Ssum);
        hipLaunchKernelGGL(scan_blocks_kernel, dim3(1), dim3(1024), 0, stream, ws.blkN, ws.blkS,
                           ws.nblocks_scan);
        hipLaunchKernelGGL(closed_form_query_kernel, dim3((unsigned)cdiv(P, 256 / kWave)),
                           dim3(256), 0, stream, ws.keys[0], Tsorted, n, ws.nblocks_scan, ws.blkN,
                           ws.blkS, ws.Nsum, ws.Ssum, tb, pr, cost_out);
        return hipGetLastError();
    }
    if (want_perm)
        hipLaunchKernelGGL((scan_reduce_kernel<true, false>), dim3(ws.nblocks_scan),
                           dim3(kScanThreads), 0, stream, ws.keys[0], ws.vals[0], T, n, ws.blkN,
                           ws.blkS, Tsorted, nullptr, nullptr);
    else
        hipLaunchKernelGGL((scan_reduce_kernel<false, false>), dim3(ws.nblocks_scan),
                           dim3(kScanThreads), 0, stream, ws.keys[0], nullptr, T, n, ws.blkN,
                           ws.blkS, Tsorted, nullptr, nullptr);
    hipLaunchKernelGGL(scan_blocks_kernel, dim3(1), dim3(1024), 0, stream, ws.blkN, ws.blkS,
                       ws.nblocks_scan);
    hipLaunchKernelGGL(scan_final_kernel, dim3(ws.nblocks_scan), dim3(kScanThreads), 0, stream,
                       ws.keys[0], ws.vals[0], Tsorted, n, ws.blkN, ws.blkS, ws.Nsum, ws.Ssum,
                       perm_out);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    return launch_closed_form(ws.keys[0], ws, n, tb, pr, cost_out, stream);
}

}  // namespace kvr
