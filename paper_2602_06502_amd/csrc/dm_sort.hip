// Stable LSD radix sort of (u64 key, u32 value) pairs, 8-bit digits.
// Per pass: tile digit histograms (digit-major), one exclusive scan over
// them, and a stable scatter.  A tile is 1024 or 2048 items; the scatter ranks
// equal digits inside each wave with ballots, orders the tile by digit in
// LDS, and writes each digit's items as one run of consecutive addresses.
#include "dm_internal.h"

namespace dm {
namespace {

constexpr int kSortThreads = 256;
constexpr int kSortWaves = kSortThreads / kWave;
// Items per thread: 8 (2048-item tiles, longer runs per digit) for large
// sorts, 4 (1024-item tiles, twice the workgroups) below kBigSort.
constexpr uint64_t kBigSort = 1ull << 22;
constexpr uint64_t tile_of(uint64_t n) { return n >= kBigSort ? 8 * kSortThreads : 4 * kSortThreads; }
constexpr int kSortSlot = kSlotSort;

template <int kSortItems>
__global__ __launch_bounds__(kSortThreads) void digit_hist_kernel(const uint64_t* __restrict__ keys,
                                                                  uint64_t n, int shift,
                                                                  uint64_t ntiles,
                                                                  uint64_t* __restrict__ cnt)
{
    constexpr uint64_t kSortTile = (uint64_t)kSortThreads * kSortItems;
    __shared__ uint32_t hist[256];
    hist[threadIdx.x] = 0;
    __syncthreads();
    const uint64_t base = blockIdx.x * kSortTile;
#pragma unroll
    for (int it = 0; it < kSortItems; it++) {
        const uint64_t i = base + it * kSortThreads + threadIdx.x;
        if (i < n)
            atomicAdd(&hist[(keys[i] >> shift) & 0xFF], 1u);
    }
    __syncthreads();
    cnt[(uint64_t)threadIdx.x * ntiles + blockIdx.x] = hist[threadIdx.x];
}

template <int kSortItems>
__global__ __launch_bounds__(kSortThreads) void digit_scatter_kernel(
    const uint64_t* __restrict__ keys, const uint32_t* __restrict__ vals, uint64_t n, int shift,
    uint64_t ntiles, const uint64_t* __restrict__ offs, uint64_t* __restrict__ okeys,
    uint32_t* __restrict__ ovals)
{
    constexpr uint64_t kSortTile = (uint64_t)kSortThreads * kSortItems;
    __shared__ uint64_t sk[kSortTile];
    __shared__ uint32_t sv[kSortTile];
    // per round (double-buffered): each wave's count of each digit, tagged
    // with the round (count | round << 16), then replaced by its offset
    __shared__ uint32_t wcnt[2][kSortWaves][256];
    __shared__ uint32_t run[256];    // items of each digit in earlier rounds
    __shared__ uint32_t dbase[256];  // the digit's first place in the tile's order
    __shared__ int64_t gshift[256];  // global place of the digit's first item - dbase
    __shared__ uint32_t wsum[kSortWaves];
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    const uint64_t lt = lane ? (~0ull >> (64 - lane)) : 0ull;
    const uint64_t base = blockIdx.x * kSortTile;
    const uint64_t tn = n - base < kSortTile ? n - base : kSortTile;
    run[t] = 0;
    // no round's tag: entries a round does not write read as zero counts
    for (int q = t; q < 2 * kSortWaves * 256; q += kSortThreads)
        (&wcnt[0][0][0])[q] = 0xFFFFFFFFu;
    uint64_t k[kSortItems];
    uint32_t v[kSortItems], rk[kSortItems];
    __syncthreads();
#pragma unroll
    for (int it = 0; it < kSortItems; it++) {
        const uint64_t i = (uint64_t)it * kSortThreads + t;  // place in the tile
        const bool ok = i < tn;
        k[it] = ok ? keys[base + i] : 0;
        v[it] = ok && vals ? vals[base + i] : 0;
        const uint32_t d = (uint32_t)((k[it] >> shift) & 0xFF);
        uint64_t peers = ballot(ok);
#pragma unroll
        for (int b = 0; b < 8; b++) {
            const bool bit = (d >> b) & 1;
            const uint64_t m = ballot(bit);
            peers &= bit ? m : ~m;
        }
        const uint32_t pr = __popcll(peers & lt);
        const int buf = it & 1;
        if (ok && pr == 0)
            wcnt[buf][w][d] = (uint32_t)__popcll(peers) | ((uint32_t)it << 16);
        __syncthreads();
        // thread t = digit t: offsets of the waves' items of this round
        {
            uint32_t r = run[t];
#pragma unroll
            for (int ww = 0; ww < kSortWaves; ww++) {
                const uint32_t x = wcnt[buf][ww][t];
                const uint32_t c = (x >> 16) == (uint32_t)it ? (x & 0xFFFFu) : 0u;
                wcnt[buf][ww][t] = r | ((uint32_t)it << 16);
                r += c;
            }
            run[t] = r;
        }
        __syncthreads();
        rk[it] = ok ? (wcnt[buf][w][d] & 0xFFFFu) + pr : 0;
    }
    // (offsets fit the 16 bits below the tag: a tile has at most 2048 items)
    // first place of each digit in the tile (exclusive scan over digits)
    {
        uint32_t x = run[t];
        // inclusive wave scan
#pragma unroll
        for (int dlt = 1; dlt < kWave; dlt <<= 1) {
            const uint32_t y = __shfl_up(x, dlt);
            if (lane >= dlt)
                x += y;
        }
        if (lane == kWave - 1)
            wsum[w] = x;
        __syncthreads();
        uint32_t add = 0;
        for (int ww = 0; ww < w; ww++)
            add += wsum[ww];
        dbase[t] = x + add - run[t];
        gshift[t] = (int64_t)offs[(uint64_t)t * ntiles + blockIdx.x] - (int64_t)(x + add - run[t]);
    }
    __syncthreads();
#pragma unroll
    for (int it = 0; it < kSortItems; it++) {
        const uint64_t i = (uint64_t)it * kSortThreads + t;
        if (i < tn) {
            const uint32_t d = (uint32_t)((k[it] >> shift) & 0xFF);
            const uint32_t at = dbase[d] + rk[it];
            sk[at] = k[it];
            if (vals)
                sv[at] = v[it];
        }
    }
    __syncthreads();
    // the tile in digit order: consecutive places of one digit go to
    // consecutive addresses
    for (uint32_t j = t; j < tn; j += kSortThreads) {
        const uint64_t x = sk[j];
        const uint32_t d = (uint32_t)((x >> shift) & 0xFF);
        const uint64_t pos = (uint64_t)(gshift[d] + (int64_t)j);
        okeys[pos] = x;
        if (ovals)
            ovals[pos] = sv[j];
    }
}

}  // namespace

uint64_t sort_scan_len(uint64_t n) { return 256 * ((n + tile_of(n) - 1) / tile_of(n)); }

// digit counts and their offsets, 256 per tile each
uint64_t sort_scratch_bytes(uint64_t n) { return 2 * sort_scan_len(n) * sizeof(uint64_t); }

hipError_t radix_sort_kv(dm_ctx* c, uint64_t* keys, uint32_t* vals, uint64_t* ktmp,
                         uint32_t* vtmp, uint64_t n, int bits)
{
    if (n < 2 || bits <= 0)
        return hipSuccess;
    const uint64_t tile = tile_of(n), ntiles = (n + tile - 1) / tile;
    hipError_t e;
    uint64_t* cnt = static_cast<uint64_t*>(scratch_get(c, kSortSlot, sort_scratch_bytes(n), &e));
    if (!cnt)
        return e;
    uint64_t* offs = cnt + 256 * ntiles;
    uint64_t *sk = keys, *dk = ktmp;
    uint32_t *sv = vals, *dv = vtmp;
    int passes = 0;
    for (int shift = 0; shift < bits; shift += 8, passes++) {
        if (n >= kBigSort)
            digit_hist_kernel<8><<<ntiles, kSortThreads, 0, c->stream>>>(sk, n, shift, ntiles, cnt);
        else
            digit_hist_kernel<4><<<ntiles, kSortThreads, 0, c->stream>>>(sk, n, shift, ntiles, cnt);
        e = exclusive_scan_u64(c, cnt, 256 * ntiles, offs, nullptr);
        if (e != hipSuccess)
            return e;
        if (n >= kBigSort)
            digit_scatter_kernel<8><<<ntiles, kSortThreads, 0, c->stream>>>(sk, sv, n, shift,
                                                                             ntiles, offs, dk, dv);
        else
            digit_scatter_kernel<4><<<ntiles, kSortThreads, 0, c->stream>>>(sk, sv, n, shift,
                                                                            ntiles, offs, dk, dv);
        std::swap(sk, dk);
        std::swap(sv, dv);
    }
    if (passes & 1) {
        e = hipMemcpyAsync(keys, sk, n * sizeof(uint64_t), hipMemcpyDeviceToDevice, c->stream);
        if (e == hipSuccess && vals)
            e = hipMemcpyAsync(vals, sv, n * sizeof(uint32_t), hipMemcpyDeviceToDevice, c->stream);
        if (e != hipSuccess)
            return e;
    }
    return hipGetLastError();
}

}  // namespace dm
