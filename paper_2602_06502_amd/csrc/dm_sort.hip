// Stable LSD radix sort of (u64 key, u32 value) pairs, 8-bit digits.
// Per pass: tile digit histograms (digit-major), one exclusive scan over
// them, and a stable scatter that ranks equal digits inside each 64-lane
// sub-tile with ballots.
#include "dm_internal.h"

namespace dm {
namespace {

constexpr int kSortThreads = 256;
constexpr int kSortItems = 4;
constexpr uint64_t kSortTile = kSortThreads * kSortItems;
constexpr int kSubtiles = kSortItems * (kSortThreads / kWave);
constexpr int kSortSlot = kSlotSort;

__global__ __launch_bounds__(kSortThreads) void digit_hist_kernel(const uint64_t* __restrict__ keys,
                                                                  uint64_t n, int shift,
                                                                  uint64_t ntiles,
                                                                  uint64_t* __restrict__ cnt)
{
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

__global__ __launch_bounds__(kSortThreads) void digit_scatter_kernel(
    const uint64_t* __restrict__ keys, const uint32_t* __restrict__ vals, uint64_t n, int shift,
    uint64_t ntiles, const uint64_t* __restrict__ offs, uint64_t* __restrict__ okeys,
    uint32_t* __restrict__ ovals)
{
    __shared__ uint32_t sub[kSubtiles][256];
    for (int k = threadIdx.x; k < kSubtiles * 256; k += kSortThreads)
        (&sub[0][0])[k] = 0;
    __syncthreads();
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const uint64_t lt = (lane ? (~0ull >> (64 - lane)) : 0ull);
    const uint64_t base = blockIdx.x * kSortTile;
    uint64_t k[kSortItems];
    uint32_t v[kSortItems], d[kSortItems], rank[kSortItems];
    bool ok[kSortItems];
#pragma unroll
    for (int it = 0; it < kSortItems; it++) {
        const uint64_t i = base + it * kSortThreads + threadIdx.x;
        ok[it] = i < n;
        k[it] = ok[it] ? keys[i] : 0;
        v[it] = ok[it] && vals ? vals[i] : 0;
        d[it] = (uint32_t)((k[it] >> shift) & 0xFF);
        uint64_t peers = ballot(ok[it]);
#pragma unroll
        for (int b = 0; b < 8; b++) {
            const bool bit = (d[it] >> b) & 1;
            const uint64_t m = ballot(bit);
            peers &= bit ? m : ~m;
        }
        rank[it] = __popcll(peers & lt);
        // the lowest lane of each peer group records the group size
        if (ok[it] && (peers & lt) == 0)
            sub[it * (kSortThreads / kWave) + w][d[it]] = __popcll(peers);
    }
    __syncthreads();
    // exclusive scan over sub-tiles, per digit (thread = digit)
    {
        uint32_t run = 0;
        for (int s = 0; s < kSubtiles; s++) {
            const uint32_t c = sub[s][threadIdx.x];
            sub[s][threadIdx.x] = run;
            run += c;
        }
    }
    __syncthreads();
#pragma unroll
    for (int it = 0; it < kSortItems; it++) {
        if (!ok[it])
            continue;
        const uint64_t pos = offs[(uint64_t)d[it] * ntiles + blockIdx.x] +
                             sub[it * (kSortThreads / kWave) + w][d[it]] + rank[it];
        okeys[pos] = k[it];
        if (ovals)
            ovals[pos] = v[it];
    }
}

}  // namespace

uint64_t sort_scan_len(uint64_t n) { return 256 * ((n + kSortTile - 1) / kSortTile); }

// digit counts and their offsets, 256 per tile each
uint64_t sort_scratch_bytes(uint64_t n) { return 2 * sort_scan_len(n) * sizeof(uint64_t); }

hipError_t radix_sort_kv(dm_ctx* c, uint64_t* keys, uint32_t* vals, uint64_t* ktmp,
                         uint32_t* vtmp, uint64_t n, int bits)
{
    if (n < 2 || bits <= 0)
        return hipSuccess;
    const uint64_t ntiles = (n + kSortTile - 1) / kSortTile;
    hipError_t e;
    uint64_t* cnt = static_cast<uint64_t*>(scratch_get(c, kSortSlot, sort_scratch_bytes(n), &e));
    if (!cnt)
        return e;
    uint64_t* offs = cnt + 256 * ntiles;
    uint64_t *sk = keys, *dk = ktmp;
    uint32_t *sv = vals, *dv = vtmp;
    int passes = 0;
    for (int shift = 0; shift < bits; shift += 8, passes++) {
        digit_hist_kernel<<<ntiles, kSortThreads, 0, c->stream>>>(sk, n, shift, ntiles, cnt);
        e = exclusive_scan_u64(c, cnt, 256 * ntiles, offs, nullptr);
        if (e != hipSuccess)
            return e;
        digit_scatter_kernel<<<ntiles, kSortThreads, 0, c->stream>>>(sk, sv, n, shift, ntiles,
                                                                     offs, dk, dv);
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
