// Exclusive prefix sums over u64 sequences (tile reduce, scan of the tile
// sums, rescan), used for per-request block offsets, stream compaction and
// the radix sort's digit offsets.
#include <vector>

#include "dm_internal.h"

namespace dm {
namespace {

constexpr int kScanThreads = 256;
constexpr int kScanItems = 4;
constexpr uint64_t kTile = kScanThreads * kScanItems;
constexpr int kScanSlot = kSlotScan;  // tile-sum levels

struct ArrayIn {
    const uint64_t* p;
    __device__ uint64_t operator()(uint64_t i) const { return p[i]; }
};

// Full blocks of request i: floor(len / B), B = 2^shift, for a prompt
// inside [0, n_tokens); a request that breaks 0 <= off[i] <= off[i+1] <=
// n_tokens counts none and sets *bad and kErrInval in the device status
// word.  When every request keeps the rule the offsets never decrease, so
// the prompts are disjoint ranges of the token array and their full blocks
// add up to at most n_tokens / B.
struct FullBlocksIn {
    const int64_t* off;
    uint32_t shift;
    uint64_t n_tokens;
    uint32_t* bad;
    uint32_t* status;
    __device__ uint64_t operator()(uint64_t i) const
    {
        const int64_t o0 = off[i], o1 = off[i + 1];
        if (o0 < 0 || o1 < o0 || (uint64_t)o1 > n_tokens) {
            atomicOr(bad, 1u);
            atomicOr(status, kErrInval);
            return 0;
        }
        return (uint64_t)(o1 - o0) >> shift;
    }
};

// Block-wide exclusive scan of one u64 per thread; also returns the total.
__device__ uint64_t block_excl_scan(uint64_t v, uint64_t* sh, uint64_t& total)
{
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const uint64_t inc = wave_incl_sum_u64(v, lane);
    if (lane == 63)
        sh[w] = inc;
    __syncthreads();
    uint64_t before = 0, tot = 0;
    for (int k = 0; k < kScanThreads / kWave; k++) {
        if (k < w)
            before += sh[k];
        tot += sh[k];
    }
    __syncthreads();
    total = tot;
    return before + inc - v;
}

template <typename In>
__global__ __launch_bounds__(kScanThreads) void tile_sum_kernel(In in, uint64_t n, uint64_t* sums)
{
    __shared__ uint64_t sh[kScanThreads / kWave];
    const uint64_t base = blockIdx.x * kTile + threadIdx.x * kScanItems;
    uint64_t s = 0;
#pragma unroll
    for (int k = 0; k < kScanItems; k++)
        if (base + k < n)
            s += in(base + k);
    uint64_t total;
    block_excl_scan(s, sh, total);
    if (threadIdx.x == 0)
        sums[blockIdx.x] = total;
}

template <typename In>
__global__ __launch_bounds__(kScanThreads) void tile_scan_kernel(In in, uint64_t n,
                                                                 const uint64_t* tile_off,
                                                                 uint64_t* out, uint64_t* total_out)
{
    __shared__ uint64_t sh[kScanThreads / kWave];
    const uint64_t base = blockIdx.x * kTile + threadIdx.x * kScanItems;
    uint64_t v[kScanItems];
    uint64_t s = 0;
#pragma unroll
    for (int k = 0; k < kScanItems; k++) {
        v[k] = base + k < n ? in(base + k) : 0;
        s += v[k];
    }
    uint64_t total;
    const uint64_t toff = tile_off ? tile_off[blockIdx.x] : 0;
    uint64_t run = block_excl_scan(s, sh, total) + toff;
#pragma unroll
    for (int k = 0; k < kScanItems; k++) {
        if (base + k < n)
            out[base + k] = run;
        run += v[k];
    }
    if (total_out && blockIdx.x == gridDim.x - 1 && threadIdx.x == 0)
        *total_out = toff + total;
}

uint64_t ntiles(uint64_t n) { return (n + kTile - 1) / kTile; }

template <typename In>
hipError_t scan_impl(dm_ctx* c, In in, uint64_t n, uint64_t* out, uint64_t* total_out)
{
    if (n == 0)
        return hipSuccess;
    // level d has n_d inputs and tiles_d tiles; n_{d+1} = tiles_d; stop at one tile
    std::vector<uint64_t> nd{n};
    while (ntiles(nd.back()) > 1)
        nd.push_back(ntiles(nd.back()));
    const size_t K = nd.size() - 1;  // levels with more than one tile: 0..K-1
    if (K == 0) {
        tile_scan_kernel<In><<<1, kScanThreads, 0, c->stream>>>(in, n, nullptr, out, total_out);
        return hipGetLastError();
    }
    // scratch: sums_d and scanned_d (tiles_d entries each) for d < K
    std::vector<uint64_t> at(K);
    uint64_t need = 0;
    for (size_t d = 0; d < K; d++) {
        at[d] = need;
        need += 2 * ntiles(nd[d]);
    }
    hipError_t e;
    uint64_t* buf = static_cast<uint64_t*>(scratch_get(c, kScanSlot, scan_scratch_bytes(n), &e));
    if (!buf)
        return e;
    auto sums = [&](size_t d) { return buf + at[d]; };
    auto scanned = [&](size_t d) { return buf + at[d] + ntiles(nd[d]); };
    tile_sum_kernel<In><<<ntiles(nd[0]), kScanThreads, 0, c->stream>>>(in, nd[0], sums(0));
    for (size_t d = 1; d < K; d++)
        tile_sum_kernel<ArrayIn><<<ntiles(nd[d]), kScanThreads, 0, c->stream>>>(
            ArrayIn{sums(d - 1)}, nd[d], sums(d));
    // top level: one tile scans sums_{K-1}
    tile_scan_kernel<ArrayIn><<<1, kScanThreads, 0, c->stream>>>(ArrayIn{sums(K - 1)}, nd[K],
                                                                  nullptr, scanned(K - 1), nullptr);
    for (size_t d = K - 1; d >= 1; d--)
        tile_scan_kernel<ArrayIn><<<ntiles(nd[d]), kScanThreads, 0, c->stream>>>(
            ArrayIn{sums(d - 1)}, nd[d], scanned(d), scanned(d - 1), nullptr);
    tile_scan_kernel<In><<<ntiles(nd[0]), kScanThreads, 0, c->stream>>>(in, nd[0], scanned(0), out,
                                                                         total_out);
    return hipGetLastError();
}

}  // namespace

// Words of tile sums a scan of n items keeps: sums and scanned sums of every
// level with more than one tile.
uint64_t scan_scratch_bytes(uint64_t n)
{
    uint64_t need = 0;
    for (uint64_t m = n; ntiles(m) > 1; m = ntiles(m))
        need += 2 * ntiles(m);
    return need * sizeof(uint64_t);
}

hipError_t exclusive_scan_u64(dm_ctx* c, const uint64_t* in, uint64_t n, uint64_t* out,
                              uint64_t* total_out)
{
    return scan_impl(c, ArrayIn{in}, n, out, total_out);
}

// starts[r] = full blocks of requests 0..r-1, for r = 0..n (starts[n] = total).
hipError_t block_starts(dm_ctx* c, const int64_t* offsets, uint64_t n, uint64_t n_tokens,
                        uint64_t* starts, uint32_t* bad)
{
    uint32_t shift = 0;
    while ((1u << shift) < c->cfg.block_size)
        shift++;
    return scan_impl(c, FullBlocksIn{offsets, shift, n_tokens, bad, c->d_status}, n, starts,
                     starts + n);
}

}  // namespace dm
