// Chained block keys and ring keys of every request (Sec. 3.2; Sec. A.1.1).
//
// Each wave takes requests in turn (one, unless the batch has more than 4 Mi
// requests) and walks each prompt 64 blocks at a time, lane l owning block l
// of the chunk:
//   - NH digest of its block from B/4 16-byte loads;
//   - the affine chain H[b] = H[b-1] P + NH(b) for all 64 lanes at once:
//     with Q = P^-1 mod 2^64, H[c+l] = P^(l+1) (G + sum_{k<=l} NH(c+k)
//     Q^(k+1)), G carrying H of the previous chunk -- a wave prefix sum of
//     u64 (register-level DPP moves) instead of a serial chain;
//   - block key mix64(H xor seed), stored for every full block;
//   - in the first chunk the f2 chain over the first K blocks (one wave
//     sum) gives the second ring key.
#include "dm_internal.h"

namespace dm {
namespace {

constexpr int kHashThreads = 256;
constexpr uint32_t kHashBlocks = 1u << 20;  // one wave per request up to 4 Mi requests

typedef int v4i __attribute__((ext_vector_type(4), aligned(4)));

// NH over the B tokens at p (4-byte aligned) with key words kk.
template <int B>
__device__ __forceinline__ uint64_t nh_block(const int32_t* p, const uint32_t* kk)
{
    uint64_t acc = 0;
#pragma unroll
    for (int j = 0; j < B; j += 4) {
        const v4i v = *reinterpret_cast<const v4i*>(p + j);
        acc += (uint64_t)((uint32_t)v.x + kk[j]) * (uint32_t)((uint32_t)v.y + kk[j + 1]);
        acc += (uint64_t)((uint32_t)v.z + kk[j + 2]) * (uint32_t)((uint32_t)v.w + kk[j + 3]);
    }
    return acc;
}

template <int B>
__device__ __forceinline__ void nh_block2(const int32_t* p, const uint32_t* k1, const uint32_t* k2,
                                          uint64_t& a1, uint64_t& a2)
{
    a1 = 0;
    a2 = 0;
#pragma unroll
    for (int j = 0; j < B; j += 4) {
        const v4i v = *reinterpret_cast<const v4i*>(p + j);
        a1 += (uint64_t)((uint32_t)v.x + k1[j]) * (uint32_t)((uint32_t)v.y + k1[j + 1]);
        a1 += (uint64_t)((uint32_t)v.z + k1[j + 2]) * (uint32_t)((uint32_t)v.w + k1[j + 3]);
        a2 += (uint64_t)((uint32_t)v.x + k2[j]) * (uint32_t)((uint32_t)v.y + k2[j + 1]);
        a2 += (uint64_t)((uint32_t)v.z + k2[j + 2]) * (uint32_t)((uint32_t)v.w + k2[j + 3]);
    }
}

struct HashArgs {
    const int32_t* tokens;
    const int64_t* offsets;
    uint64_t n;             // batch size (key_out holds 2n keys)
    uint64_t r0, r1;        // requests of this launch
    const HashParams* hp;
    uint32_t key_blocks;
    const uint64_t* bstart;  // [n+1]
    const uint32_t* bad;     // offsets break the batch's rule (set by the block-start scan)
    uint64_t* hkeys;         // [bstart[n]] f1 block keys
    uint64_t* key_out;       // [2n]
    uint32_t* status;
};

template <int B>
__global__ __launch_bounds__(kHashThreads) void hash_kernel(HashArgs a)
{
    const int lane = lane_id();
    const uint64_t gw = ((uint64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    const uint64_t nw = ((uint64_t)gridDim.x * blockDim.x) >> 6;
    const HashParams* hp = a.hp;
    const uint64_t seed1 = hp->seed[0], seed2 = hp->seed[1];
    const uint64_t H01 = hp->H0[0], H02 = hp->H0[1];
    const uint64_t q1 = hp->qpow[0][lane], p1 = hp->ppow[0][lane], q2 = hp->qpow[1][lane];
    // Malformed offsets (reported by the block-start scan): ring keys 0, no
    // block key.  No store precedes the parameter loads, so they stay scalar.
    const bool bad = *a.bad != 0;
    uint32_t k1[B], k2[B];
#pragma unroll
    for (int j = 0; j < B; j++) {
        k1[j] = hp->kk[0][j];
        k2[j] = hp->kk[1][j];
    }
    // The next request's offsets and block start are fetched while this one
    // is hashed, so no wave waits on them between requests.
    int64_t o0 = 0, o1 = 0;
    uint64_t bs = 0;
    if (a.r0 + gw < a.r1) {
        o0 = a.offsets[a.r0 + gw];
        o1 = a.offsets[a.r0 + gw + 1];
        bs = a.bstart[a.r0 + gw];
    }
    for (uint64_t r = a.r0 + gw; r < a.r1; r += nw) {
        const uint64_t rn = r + nw;
        int64_t no0 = 0, no1 = 0;
        uint64_t nbs = 0;
        if (rn < a.r1) {
            no0 = a.offsets[rn];
            no1 = a.offsets[rn + 1];
            nbs = a.bstart[rn];
        }
        const int64_t len = o1 - o0;
        if (bad) {
            if (lane == 0) {
                a.key_out[r] = 0;
                a.key_out[a.n + r] = 0;
            }
            o0 = no0;
            o1 = no1;
            bs = nbs;
            continue;
        }
        const uint64_t nfull = (uint64_t)len / B;
        const uint32_t kr = (uint32_t)(nfull < a.key_blocks ? nfull : a.key_blocks);
        const int32_t* tp = a.tokens + o0;
        uint64_t* hk = a.hkeys + bs;
        uint64_t x1 = mix64(H01 ^ seed1), x2 = mix64(H02 ^ seed2);  // empty-prefix keys
        uint64_t G = H01;
        for (uint64_t cb = 0; cb < nfull; cb += kWave) {
            const uint64_t b = cb + lane;
            const bool valid = b < nfull;
            uint64_t nh1 = 0, nh2 = 0;
            if (cb == 0) {
                if (valid)
                    nh_block2<B>(tp + b * B, k1, k2, nh1, nh2);
            } else if (valid) {
                nh1 = nh_block<B>(tp + b * B, k1);
            }
            const uint64_t S = wave_incl_sum_u64(nh1 * q1, lane);
            const uint64_t H = (G + S) * p1;
            const uint64_t h = mix64(H ^ seed1);
            if (valid)
                hk[b] = h;
            G = readlane_u64(H, kWave - 1);
            if (cb == 0) {
                x1 = readlane_u64(h, (int)kr - 1);
                const uint64_t S2 = wave_sum_u64(lane < (int)kr ? nh2 * q2 : 0);
                x2 = mix64(((H02 + S2) * hp->ppow[1][kr - 1]) ^ seed2);
            }
        }
        if (lane == 0) {
            a.key_out[r] = x1;
            a.key_out[a.n + r] = x2;
        }
        o0 = no0;
        o1 = no1;
        bs = nbs;
    }
}

template <int B>
void launch_hash(const HashArgs& a, uint32_t grid, hipStream_t s)
{
    hash_kernel<B><<<grid, kHashThreads, 0, s>>>(a);
}

}  // namespace

hipError_t hash_blocks(dm_ctx* c, const int32_t* tokens, const int64_t* offsets, uint64_t n,
                       const uint64_t* bstart, const uint32_t* bad, uint64_t* hkeys,
                       uint64_t* key_out, uint64_t r0, uint64_t r1)
{
    HashArgs ha{tokens, offsets, n,     r0,      r1,        c->d_hp,
                c->cfg.key_blocks, bstart, bad, hkeys, key_out, c->d_status};
    const uint32_t grid = grid_for(r1 > r0 ? r1 - r0 : 0, kHashThreads / kWave, kHashBlocks);
    switch (c->cfg.block_size) {
        case 4: launch_hash<4>(ha, grid, c->stream); break;
        case 8: launch_hash<8>(ha, grid, c->stream); break;
        case 16: launch_hash<16>(ha, grid, c->stream); break;
        case 32: launch_hash<32>(ha, grid, c->stream); break;
        case 64: launch_hash<64>(ha, grid, c->stream); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace dm
