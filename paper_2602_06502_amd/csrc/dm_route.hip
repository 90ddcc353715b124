// dm_route_batch: batched dual-mapping routing (Sec. 3.2; Sec. A.1.1).
//
// Kernel 1 (hash_match): one wave per request.  The wave walks the prompt
// 64 blocks at a time, lane l owning block l of the chunk:
//   - NH digest of its block from B/4 16-byte loads;
//   - the affine chain H[b] = H[b-1] P + NH(b) evaluated for all 64 lanes at
//     once: with Q = P^-1 mod 2^64, H[c+l] = P^(l+1) (G + sum_{k<=l} NH(c+k)
//     Q^(k+1)) where G carries H of the previous chunk -- one wave prefix
//     sum of u64 instead of a serial chain;
//   - block key mix64(H xor seed);
//   - in the first chunk, the f2 chain over the first K blocks (one wave
//     sum) and both ring lookups give the candidate pair;
//   - first-miss probing of both candidates' tables: each round 8 groups of
//     8 lanes read one 64-byte bucket for up to 4 blocks per candidate (8
//     when one candidate is done) and stop at the first block missing.
// Kernel 2 (select): the SLO-aware choice in request order with loads kept
// in registers of one wave and updated after every request.
#include <algorithm>

#include "dm_internal.h"

namespace dm {
namespace {

constexpr int kRouteThreads = 256;

struct RouteArgs {
    const int32_t* tokens;
    const int64_t* offsets;
    uint64_t n;
    const HashParams* hp;
    uint32_t key_blocks;
    RingView r1, r2;
    const uint32_t* next_live;
    uint32_t n_live;
    const uint64_t* tables;
    uint32_t log2slots;
    const uint64_t* bstart;   // [n+1] or null
    uint64_t* block_keys;     // or null
    uint64_t* key_out;
    uint32_t* cand_out;
    uint32_t* match_out;
    uint8_t* flags_out;
    uint32_t* status;
};

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

// Bit g (g = 0..7) = bit 8g of m: one flag per 8-lane group.
__device__ __forceinline__ uint32_t group_bits(uint64_t m)
{
    uint32_t r = 0;
#pragma unroll
    for (int g = 0; g < 8; g++)
        r |= (uint32_t)((m >> (8 * g)) & 1) << g;
    return r;
}

template <int B>
__global__ __launch_bounds__(kRouteThreads) void hash_match_kernel(RouteArgs a)
{
    const int lane = lane_id();
    const uint64_t gw = ((uint64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    const uint64_t nw = ((uint64_t)gridDim.x * blockDim.x) >> 6;
    const HashParams* hp = a.hp;
    const uint64_t seed1 = hp->seed[0], seed2 = hp->seed[1];
    const uint64_t H01 = hp->H0[0], H02 = hp->H0[1];
    const uint64_t q1 = hp->qpow[0][lane], p1 = hp->ppow[0][lane], q2 = hp->qpow[1][lane];
    uint32_t k1[B], k2[B];
#pragma unroll
    for (int j = 0; j < B; j++) {
        k1[j] = hp->kk[0][j];
        k2[j] = hp->kk[1][j];
    }
    const uint64_t nbk = 1ull << (a.log2slots - 3);
    const int g = lane >> 3, sl = lane & 7;

    for (uint64_t r = gw; r < a.n; r += nw) {
        const int64_t o0 = a.offsets[r], o1 = a.offsets[r + 1];
        const int64_t len = o1 - o0;
        if (o0 < 0 || len < 0) {
            if (lane == 0) {
                atomicOr(a.status, kErrInval);
                a.key_out[r] = 0;
                a.key_out[a.n + r] = 0;
                a.cand_out[r] = 0;
                a.cand_out[a.n + r] = 0;
                a.match_out[r] = 0;
                a.match_out[a.n + r] = 0;
                a.flags_out[r] = 0;
            }
            continue;
        }
        const uint64_t nfull = (uint64_t)len / B;
        const uint32_t kr = (uint32_t)(nfull < a.key_blocks ? nfull : a.key_blocks);
        const int32_t* tp = a.tokens + o0;
        uint64_t* bk = a.block_keys ? a.block_keys + a.bstart[r] : nullptr;

        uint64_t x1 = 0, x2 = 0;
        uint32_t c1 = 0, c2 = 0;
        bool fix = false;
        uint64_t nx1 = 0, nx2 = 0;  // leading blocks confirmed cached
        bool a1 = true, a2 = true;  // candidate still matching

        auto lookup = [&]() {
            uint32_t own = 0;
            if (lane < 2)
                own = ring_owner(lane ? a.r2 : a.r1, lane ? x2 : x1);
            c1 = __builtin_amdgcn_readlane(own, 0);
            const uint32_t raw2 = __builtin_amdgcn_readlane(own, 1);
            if (raw2 != c1) {
                c2 = raw2;
            } else {
                fix = true;
                c2 = a.n_live >= 2 ? a.next_live[c1] : c1;
            }
            if (c2 == c1)
                a2 = false;  // a single live instance: both candidates are one
        };

        if (nfull == 0) {
            x1 = mix64(H01 ^ seed1);
            x2 = mix64(H02 ^ seed2);
            lookup();
        }

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
            if (bk && valid)
                bk[b] = h;
            G = readlane_u64(H, kWave - 1);
            if (cb == 0) {
                x1 = readlane_u64(h, (int)kr - 1);
                const uint64_t S2 = wave_sum_u64(lane < (int)kr ? nh2 * q2 : 0);
                x2 = mix64(((H02 + S2) * hp->ppow[1][kr - 1]) ^ seed2);
                lookup();
            }
            // first-miss probing of the blocks of this chunk
            const uint64_t cend = cb + kWave < nfull ? cb + kWave : nfull;
            while ((a1 && nx1 < cend) || (a2 && nx2 < cend)) {
                const bool both = a1 && a2 && nx1 < cend && nx2 < cend;
                const int solo = (a1 && nx1 < cend) ? 0 : 1;  // the prober when not both
                int cs, gi;
                uint64_t blk;
                if (both) {
                    cs = g >> 2;
                    gi = g & 3;
                } else {
                    cs = solo;
                    gi = g;
                }
                blk = (cs ? nx2 : nx1) + gi;
                const bool act = blk < cend;
                const uint64_t key = canon_key(shfl_u64(h, (int)((act ? blk : cb) - cb)));
                const uint64_t* tab = a.tables + ((uint64_t)(cs ? c2 : c1) << a.log2slots);
                uint64_t bkt = home_bucket(key, a.log2slots);
                bool pend = act, hit = false;
                for (uint64_t step = 0;; step++) {
                    const uint64_t v = pend ? tab[bkt * kBucket + sl] : 0;
                    const uint64_t eqm = ballot(pend && v == key);
                    const uint64_t emm = ballot(pend && v == kEmpty);
                    const uint64_t gm = 0xFFull << (8 * g);
                    if (pend) {
                        if (eqm & gm) {
                            hit = true;
                            pend = false;
                        } else if (emm & gm) {
                            pend = false;
                        } else if (step + 1 >= nbk) {
                            pend = false;  // whole table scanned: absent
                        }
                    }
                    if (!ballot(pend))
                        break;
                    bkt = (bkt + 1) & (nbk - 1);
                }
                const uint32_t gact = group_bits(ballot(act)), ghit = group_bits(ballot(hit));
                // candidate 0 owns groups [0, 4) when both probe, else all 8 (if cs = 0)
                for (int cc = 0; cc < 2; cc++) {
                    uint32_t own;
                    if (both)
                        own = cc == 0 ? 0x0Fu : 0xF0u;
                    else
                        own = solo == cc ? 0xFFu : 0u;
                    const uint32_t am = gact & own;
                    if (!am)
                        continue;
                    const uint32_t miss = am & ~ghit;
                    const int first = __builtin_ctz(own);
                    uint64_t& nx = cc ? nx2 : nx1;
                    if (miss) {
                        nx += (uint64_t)(__builtin_ctz(miss) - first);
                        (cc ? a2 : a1) = false;
                    } else {
                        nx += (uint64_t)__builtin_popcount(am);
                    }
                }
            }
        }
        if (c1 == c2)
            nx2 = nx1;
        if (lane == 0) {
            a.key_out[r] = x1;
            a.key_out[a.n + r] = x2;
            a.cand_out[r] = c1;
            a.cand_out[a.n + r] = c2;
            a.match_out[r] = (uint32_t)nx1;
            a.match_out[a.n + r] = (uint32_t)nx2;
            a.flags_out[r] = fix ? 8 : 0;
        }
    }
}

// In-order SLO-aware selection.  One wave; loads of slots < 64*R live in
// registers (lane l holds slot 64k + l in L[k]); each request reads its two
// candidates' loads with readlane, decides, and adds its uncached tokens to
// the chosen slot.  Records are fetched 64 at a time, one per lane.
template <int R>
__global__ __launch_bounds__(kWave) void select_kernel(const int64_t* __restrict__ offsets,
                                                       uint64_t n, uint32_t bshift,
                                                       const uint32_t* __restrict__ cand,
                                                       const uint32_t* __restrict__ match,
                                                       uint8_t* __restrict__ flags,
                                                       uint32_t* __restrict__ chosen,
                                                       int64_t* __restrict__ ttft,
                                                       int64_t* __restrict__ loads, uint32_t S,
                                                       int64_t base, int64_t per, uint32_t qshift,
                                                       int64_t slo)
{
    const int lane = lane_id();
    int64_t L[R];
#pragma unroll
    for (int k = 0; k < R; k++) {
        const uint32_t i = 64 * k + lane;
        L[k] = i < S ? loads[i] : 0;
    }
    auto get = [&](uint32_t c) -> int64_t {
        int64_t v = 0;
#pragma unroll
        for (int k = 0; k < R; k++) {
            const int64_t t = (int64_t)readlane_u64((uint64_t)L[k], c & 63);
            if ((c >> 6) == (uint32_t)k)
                v = t;
        }
        return v;
    };
    for (uint64_t r0 = 0; r0 < n; r0 += kWave) {
        const uint64_t r = r0 + lane;
        const bool ok = r < n;
        const uint32_t c1v = ok ? cand[r] : 0, c2v = ok ? cand[n + r] : 0;
        const uint32_t m1v = ok ? match[r] : 0, m2v = ok ? match[n + r] : 0;
        const int64_t lenv = ok ? offsets[r + 1] - offsets[r] : 0;
        const uint32_t fv = ok ? flags[r] : 0;
        uint32_t my_ch = 0, my_fl = 0;
        int64_t my_t = 0;
        const int cnt = (int)(n - r0 < (uint64_t)kWave ? n - r0 : kWave);
        for (int j = 0; j < cnt; j++) {
            const uint32_t C1 = __builtin_amdgcn_readlane(c1v, j);
            const uint32_t C2 = __builtin_amdgcn_readlane(c2v, j);
            const uint32_t M1 = __builtin_amdgcn_readlane(m1v, j);
            const uint32_t M2 = __builtin_amdgcn_readlane(m2v, j);
            const int64_t LEN = (int64_t)readlane_u64((uint64_t)lenv, j);
            uint32_t f = __builtin_amdgcn_readlane(fv, j);
            const int64_t L1 = get(C1), L2 = get(C2);
            const int64_t u1 = LEN - ((int64_t)M1 << bshift), u2 = LEN - ((int64_t)M2 << bshift);
            const int64_t t1 = base + per * u1 + (L1 >> qshift);
            const int64_t t2 = base + per * u2 + (L2 >> qshift);
            if (t1 > slo && t2 > slo)
                f |= 2;
            bool pick1;
            if (M1 == M2) {
                f |= 4;
                pick1 = L1 <= L2;
            } else {
                const bool aff1 = M1 > M2;
                const int64_t ta = aff1 ? t1 : t2, La = aff1 ? L1 : L2, Lo = aff1 ? L2 : L1;
                if (ta <= slo || !(Lo < La)) {
                    pick1 = aff1;
                } else {
                    pick1 = !aff1;
                    f |= 1;
                }
            }
            const uint32_t ch = pick1 ? C1 : C2;
            const int64_t add = pick1 ? u1 : u2;
#pragma unroll
            for (int k = 0; k < R; k++)
                if ((ch >> 6) == (uint32_t)k && lane == (int)(ch & 63))
                    L[k] += add;
            if (lane == j) {
                my_ch = ch;
                my_t = pick1 ? t1 : t2;
                my_fl = f;
            }
        }
        if (ok) {
            chosen[r] = my_ch;
            ttft[r] = my_t;
            flags[r] = (uint8_t)my_fl;
        }
    }
#pragma unroll
    for (int k = 0; k < R; k++) {
        const uint32_t i = 64 * k + lane;
        if (i < S)
            loads[i] = L[k];
    }
}

// Same rule with loads in LDS, for large slot spaces.
__global__ __launch_bounds__(kWave) void select_lds_kernel(const int64_t* __restrict__ offsets,
                                                           uint64_t n, uint32_t bshift,
                                                           const uint32_t* __restrict__ cand,
                                                           const uint32_t* __restrict__ match,
                                                           uint8_t* __restrict__ flags,
                                                           uint32_t* __restrict__ chosen,
                                                           int64_t* __restrict__ ttft,
                                                           int64_t* __restrict__ loads, uint32_t S,
                                                           int64_t base, int64_t per,
                                                           uint32_t qshift, int64_t slo)
{
    __shared__ int64_t L[kMaxSlots];
    const int lane = lane_id();
    for (uint32_t i = lane; i < S; i += kWave)
        L[i] = loads[i];
    __syncthreads();
    for (uint64_t r0 = 0; r0 < n; r0 += kWave) {
        const uint64_t r = r0 + lane;
        const bool ok = r < n;
        const uint32_t c1v = ok ? cand[r] : 0, c2v = ok ? cand[n + r] : 0;
        const uint32_t m1v = ok ? match[r] : 0, m2v = ok ? match[n + r] : 0;
        const int64_t lenv = ok ? offsets[r + 1] - offsets[r] : 0;
        const uint32_t fv = ok ? flags[r] : 0;
        uint32_t my_ch = 0, my_fl = 0;
        int64_t my_t = 0;
        const int cnt = (int)(n - r0 < (uint64_t)kWave ? n - r0 : kWave);
        for (int j = 0; j < cnt; j++) {
            const uint32_t C1 = __builtin_amdgcn_readlane(c1v, j);
            const uint32_t C2 = __builtin_amdgcn_readlane(c2v, j);
            const uint32_t M1 = __builtin_amdgcn_readlane(m1v, j);
            const uint32_t M2 = __builtin_amdgcn_readlane(m2v, j);
            const int64_t LEN = (int64_t)readlane_u64((uint64_t)lenv, j);
            uint32_t f = __builtin_amdgcn_readlane(fv, j);
            const int64_t L1 = L[C1], L2 = L[C2];
            const int64_t u1 = LEN - ((int64_t)M1 << bshift), u2 = LEN - ((int64_t)M2 << bshift);
            const int64_t t1 = base + per * u1 + (L1 >> qshift);
            const int64_t t2 = base + per * u2 + (L2 >> qshift);
            if (t1 > slo && t2 > slo)
                f |= 2;
            bool pick1;
            if (M1 == M2) {
                f |= 4;
                pick1 = L1 <= L2;
            } else {
                const bool aff1 = M1 > M2;
                const int64_t ta = aff1 ? t1 : t2, La = aff1 ? L1 : L2, Lo = aff1 ? L2 : L1;
                if (ta <= slo || !(Lo < La)) {
                    pick1 = aff1;
                } else {
                    pick1 = !aff1;
                    f |= 1;
                }
            }
            const uint32_t ch = pick1 ? C1 : C2;
            const int64_t nv = (pick1 ? L1 : L2) + (pick1 ? u1 : u2);
            __syncthreads();
            if (lane == 0)
                L[ch] = nv;
            __syncthreads();
            if (lane == j) {
                my_ch = ch;
                my_t = pick1 ? t1 : t2;
                my_fl = f;
            }
        }
        if (ok) {
            chosen[r] = my_ch;
            ttft[r] = my_t;
            flags[r] = (uint8_t)my_fl;
        }
    }
    __syncthreads();
    for (uint32_t i = lane; i < S; i += kWave)
        loads[i] = L[i];
}

template <int B>
void launch_hash(const RouteArgs& a, uint32_t grid, hipStream_t s)
{
    hash_match_kernel<B><<<grid, kRouteThreads, 0, s>>>(a);
}

}  // namespace

hipError_t route(dm_ctx* c, const int32_t* tokens, const int64_t* offsets, uint64_t n,
                 int64_t* loads, const dm_route_out* out)
{
    hipError_t e = hipSuccess;
    uint64_t* bstart = nullptr;
    if (c->timing) {
        c->timed_bk = out->block_keys != nullptr;
        e = hipEventRecord(c->ev[0], c->stream);
        if (e != hipSuccess)
            return e;
    }
    if (out->block_keys) {
        bstart = static_cast<uint64_t*>(scratch_get(c, 0, (n + 1) * sizeof(uint64_t), &e));
        if (!bstart)
            return e;
        e = block_starts(c, offsets, n, bstart);
        if (e != hipSuccess)
            return e;
    }
    RouteArgs a;
    a.tokens = tokens;
    a.offsets = offsets;
    a.n = n;
    a.hp = c->d_hp;
    a.key_blocks = c->cfg.key_blocks;
    a.r1 = view(c->ring[c->cur][0]);
    a.r2 = view(c->ring[c->cur][1]);
    a.next_live = c->d_next_live;
    a.n_live = c->n_live;
    a.tables = c->d_tables;
    a.log2slots = c->cfg.index_log2_slots;
    a.bstart = bstart;
    a.block_keys = out->block_keys;
    a.key_out = out->key;
    a.cand_out = out->cand;
    a.match_out = out->match;
    a.flags_out = out->flags;
    a.status = c->d_status;
    if (c->timing && (e = hipEventRecord(c->ev[1], c->stream)) != hipSuccess)
        return e;
    const uint64_t waves_per_block = kRouteThreads / kWave;
    const uint64_t want = (n + waves_per_block - 1) / waves_per_block;
    const uint32_t grid = (uint32_t)std::min<uint64_t>(want, 1u << 20);
    switch (c->cfg.block_size) {
        case 4: launch_hash<4>(a, grid, c->stream); break;
        case 8: launch_hash<8>(a, grid, c->stream); break;
        case 16: launch_hash<16>(a, grid, c->stream); break;
        case 32: launch_hash<32>(a, grid, c->stream); break;
        case 64: launch_hash<64>(a, grid, c->stream); break;
        default: return hipErrorInvalidValue;
    }
    e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    if (c->timing && (e = hipEventRecord(c->ev[2], c->stream)) != hipSuccess)
        return e;
    uint32_t bshift = 0;
    while ((1u << bshift) < c->cfg.block_size)
        bshift++;
    const uint32_t S = c->cfg.max_slots;
    const dm_config& k = c->cfg;
    if (S <= 64)
        select_kernel<1><<<1, kWave, 0, c->stream>>>(offsets, n, bshift, out->cand, out->match,
                                                      out->flags, out->chosen, out->ttft_us, loads, S,
                                                      k.ttft_base_us, k.ttft_per_token_us,
                                                      c->shift_div, k.slo_us);
    else if (S <= 256)
        select_kernel<4><<<1, kWave, 0, c->stream>>>(offsets, n, bshift, out->cand, out->match,
                                                      out->flags, out->chosen, out->ttft_us, loads, S,
                                                      k.ttft_base_us, k.ttft_per_token_us,
                                                      c->shift_div, k.slo_us);
    else
        select_lds_kernel<<<1, kWave, 0, c->stream>>>(offsets, n, bshift, out->cand, out->match,
                                                      out->flags, out->chosen, out->ttft_us, loads,
                                                      S, k.ttft_base_us, k.ttft_per_token_us,
                                                      c->shift_div, k.slo_us);
    e = hipGetLastError();
    if (e == hipSuccess && c->timing)
        e = hipEventRecord(c->ev[3], c->stream);
    return e;
}

}  // namespace dm
