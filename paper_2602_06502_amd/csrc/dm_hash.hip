// Chained block keys, ring keys and longest cached prefixes (Sec. 3.2;
// Sec. A.1.1; the per-block KV metadata of Sec. A.3.2).
//
// One wave per request walks the prompt 64 blocks at a time, lane l owning
// block l of the chunk:
//   - NH digest of its block from B/4 16-byte loads;
//   - the affine chain H[b] = H[b-1] P + NH(b) for all 64 lanes at once:
//     with Q = P^-1 mod 2^64, H[c+l] = P^(l+1) (G + sum_{k<=l} NH(c+k)
//     Q^(k+1)), G carrying H of the previous chunk -- a wave prefix sum of
//     u64 (register-level DPP moves) instead of a serial chain;
//   - block key mix64(H xor seed).
// Three passes use this walk (dm_route.hip runs them in this order):
//   prefix   both chains over the first min(K, full blocks) blocks only:
//            the two ring keys (ring_key_kernel: several requests per wave);
//            with the prefix hotness tree on, requests whose depth-K prefix
//            is extended go on down the tree (extend_kernel) to their key
//            length K_r, both chains, and take the ring keys of depth K_r;
//   leaders  one request per group of equal ring keys (dm_probe.hip): the
//            full f1 chain, stored; each chunk's keys are probed against
//            both candidates' tables, lanes from the first unresolved block
//            (two first, then the rest of the chunk), until each
//            candidate's first absent block;
//   members  every other request: the full f1 chain (stored only when the
//            caller asks for block keys).  While within one block past the
//            leader's longer match, each chunk's keys are compared with the
//            leader's stored keys (one ballot): blocks before the first
//            disagreement s hold the leader's keys, so on a candidate where
//            the leader's match ends before s the request's match is the
//            leader's; elsewhere the request's first s blocks are present
//            and its keys are probed from block s on, chunk by chunk.
// The comparison is of keys and the probes are of keys, so every match is
// the definition's (leading blocks whose f1 keys are all in the candidate's
// index) whatever the keys are.  Requests that share a prefix with their
// leader read the leader's 8-byte keys (cache-resident) instead of probing
// 64-byte buckets for it, and no request reads its own keys back.
#include "dm_internal.h"

namespace dm {
namespace {

constexpr int kHashThreads = 256;
constexpr uint32_t kHashBlocks = 1u << 20;  // one wave per unit up to 4 Mi units
constexpr uint32_t kLeaderBlocks = 2048;    // tree walk, resume walk: at most 8,192 waves
constexpr uint32_t kLeaderGrid = 8192;      // leaders: up to 32,768 waves, one leader each

enum : int { kLeaders = 1, kResume = 2 };
constexpr uint64_t kPendKeys = 8;  // keys kept per request for the pending probes

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
    uint64_t n;               // batch size (key_out, cand and match hold 2n entries)
    const HashParams* hp;
    uint32_t key_blocks;
    uint32_t write_keys;      // members: store the block keys as well
    const uint64_t* bstart;   // [n + 1] where each request's block keys go
    const uint32_t* bad;      // offsets break the batch's rule (set by the block-start scan)
    uint64_t* hkeys;          // f1 block keys
    uint64_t* key_out;        // prefix: [2n] ring keys
    GroupView gv;
    const uint32_t* cand;     // [2n]
    uint32_t* match;          // [2n]
    const uint64_t* tables;
    uint32_t log2slots;
    uint32_t* status;
    // members pass
    const struct MemberRec* rec;  // [n]
    uint64_t* pkeys;              // [n * kPendKeys]
    uint64_t* pend;               // [n]
    const uint64_t* resume;       // resume list
    const unsigned long long* resume_count;
    // prefix hotness tree (kl_on = 0: fixed K)
    uint32_t kl_on;
    uint32_t kl_log2;
    const uint64_t* kl_tab;       // extended prefixes
    uint32_t* ext_list;           // requests whose depth-K prefix is extended
    unsigned long long* ext_count;
    const unsigned long long* ext_count_in;
    uint32_t* key_len;            // [n] or null
    // f1 digests NH(j) of blocks j < min(K, full blocks), [n * key_blocks]:
    // written by the prefix pass so that the members pass need not read
    // those tokens again (null: not kept)
    uint64_t* nh0;
};

// Index of this wave in the grid, in a scalar register: the compiler cannot
// see that threadIdx.x / 64 is the same for the whole wave, and everything
// derived from a vector index (a request's record, its offsets) would take
// vector loads and vector registers.
__device__ __forceinline__ uint64_t wave_index()
{
    const uint32_t w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    return (uint64_t)blockIdx.x * (blockDim.x >> 6) + w;
}

// First block absent from table tab among this chunk's blocks [pb, hi)
// (cb <= pb, hi <= cb + 64), lanes pb and pb + 1 first and the rest only if
// both are present.  Returns false when every probed block is present.
__device__ __forceinline__ bool chunk_first_absent(const uint64_t* tab, uint32_t ls, uint64_t ck,
                                                   uint64_t cb, uint64_t pb, uint64_t hi, int lane,
                                                   uint64_t* first)
{
    const uint64_t b = cb + lane;
    const bool in_a = b >= pb && b < pb + 2 && b < hi;
    uint64_t m = ballot(in_a && !table_has(tab, ls, ck));
    if (!m && pb + 2 < hi) {
        const bool in_b = b >= pb + 2 && b < hi;
        m = ballot(in_b && !table_has(tab, ls, ck));
    }
    if (!m)
        return false;
    *first = cb + (uint64_t)__builtin_ctzll(m);
    return true;
}

// Ring keys of every request: lane group of g = 2^k >= K lanes per request
// (64 / g requests per wave), lane j of a group holding block j.  The ring
// key is block K_r - 1's, K_r = min(K, full blocks): with the chain's
// closed form H[K_r - 1] = P^K_r (H[-1] + sum_{j<K_r} NH(j) Q^(j+1)), a sum
// over the group's lanes (xor shuffles) replaces the scan.
template <int B>
__global__ __launch_bounds__(kHashThreads) void ring_key_kernel(HashArgs a, uint32_t glog)
{
    const int lane = lane_id();
    const uint32_t g = 1u << glog, j = (uint32_t)lane & (g - 1);
    const uint64_t gw = wave_index();
    const uint64_t nw = ((uint64_t)gridDim.x * blockDim.x) >> 6;
    const uint64_t per_wave = kWave >> glog;
    const HashParams* hp = a.hp;
    const uint64_t seed1 = hp->seed[0], seed2 = hp->seed[1];
    const uint64_t H01 = hp->H0[0], H02 = hp->H0[1];
    const uint64_t q1 = hp->qpow[0][j], q2 = hp->qpow[1][j];
    const bool bad = *a.bad != 0;
    uint32_t k1[B], k2[B];
#pragma unroll
    for (int t = 0; t < B; t++) {
        k1[t] = hp->kk[0][t];
        k2[t] = hp->kk[1][t];
    }
    for (uint64_t base = gw * per_wave; base < a.n; base += nw * per_wave) {
        const uint64_t r = base + ((uint32_t)lane >> glog);
        uint32_t kr = 0;
        int64_t o0 = 0;
        uint64_t nfull = 0;
        if (r < a.n && !bad) {
            o0 = a.offsets[r];
            nfull = (uint64_t)(a.offsets[r + 1] - o0) / B;
            kr = (uint32_t)(nfull < a.key_blocks ? nfull : a.key_blocks);
        }
        uint64_t nh1 = 0, nh2 = 0;
        if (j < kr)
            nh_block2<B>(a.tokens + o0 + (uint64_t)j * B, k1, k2, nh1, nh2);
        if (a.nh0 && j < kr)
            a.nh0[r * a.key_blocks + j] = nh1;
        uint64_t s1 = nh1 * q1, s2 = nh2 * q2;
        for (uint32_t d = 1; d < g; d <<= 1) {
            s1 += shfl_xor_u64(s1, (int)d);
            s2 += shfl_xor_u64(s2, (int)d);
        }
        bool down = false;  // the depth-K prefix is extended: go on down the tree
        if (r < a.n && j == 0) {
            uint64_t x1 = mix64(H01 ^ seed1), x2 = mix64(H02 ^ seed2);  // empty-prefix keys
            if (kr > 0) {
                x1 = mix64(((H01 + s1) * hp->ppow[0][kr - 1]) ^ seed1);
                x2 = mix64(((H02 + s2) * hp->ppow[1][kr - 1]) ^ seed2);
            }
            a.key_out[r] = bad ? 0 : x1;
            a.key_out[a.n + r] = bad ? 0 : x2;
            if (a.key_len)
                a.key_len[r] = kr;
            // x1 is the f1 key of block K - 1: the request's depth-K prefix
            if (a.kl_on && !bad && nfull > a.key_blocks)
                down = table_has(a.kl_tab, a.kl_log2, canon_key(x1));
        }
        if (a.kl_on) {
            // one append per wave for the requests going down the tree
            const uint64_t m = ballot(down);
            if (m) {
                unsigned long long at = 0;
                if (lane == (int)__builtin_ctzll(m))
                    at = atomicAdd(a.ext_count, (unsigned long long)__builtin_popcountll(m));
                at = (unsigned long long)readlane_u64((uint64_t)at, (int)__builtin_ctzll(m));
                if (down)
                    a.ext_list[at + __builtin_popcountll(m & ((1ull << lane) - 1))] = (uint32_t)r;
            }
        }
    }
}

// Requests whose depth-K prefix is extended walk down the tree: both chains
// 64 blocks at a time from the start; K_r is the first depth d > K whose
// prefix (f1 key of block d - 1) is not extended, or the full-block count.
// The ring keys become the depth-K_r keys.
template <int B>
__global__ __launch_bounds__(kHashThreads) void extend_kernel(HashArgs a)
{
    const int lane = lane_id();
    const uint64_t gw = wave_index();
    const uint64_t nw = ((uint64_t)gridDim.x * blockDim.x) >> 6;
    const HashParams* hp = a.hp;
    const uint64_t seed1 = hp->seed[0], seed2 = hp->seed[1];
    const uint64_t q1 = hp->qpow[0][lane], p1 = hp->ppow[0][lane];
    const uint64_t q2 = hp->qpow[1][lane], p2 = hp->ppow[1][lane];
    uint32_t k1[B], k2[B];
#pragma unroll
    for (int t = 0; t < B; t++) {
        k1[t] = hp->kk[0][t];
        k2[t] = hp->kk[1][t];
    }
    const uint64_t K = a.key_blocks;
    const uint64_t units = *a.ext_count_in;
    for (uint64_t u = gw; u < units; u += nw) {
        const uint32_t r = a.ext_list[u];
        const int64_t o0 = a.offsets[r];
        const uint64_t nfull = (uint64_t)(a.offsets[(uint64_t)r + 1] - o0) / B;
        const int32_t* tp = a.tokens + o0;
        uint64_t G1 = hp->H0[0], G2 = hp->H0[1];
        uint64_t kr = nfull, x1 = 0, x2 = 0;
        for (uint64_t cb = 0; cb < nfull; cb += kWave) {
            const uint64_t b = cb + lane, d = b + 1;
            const bool valid = b < nfull;
            uint64_t nh1 = 0, nh2 = 0;
            if (valid)
                nh_block2<B>(tp + b * B, k1, k2, nh1, nh2);
            const uint64_t H1 = (G1 + wave_incl_sum_u64(nh1 * q1, lane)) * p1;
            const uint64_t H2 = (G2 + wave_incl_sum_u64(nh2 * q2, lane)) * p2;
            G1 = readlane_u64(H1, kWave - 1);
            G2 = readlane_u64(H2, kWave - 1);
            const uint64_t h1 = mix64(H1 ^ seed1);
            // the path ends at the first depth past K that is not extended
            const bool below = valid && d > K;
            const uint64_t stop =
                ballot(below && (d == nfull || !table_has(a.kl_tab, a.kl_log2, canon_key(h1))));
            if (stop) {
                const int f = __builtin_ctzll(stop);
                kr = cb + f + 1;
                x1 = readlane_u64(h1, f);
                x2 = readlane_u64(mix64(H2 ^ seed2), f);
                break;
            }
        }
        if (lane == 0) {
            a.key_out[r] = x1;
            a.key_out[a.n + r] = x2;
            if (a.key_len)
                a.key_len[r] = (uint32_t)kr;
        }
    }
}

// Walk of whole chains with probes from the chain's chunks (leaders, and
// the rare requests whose pending probes ran past the keys the members pass
// kept): the full f1 chain, each chunk's keys probed against the
// candidates still unresolved, from each one's start block.
//   kLeaders  unit g: group g's leader, both candidates from block 0, keys
//             stored (members compare with them), until both are resolved;
//   kResume   unit i: entry i of the resume list, one candidate from its
//             start block, nothing stored.
template <int B, int MODE>
__global__ __launch_bounds__(kHashThreads) void walk_kernel(HashArgs a)
{
    const int lane = lane_id();
    const uint64_t gw = wave_index();
    const uint64_t nw = ((uint64_t)gridDim.x * blockDim.x) >> 6;
    const HashParams* hp = a.hp;
    const uint64_t seed1 = hp->seed[0];
    const uint64_t H01 = hp->H0[0];
    const uint64_t q1 = hp->qpow[0][lane], p1 = hp->ppow[0][lane];
    // Malformed offsets (reported by the block-start scan): no full block
    // anywhere.  No store precedes the parameter loads, so they stay scalar.
    const bool bad = *a.bad != 0;
    uint32_t k1[B];
#pragma unroll
    for (int j = 0; j < B; j++)
        k1[j] = hp->kk[0][j];
    const uint32_t ls = a.log2slots;
    const uint64_t units = MODE == kLeaders ? *a.gv.groups : *a.resume_count;
    for (uint64_t u = gw; u < units; u += nw) {
        uint32_t r;
        bool pend0 = true, pend1 = true;
        uint64_t pb0 = 0, pb1 = 0;
        if (MODE == kLeaders) {
            r = a.gv.leader[u];
        } else {
            const uint64_t e = a.resume[u];
            r = (uint32_t)e;
            const bool side1 = (e >> 32) & 1;
            pend0 = !side1;
            pend1 = side1;
            pb0 = pb1 = e >> 33;
        }
        const int64_t o0 = a.offsets[r], o1 = a.offsets[(uint64_t)r + 1];
        uint64_t nfull = bad ? 0 : (uint64_t)(o1 - o0) / B;
        if (nfull > 0xFFFFFFFFull) {
            // match lengths are 32-bit
            if (lane == 0)
                atomicOr(a.status, kErrInval);
            nfull = 0;
        }
        const int32_t* tp = a.tokens + o0;
        const uint64_t* t0 = a.tables + ((uint64_t)a.cand[r] << ls);
        const uint64_t* t1 = a.tables + ((uint64_t)a.cand[a.n + r] << ls);
        uint64_t* hk = a.hkeys + a.bstart[r];
        // a candidate still probing at the end has every block present
        pend0 = pend0 && pb0 < nfull;
        pend1 = pend1 && pb1 < nfull;
        uint64_t m0 = nfull, m1 = nfull;
        uint64_t G = H01;
        for (uint64_t cb = 0; cb < nfull; cb += kWave) {
            const uint64_t b = cb + lane;
            const bool valid = b < nfull;
            const uint64_t nh1 = valid ? nh_block<B>(tp + b * B, k1) : 0;
            const uint64_t S = wave_incl_sum_u64(nh1 * q1, lane);
            const uint64_t H = (G + S) * p1;
            const uint64_t h = mix64(H ^ seed1);
            if (MODE == kLeaders && valid)
                hk[b] = h;
            G = readlane_u64(H, kWave - 1);
            const uint64_t hi = nfull < cb + kWave ? nfull : cb + kWave;
            const uint64_t ck = canon_key(h);
            uint64_t f = 0;
            if (pend0 && pb0 < hi) {
                if (chunk_first_absent(t0, ls, ck, cb, pb0, hi, lane, &f)) {
                    m0 = f;
                    pend0 = false;
                } else {
                    pb0 = hi;
                }
            }
            if (pend1 && pb1 < hi) {
                if (chunk_first_absent(t1, ls, ck, cb, pb1, hi, lane, &f)) {
                    m1 = f;
                    pend1 = false;
                } else {
                    pb1 = hi;
                }
            }
            // Both candidates resolved: a resumed walk is done; a leader's
            // keys are stored up to here, past one block beyond its longer
            // match (as far as its members compare), and the members pass
            // hashes the rest of its prompt.
            if (!pend0 && !pend1)
                break;
        }
        if (lane == 0) {
            if (MODE == kLeaders) {
                a.match[r] = (uint32_t)m0;
                a.match[a.n + r] = (uint32_t)m1;
            } else if ((a.resume[u] >> 32) & 1) {
                a.match[a.n + r] = (uint32_t)m1;
            } else {
                a.match[r] = (uint32_t)m0;
            }
        }
    }
}

// Per-request record of the members pass (48 bytes, read with one scalar
// load): where the prompt and its keys are, the leader's keys, how far to
// compare and the leader's matches.  lim == kLeaderMark marks a leader.
struct alignas(16) MemberRec {
    int64_t o0;          // prompt start
    uint64_t bs;         // own block keys (when stored)
    uint64_t bs_lead;    // the leader's block keys
    uint32_t nfull;      // full blocks
    uint32_t lim;        // blocks compared with the leader
    uint32_t m_lead[2];  // the leader's matches
    uint32_t pad[2];
};
constexpr uint32_t kLeaderMark = 0xFFFFFFFFu;

__global__ void member_record_kernel(const int64_t* __restrict__ offsets, uint64_t n,
                                     uint32_t bshift, const uint64_t* __restrict__ bstart,
                                     const uint32_t* bad_p, GroupView gv,
                                     const uint32_t* __restrict__ cand,
                                     const uint32_t* __restrict__ match,
                                     MemberRec* __restrict__ rec,
                                     unsigned long long* __restrict__ resume_count)
{
    const bool bad = *bad_p != 0;
    if (blockIdx.x == 0 && threadIdx.x == 0)
        *resume_count = 0;
    for (uint64_t r = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; r < n;
         r += (uint64_t)gridDim.x * blockDim.x) {
        const uint32_t L = gv.leader[gv.group_of[r]];
        MemberRec m{};
        m.o0 = offsets[r];
        m.bs = bstart[r];
        uint64_t nr = bad ? 0 : (uint64_t)(offsets[r + 1] - m.o0) >> bshift;
        nr = nr > 0xFFFFFFFFull ? 0 : nr;  // reported by the leaders' walk kernel if a leader
        m.nfull = (uint32_t)nr;
        if (L == r) {
            m.lim = kLeaderMark;
        } else {
            uint64_t nl = bad ? 0 : (uint64_t)(offsets[(uint64_t)L + 1] - offsets[L]) >> bshift;
            nl = nl > 0xFFFFFFFFull ? 0 : nl;
            m.bs_lead = bstart[L];
            m.m_lead[0] = match[L];
            m.m_lead[1] = match[n + L];
            const uint64_t M = m.m_lead[0] > m.m_lead[1] ? m.m_lead[0] : m.m_lead[1];
            uint64_t lim = M + 1 < nr ? M + 1 : nr;
            lim = lim < nl ? lim : nl;
            // the leader's matches are on its candidates: a request whose
            // candidates differ (only on a ring-key collision) is probed on
            // its own from block 0
            if (cand[r] != cand[L] || cand[n + r] != cand[n + L])
                lim = 0;
            m.lim = (uint32_t)lim;
        }
        rec[r] = m;
    }
}

// Tokens of one chunk, lane l holding block l's B tokens as B/4 16-byte
// words (loaded a chunk ahead of their use by the members pass).
template <int B>
struct ChunkTokens {
    v4i t[B / 4];
};

template <int B>
__device__ __forceinline__ void load_chunk(ChunkTokens<B>& c, const int32_t* tp, uint64_t b,
                                           bool valid)
{
#pragma unroll
    for (int j = 0; j < B / 4; j++)
        c.t[j] = valid ? *reinterpret_cast<const v4i*>(tp + b * B + 4 * j) : v4i{0, 0, 0, 0};
}

// NH of a block held in registers, with key words kk.
template <int B>
__device__ __forceinline__ uint64_t nh_regs(const ChunkTokens<B>& c, const uint32_t* kk)
{
    uint64_t acc = 0;
#pragma unroll
    for (int j = 0; j < B / 4; j++) {
        const v4i v = c.t[j];
        acc += (uint64_t)((uint32_t)v.x + kk[4 * j]) * (uint32_t)((uint32_t)v.y + kk[4 * j + 1]);
        acc += (uint64_t)((uint32_t)v.z + kk[4 * j + 2]) * (uint32_t)((uint32_t)v.w + kk[4 * j + 3]);
    }
    return acc;
}

// A member record in registers (three 16-byte loads issued together).
struct RecRegs {
    int64_t o0;
    uint64_t bs, bs_lead;
    uint32_t nfull, lim, m_lead0, m_lead1;
};

__device__ __forceinline__ RecRegs load_rec(const MemberRec* rec, uint64_t r)
{
    typedef unsigned int u4 __attribute__((ext_vector_type(4)));
    const u4* p = reinterpret_cast<const u4*>(rec + r);
    const u4 x = p[0], y = p[1], z = p[2];
    RecRegs m;
    m.o0 = (int64_t)(((uint64_t)x.y << 32) | x.x);
    m.bs = ((uint64_t)x.w << 32) | x.z;
    m.bs_lead = ((uint64_t)y.y << 32) | y.x;
    m.nfull = y.z;
    m.lim = y.w;
    m.m_lead0 = z.x;
    m.m_lead1 = z.y;
    return m;
}

// Blocks of a record compared with its leader (none for a leader itself).
__device__ __forceinline__ uint32_t cmp_lim(const RecRegs& m)
{
    return m.lim == kLeaderMark ? 0u : m.lim;
}

// Every request's full f1 chain (stored when the caller asks for block
// keys).  A request that is not a leader is compared chunk by chunk with its
// leader's keys over blocks [0, lim) (one ballot per chunk) to find the
// first disagreement s.  Per candidate, the leader's match where it ends
// before s, the request's length where s reaches it, or pending: the
// request's keys of blocks [s, s + 8) are kept in pkeys (8 per request) and
// pend[r] = s | side mask << 32 for probe_pending_kernel (0 for leaders and
// requests with nothing pending).  Probing is left
// out of this pass: its latency would hold the wave with no tokens in
// flight.
//
// A wave keeps one chunk's loads in flight while it hashes the chunk
// before: the next chunk's tokens and leader keys, or, on a request's last
// chunk, the next request's first chunk (its record is loaded a request
// ahead), when a wave has more than one request.  (Persistent waves claiming
// blocks of requests through per-XCD counters were measured 13% slower.)
template <int B, bool MULTI>
__global__ __launch_bounds__(kHashThreads) void member_kernel(HashArgs a)
{
    const int lane = lane_id();
    const HashParams* hp = a.hp;
    const uint64_t seed1 = hp->seed[0];
    const uint64_t H01 = hp->H0[0];
    const uint64_t q1 = hp->qpow[0][lane], p1 = hp->ppow[0][lane];
    uint32_t k1[B];
#pragma unroll
    for (int j = 0; j < B; j++)
        k1[j] = hp->kk[0][j];
    // requests of this wave: its index, then every grid's worth of waves on
    // (one request per wave unless the batch has more than 4 Mi requests)
    const uint64_t nw = ((uint64_t)gridDim.x * blockDim.x) >> 6;
    uint64_t r = wave_index();
    bool have = r < a.n;
    RecRegs cur{};
    if (have)
        cur = load_rec(a.rec, r);
    // blocks whose f1 digests the prefix pass kept (their tokens are not
    // read again)
    const uint64_t K = a.key_blocks;
    auto kept = [&](uint64_t nfull) -> uint64_t { return a.nh0 ? (nfull < K ? nfull : K) : 0; };
    ChunkTokens<B> nx;
    uint64_t nlk = 0, pnh = 0;
    {
        const uint64_t kp = have ? kept(cur.nfull) : 0;
        const bool v = have && (uint64_t)lane < cur.nfull && (uint64_t)lane >= kp;
        load_chunk<B>(nx, a.tokens + cur.o0, (uint64_t)lane, v);
        nlk = have && (uint32_t)lane < cmp_lim(cur) ? a.hkeys[cur.bs_lead + lane] : 0;
        pnh = (uint64_t)lane < kp ? a.nh0[r * K + lane] : 0;
    }
    while (have) {
        // this request, then the wave's next one and its record
        const uint64_t rc = r, rn = r + nw;
        const bool have_n = MULTI && rn < a.n;  // a grid of one request per wave has none
        RecRegs nxt{};
        if (have_n)
            nxt = load_rec(a.rec, rn);
        const bool lead = cur.lim == kLeaderMark;
        const uint64_t nfull = cur.nfull, lim = cmp_lim(cur), kp = kept(nfull);
        const uint64_t pre = pnh;
        uint64_t pnh_n = 0;
        const int32_t* tp = a.tokens + cur.o0;
        const uint64_t* lk = a.hkeys + cur.bs_lead;
        uint64_t* hk = a.hkeys + cur.bs;
        uint64_t* pk = a.pkeys + rc * kPendKeys;
        bool cmp = lim > 0;
        // s = 0 when there is nothing to compare
        uint64_t s = 0, emit_lo = 0, emit_hi = 0;
        uint32_t mask = 0;  // candidates left to probe
        uint32_t m0 = (uint32_t)nfull, m1 = (uint32_t)nfull;
        auto resolve = [&](uint64_t s_) {
            s = s_;
            if (cur.m_lead0 < s)
                m0 = cur.m_lead0;
            else if (s < nfull)
                mask |= 1;
            if (cur.m_lead1 < s)
                m1 = cur.m_lead1;
            else if (s < nfull)
                mask |= 2;
            emit_lo = s;
            emit_hi = mask ? (s + kPendKeys < nfull ? s + kPendKeys : nfull) : s;
        };
        if (!cmp && !lead)
            resolve(0);
        uint64_t G = H01;
        for (uint64_t cb = 0; cb < nfull; cb += kWave) {
            const uint64_t b = cb + lane;
            const bool valid = b < nfull;
            const ChunkTokens<B> tc = nx;
            const uint64_t lkey = nlk;
            // loads of the following chunk go out before this one is hashed
            const uint64_t b2 = b + kWave;
            if (cb + kWave < nfull) {
                load_chunk<B>(nx, tp, b2, b2 < nfull);
                nlk = cmp && b2 < lim ? lk[b2] : 0;
            } else if (have_n) {
                const uint64_t kn = kept(nxt.nfull);
                load_chunk<B>(nx, a.tokens + nxt.o0, (uint64_t)lane,
                              (uint64_t)lane < nxt.nfull && (uint64_t)lane >= kn);
                nlk = (uint32_t)lane < cmp_lim(nxt) ? a.hkeys[nxt.bs_lead + lane] : 0;
                pnh_n = (uint64_t)lane < kn ? a.nh0[rn * K + lane] : 0;
            }
            const uint64_t nh1 = valid ? (b < kp ? pre : nh_regs<B>(tc, k1)) : 0;
            const uint64_t S = wave_incl_sum_u64(nh1 * q1, lane);
            const uint64_t H = (G + S) * p1;
            const uint64_t h = mix64(H ^ seed1);
            if (a.write_keys && valid)
                hk[b] = h;
            G = readlane_u64(H, kWave - 1);
            if (cmp) {
                const bool in = b < lim;
                const uint64_t diff = ballot(in && lkey != h);
                if (diff) {
                    cmp = false;
                    resolve(cb + (uint64_t)__builtin_ctzll(diff));
                } else if (cb + kWave >= lim) {
                    cmp = false;
                    resolve(lim);
                }
            }
            if (!cmp && b >= emit_lo && b < emit_hi)
                pk[b - emit_lo] = h;
        }
        if (nfull == 0 && have_n) {
            // nothing of the next request was loaded ahead yet
            const uint64_t kn = kept(nxt.nfull);
            load_chunk<B>(nx, a.tokens + nxt.o0, (uint64_t)lane,
                          (uint64_t)lane < nxt.nfull && (uint64_t)lane >= kn);
            nlk = (uint32_t)lane < cmp_lim(nxt) ? a.hkeys[nxt.bs_lead + lane] : 0;
            pnh_n = (uint64_t)lane < kn ? a.nh0[rn * K + lane] : 0;
        }
        if (lane == 0) {
            if (!lead) {
                a.match[rc] = m0;
                a.match[a.n + rc] = m1;
            }
            a.pend[rc] = s | ((uint64_t)mask << 32);  // 0 for a leader
        }
        r = rn;
        cur = nxt;
        pnh = pnh_n;
        have = have_n;
    }
}

// Pending candidates of the members pass, one thread per request: probe
// its kept keys of blocks [s, s + 8) in order up to the first absent one.
// If all are present and blocks remain, the (request, candidate) goes to
// the resume list (walked again from block s + 8 by walk_kernel<kResume>).
__global__ void probe_pending_kernel(uint64_t n, const uint64_t* __restrict__ pend,
                                     const MemberRec* __restrict__ rec,
                                     const uint64_t* __restrict__ pkeys,
                                     const uint32_t* __restrict__ cand,
                                     const uint64_t* __restrict__ tables, uint32_t ls,
                                     uint32_t* __restrict__ match, uint64_t* __restrict__ resume,
                                     unsigned long long* __restrict__ resume_count)
{
    for (uint64_t r = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; r < n;
         r += (uint64_t)gridDim.x * blockDim.x) {
        const uint64_t p = pend[r];  // nothing pending for leaders
        const uint32_t mask = (uint32_t)(p >> 32);
        if (!mask)
            continue;
        const uint64_t s = (uint32_t)p, nfull = rec[r].nfull;
        const uint64_t k_end = s + kPendKeys < nfull ? s + kPendKeys : nfull;
        for (int side = 0; side < 2; side++) {
            if (!(mask & (1u << side)))
                continue;
            const uint64_t* tab = tables + ((uint64_t)cand[side * n + r] << ls);
            uint64_t b = s;
            while (b < k_end && table_has(tab, ls, canon_key(pkeys[r * kPendKeys + (b - s)])))
                b++;
            if (b < k_end || b == nfull) {
                match[side * n + r] = (uint32_t)b;
            } else {
                const unsigned long long at = atomicAdd(resume_count, 1ull);
                resume[at] = (uint64_t)r | ((uint64_t)side << 32) | (b << 33);
            }
        }
    }
}

template <int MODE>
hipError_t launch_walk(dm_ctx* c, const HashArgs& a, uint32_t grid)
{
    switch (c->cfg.block_size) {
        case 4: walk_kernel<4, MODE><<<grid, kHashThreads, 0, c->stream>>>(a); break;
        case 8: walk_kernel<8, MODE><<<grid, kHashThreads, 0, c->stream>>>(a); break;
        case 16: walk_kernel<16, MODE><<<grid, kHashThreads, 0, c->stream>>>(a); break;
        case 32: walk_kernel<32, MODE><<<grid, kHashThreads, 0, c->stream>>>(a); break;
        case 64: walk_kernel<64, MODE><<<grid, kHashThreads, 0, c->stream>>>(a); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <int B>
hipError_t launch_members_b(dm_ctx* c, const HashArgs& a)
{
    // one request per wave (the register-lean form, 8 waves per SIMD) unless
    // the batch outnumbers the grid
    const uint32_t grid = grid_for(a.n, kHashThreads / kWave, kHashBlocks);
    if ((uint64_t)grid * (kHashThreads / kWave) < a.n)
        member_kernel<B, true><<<grid, kHashThreads, 0, c->stream>>>(a);
    else
        member_kernel<B, false><<<grid, kHashThreads, 0, c->stream>>>(a);
    return hipGetLastError();
}

hipError_t launch_members(dm_ctx* c, const HashArgs& a)
{
    switch (c->cfg.block_size) {
        case 4: return launch_members_b<4>(c, a);
        case 8: return launch_members_b<8>(c, a);
        case 16: return launch_members_b<16>(c, a);
        case 32: return launch_members_b<32>(c, a);
        case 64: return launch_members_b<64>(c, a);
        default: return hipErrorInvalidValue;
    }
}

HashArgs base_args(dm_ctx* c, const int32_t* tokens, const int64_t* offsets, uint64_t n,
                   const uint32_t* bad)
{
    HashArgs a{};
    a.tokens = tokens;
    a.offsets = offsets;
    a.n = n;
    a.hp = c->d_hp;
    a.key_blocks = c->cfg.key_blocks;
    a.bad = bad;
    a.tables = c->d_tables;
    a.log2slots = c->cfg.index_log2_slots;
    a.status = c->d_status;
    return a;
}

// Work arrays of the members pass for n requests, in layout order: records,
// kept keys, pending words, the resume list (two entries per request at
// most) and its count.
struct MemberWork {
    MemberRec* rec;
    uint64_t *pkeys, *pend, *resume;
    unsigned long long* resume_count;
};

size_t up256m(size_t x) { return (x + 255) & ~size_t(255); }

size_t member_layout(uint64_t n, uint8_t* w, MemberWork* mw)
{
    const size_t sz[] = {up256m(n * sizeof(MemberRec)), up256m(n * kPendKeys * 8), up256m(8 * n),
                         up256m(16 * n), 256};
    size_t at[5], off = 0;
    for (int i = 0; i < 5; i++) {
        at[i] = off;
        off += sz[i];
    }
    if (mw) {
        mw->rec = reinterpret_cast<MemberRec*>(w + at[0]);
        mw->pkeys = reinterpret_cast<uint64_t*>(w + at[1]);
        mw->pend = reinterpret_cast<uint64_t*>(w + at[2]);
        mw->resume = reinterpret_cast<uint64_t*>(w + at[3]);
        mw->resume_count = reinterpret_cast<unsigned long long*>(w + at[4]);
    }
    return off;
}

}  // namespace

// The tree's fields of HashArgs (kl_on = 0 when the tree is off).
static void tree_args(dm_ctx* c, HashArgs& a)
{
    const KeyLen& k = c->kl;
    a.kl_on = k.on ? 1u : 0u;
    if (!k.on)
        return;
    a.kl_log2 = k.log2;
    a.kl_tab = k.tab[k.cur];
}

hipError_t hash_prefix(dm_ctx* c, const int32_t* tokens, const int64_t* offsets, uint64_t n,
                       const uint32_t* bad, uint64_t* key_out, uint32_t* key_len,
                       uint32_t* ext_list, unsigned long long* ext_count, uint64_t* nh0)
{
    HashArgs a = base_args(c, tokens, offsets, n, bad);
    a.nh0 = nh0;
    a.key_out = key_out;
    a.key_len = key_len;
    tree_args(c, a);
    a.ext_list = ext_list;
    a.ext_count = ext_count;
    uint32_t glog = 0;
    while ((1u << glog) < c->cfg.key_blocks)
        glog++;
    const uint64_t waves = (n + (kWave >> glog) - 1) / (kWave >> glog);
    const uint32_t grid = grid_for(waves, kHashThreads / kWave, kHashBlocks);
    switch (c->cfg.block_size) {
        case 4: ring_key_kernel<4><<<grid, kHashThreads, 0, c->stream>>>(a, glog); break;
        case 8: ring_key_kernel<8><<<grid, kHashThreads, 0, c->stream>>>(a, glog); break;
        case 16: ring_key_kernel<16><<<grid, kHashThreads, 0, c->stream>>>(a, glog); break;
        case 32: ring_key_kernel<32><<<grid, kHashThreads, 0, c->stream>>>(a, glog); break;
        case 64: ring_key_kernel<64><<<grid, kHashThreads, 0, c->stream>>>(a, glog); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t hash_extend(dm_ctx* c, const int32_t* tokens, const int64_t* offsets, uint64_t n,
                       const uint32_t* bad, uint64_t* key_out, uint32_t* key_len,
                       const uint32_t* ext_list, const unsigned long long* ext_count)
{
    HashArgs a = base_args(c, tokens, offsets, n, bad);
    a.key_out = key_out;
    a.key_len = key_len;
    tree_args(c, a);
    a.ext_list = const_cast<uint32_t*>(ext_list);
    a.ext_count_in = ext_count;
    // the listed count is on the device: a bounded grid strides over it
    const uint32_t grid = grid_for(n, kHashThreads / kWave, kLeaderBlocks);
    switch (c->cfg.block_size) {
        case 4: extend_kernel<4><<<grid, kHashThreads, 0, c->stream>>>(a); break;
        case 8: extend_kernel<8><<<grid, kHashThreads, 0, c->stream>>>(a); break;
        case 16: extend_kernel<16><<<grid, kHashThreads, 0, c->stream>>>(a); break;
        case 32: extend_kernel<32><<<grid, kHashThreads, 0, c->stream>>>(a); break;
        case 64: extend_kernel<64><<<grid, kHashThreads, 0, c->stream>>>(a); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t hash_leaders(dm_ctx* c, const int32_t* tokens, const int64_t* offsets, uint64_t n,
                        const uint64_t* bstart, const uint32_t* bad, const GroupView& gv,
                        const uint32_t* cand, uint64_t* hkeys, uint32_t* match)
{
    HashArgs a = base_args(c, tokens, offsets, n, bad);
    a.bstart = bstart;
    a.hkeys = hkeys;
    a.gv = gv;
    a.cand = cand;
    a.match = match;
    // the group count is on the device: a bounded grid strides over it
    return launch_walk<kLeaders>(c, a, grid_for(n, kHashThreads / kWave, kLeaderGrid));
}

uint64_t member_scratch_bytes(uint64_t n) { return member_layout(n, nullptr, nullptr); }

hipError_t hash_members(dm_ctx* c, const int32_t* tokens, const int64_t* offsets, uint64_t n,
                        const uint64_t* bstart, const uint32_t* bad, const GroupView& gv,
                        const uint32_t* cand, uint64_t* hkeys, bool write_keys, uint32_t* match,
                        const uint64_t* nh0)
{
    hipError_t e = hipSuccess;
    uint8_t* w = static_cast<uint8_t*>(scratch_get(c, kSlotMembers, member_scratch_bytes(n), &e));
    if (!w)
        return e;
    MemberWork mw;
    member_layout(n, w, &mw);
    uint32_t bshift = 0;
    while ((1u << bshift) < c->cfg.block_size)
        bshift++;
    member_record_kernel<<<grid_for(n, 256, 8192), 256, 0, c->stream>>>(
        offsets, n, bshift, bstart, bad, gv, cand, match, mw.rec, mw.resume_count);
    HashArgs a = base_args(c, tokens, offsets, n, bad);
    a.bstart = bstart;
    a.hkeys = hkeys;
    a.write_keys = write_keys ? 1u : 0u;
    a.nh0 = const_cast<uint64_t*>(nh0);
    a.gv = gv;
    a.cand = cand;
    a.match = match;
    a.rec = mw.rec;
    a.pkeys = mw.pkeys;
    a.pend = mw.pend;
    a.resume = mw.resume;
    a.resume_count = mw.resume_count;
    if ((e = launch_members(c, a)) != hipSuccess)
        return e;
    probe_pending_kernel<<<grid_for(n, 256, 8192), 256, 0, c->stream>>>(
        n, mw.pend, mw.rec, mw.pkeys, cand, c->d_tables, c->cfg.index_log2_slots, match,
        mw.resume, mw.resume_count);
    // the rare (request, candidate) whose kept keys were all present
    return launch_walk<kResume>(c, a, grid_for(2 * n, kHashThreads / kWave, kLeaderBlocks));
}

}  // namespace dm
