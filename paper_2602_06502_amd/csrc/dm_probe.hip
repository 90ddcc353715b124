// Candidates and request groups (Sec. 3.2; Sec. A.1.1).
//
// lookup_kernel: one thread per request finds the owners of its two ring
//   keys and applies the distinct-candidate adjustment (and writes the
//   ordering's sort input).
// Then requests are ordered by the top 16 bits of their first ring key
// (stable radix sort) and grouped: a group is a maximal run of the order
// with equal first ring keys, so its requests have the same first
// candidate and, but for a key collision, the same second one and the same
// first blocks.  Each group's leader is its longest request among its first
// 64; dm_hash.hip probes leaders and resolves every other request against
// its leader's keys.  Grouping is only a matter of speed: any request could
// lead any group and the matches would be the same (a member whose
// candidates differ from its leader's is probed on its own).
#include <algorithm>

#include "dm_internal.h"

namespace dm {
namespace {

constexpr int kOrderBits = 16;  // top bits of the first ring key used for ordering

__global__ void lookup_kernel(uint64_t n, const uint64_t* __restrict__ key, RingView r1,
                              RingView r2, const uint32_t* __restrict__ next_live,
                              uint32_t n_live, uint32_t* __restrict__ cand,
                              uint8_t* __restrict__ flags, uint64_t* __restrict__ skeys,
                              uint32_t* __restrict__ svals)
{
    for (uint64_t r = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; r < n;
         r += (uint64_t)gridDim.x * blockDim.x) {
        const uint64_t x = key[r];
        // the ordering's sort input: the first ring key rotated so that its
        // top kOrderBits bits are the low ones the sort orders by (the sort
        // carries the whole key along), and the request
        skeys[r] = (x << kOrderBits) | (x >> (64 - kOrderBits));
        svals[r] = (uint32_t)r;
        const uint32_t c1 = ring_owner(r1, x);
        uint32_t c2 = ring_owner(r2, key[n + r]);
        uint8_t f = 0;
        if (c2 == c1) {
            f = 8;
            c2 = n_live >= 2 ? next_live[c1] : c1;
        }
        cand[r] = c1;
        cand[n + r] = c2;
        flags[r] = f;
    }
}

// Group heads of the ordered list: position i starts a group when its
// first ring key differs from position i - 1's (the sorted keys are
// compared, no gather).  head[i] is 0 or 1 (u64, for the scan); len[i] is
// the request's full blocks (capped at 2^32 - 1), for the leader choice.
__global__ void group_head_kernel(const uint64_t* __restrict__ skeys,
                                  const uint32_t* __restrict__ order, uint64_t m,
                                  const uint64_t* __restrict__ bstart, const uint32_t* bad_p,
                                  uint64_t* __restrict__ head, uint32_t* __restrict__ len)
{
    const bool bad = *bad_p != 0;
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < m;
         i += (uint64_t)gridDim.x * blockDim.x) {
        head[i] = (i == 0 || skeys[i] != skeys[i - 1]) ? 1 : 0;
        const uint32_t r = order[i];
        const uint64_t l = bad ? 0 : bstart[(uint64_t)r + 1] - bstart[r];
        len[i] = l < 0xFFFFFFFFull ? (uint32_t)l : 0xFFFFFFFFu;
    }
}

// Leader of each group (a head at i leads group gpos[i]): the longest
// request among the group's positions [i, i + 64), ties to the earliest;
// and every request's group (group_of[order[i]]).
// One wave per 64 positions holds positions [64w, 64w + 128), two per lane,
// as (full blocks << 32 | ~position) so that the larger value is the longer
// and then earlier request.  A segmented suffix maximum by doubling over
// both halves (each lane's span doubles six times, to 64 positions, and
// stops at the next head) gives every head lane of the first half its
// leader; positions past the list act as heads.
__global__ __launch_bounds__(256) void group_leader_kernel(const uint32_t* __restrict__ order,
                                                           uint64_t m,
                                                           const uint64_t* __restrict__ head,
                                                           const uint32_t* __restrict__ len,
                                                           const uint64_t* __restrict__ gpos,
                                                           uint32_t* __restrict__ leader,
                                                           uint32_t* __restrict__ group_of)
{
    const int lane = lane_id();
    const uint64_t waves = (m + kWave - 1) / kWave;
    const uint64_t nw = ((uint64_t)gridDim.x * blockDim.x) / kWave;
    for (uint64_t w = ((uint64_t)blockIdx.x * blockDim.x + threadIdx.x) / kWave; w < waves;
         w += nw) {
        const uint64_t i0 = w * kWave + lane, i1 = i0 + kWave;
        const bool h0 = i0 >= m || head[i0] != 0, h1 = i1 >= m || head[i1] != 0;
        uint64_t v0 = i0 < m ? ((uint64_t)len[i0] << 32) | (uint32_t)~(uint32_t)i0 : 0;
        uint64_t v1 = i1 < m ? ((uint64_t)len[i1] << 32) | (uint32_t)~(uint32_t)i1 : 0;
        const uint64_t H0 = ballot(h0), H1 = ballot(h1);
        // done: this lane's span already ends at a head (or the window end)
        bool done0 = lane < kWave - 1 ? (H0 >> (lane + 1)) & 1 : H1 & 1;
        bool done1 = lane < kWave - 1 ? (H1 >> (lane + 1)) & 1 : true;
#pragma unroll
        for (int d = 1; d < kWave; d <<= 1) {
            const int src = (lane + d) & (kWave - 1);
            const bool hi = lane + d >= kWave;  // partner in the second half
            const uint64_t a0 = shfl_u64(v0, src), a1 = shfl_u64(v1, src);
            const uint64_t D0 = ballot(done0), D1 = ballot(done1);
            const uint64_t p0 = hi ? a1 : a0;
            const bool pd0 = hi ? (D1 >> src) & 1 : (D0 >> src) & 1;
            if (!done0) {
                v0 = v0 > p0 ? v0 : p0;
                done0 = pd0;
            }
            if (!done1) {
                if (hi) {
                    done1 = true;
                } else {
                    v1 = v1 > a1 ? v1 : a1;
                    done1 = (D1 >> src) & 1;
                }
            }
        }
        if (i0 < m) {
            // the group of position i0, for its request; a head names the
            // group's leader
            const uint64_t g = gpos[i0] + (h0 ? 1 : 0) - 1;
            group_of[order[i0]] = (uint32_t)g;
            if (h0)
                leader[g] = order[(uint32_t)~(uint32_t)v0];
        }
    }
}


// Work arrays of grouping for m requests, in layout order: sort keys and
// request order (each twice, for the sort's passes), group heads, group
// indices by position, leaders, each request's group, and the group count.
struct GroupWork {
    uint64_t *keys, *ktmp;
    uint32_t *order, *vtmp;
    uint64_t *head, *gpos;
    uint32_t *leader, *group_of, *len;
    uint64_t* groups;
};

size_t up256z(size_t x) { return (x + 255) & ~size_t(255); }

size_t group_layout(uint64_t m, uint8_t* w, GroupWork* gw)
{
    const size_t sz[] = {up256z(8 * m), up256z(8 * m), up256z(4 * m), up256z(4 * m),
                         up256z(8 * m), up256z(8 * m), up256z(4 * m), up256z(4 * m), 256};
    size_t at[9], off = 0;
    for (int i = 0; i < 9; i++) {
        at[i] = off;
        off += sz[i];
    }
    if (gw) {
        gw->keys = reinterpret_cast<uint64_t*>(w + at[0]);
        gw->ktmp = reinterpret_cast<uint64_t*>(w + at[1]);
        gw->order = reinterpret_cast<uint32_t*>(w + at[2]);
        gw->vtmp = reinterpret_cast<uint32_t*>(w + at[3]);
        gw->head = reinterpret_cast<uint64_t*>(w + at[4]);
        gw->gpos = reinterpret_cast<uint64_t*>(w + at[5]);
        gw->leader = reinterpret_cast<uint32_t*>(w + at[6]);
        gw->group_of = reinterpret_cast<uint32_t*>(w + at[7]);
        gw->groups = reinterpret_cast<uint64_t*>(w + at[8]);
    }
    return off;
}

}  // namespace

uint64_t probe_scratch_bytes(uint64_t m) { return group_layout(m, nullptr, nullptr); }

hipError_t lookup_group(dm_ctx* c, uint64_t n, const uint64_t* key, const uint64_t* bstart,
                        const uint32_t* bad, uint32_t* cand, uint8_t* flags, GroupView* gv)
{
    hipError_t e = hipSuccess;
    hipStream_t st = c->stream;
    if (n == 0)
        return hipSuccess;
    if (n > 0xFFFFFFFFull)
        return hipErrorInvalidValue;
    uint8_t* w = static_cast<uint8_t*>(scratch_get(c, kSlotProbe, probe_scratch_bytes(n), &e));
    if (!w)
        return e;
    GroupWork g;
    group_layout(n, w, &g);
    lookup_kernel<<<grid_for(n, 256, 8192), 256, 0, st>>>(
        n, key, view(c->ring[c->cur][0]), view(c->ring[c->cur][1]), c->d_next_live, c->n_live,
        cand, flags, g.keys, g.order);
    g.len = g.vtmp;  // the sort's spare value array is free once it has run
    // requests ordered by the top bits of their first ring key (stable radix sort)
    if ((e = radix_sort_kv(c, g.keys, g.order, g.ktmp, g.vtmp, n, kOrderBits)) != hipSuccess)
        return e;
    group_head_kernel<<<grid_for(n, 256, 8192), 256, 0, st>>>(g.keys, g.order, n, bstart, bad,
                                                              g.head, g.len);
    if ((e = exclusive_scan_u64(c, g.head, n, g.gpos, g.groups)) != hipSuccess)
        return e;
    group_leader_kernel<<<grid_for((n + kWave - 1) / kWave, 256 / kWave, 8192), 256, 0, st>>>(
        g.order, n, g.head, g.len, g.gpos, g.leader, g.group_of);
    *gv = GroupView{g.group_of, g.leader, g.groups};
    return hipGetLastError();
}

}  // namespace dm
