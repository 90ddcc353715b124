// dm_route_batch: batched dual-mapping routing (Sec. 3.2; Sec. A.1.1).
//
//   block_starts   exclusive sum of full blocks per request: where each
//                  request's block keys live;
//   hash_blocks    chained block keys and both ring keys (dm_hash.hip);
//   lookup_probe   candidates on the two rings and the longest cached prefix
//                  on each (dm_probe.hip);
//   select_batch   SLO-aware choice in request order, loads updated
//                  (dm_select.hip).
// With timing on, events between the stages give the per-stage times that
// dm_route_stage_ms reports.  With pipelining on, the selection stage runs
// on the context's selection stream: it waits for this batch's probe stage
// (an event) and, being on one stream, for the previous batch's selection,
// so the next batch's hashing and probing overlap it.
#include "dm_internal.h"

namespace dm {
namespace {

constexpr int kKeySlot = 4;  // block keys when the caller keeps none

}  // namespace

hipError_t route(dm_ctx* c, const int32_t* tokens, const int64_t* offsets, uint64_t n,
                 int64_t* loads, const dm_route_out* out)
{
    hipError_t e = hipSuccess;
    hipStream_t st = c->stream;
    hipStream_t ss = c->pipelined ? c->sel_stream : st;
    hipEvent_t* ev = nullptr;
    if (c->timing) {
        ev = &c->tev[(c->tcount % dm_ctx::kTimingRing) * 5];
        c->tcount++;
    }
    if (ev && (e = hipEventRecord(ev[0], st)) != hipSuccess)
        return e;
    uint64_t* bstart = static_cast<uint64_t*>(scratch_get(c, 0, (n + 1) * sizeof(uint64_t), &e));
    if (!bstart)
        return e;
    if ((e = block_starts(c, offsets, n, bstart)) != hipSuccess)
        return e;
    uint64_t* hkeys = out->block_keys;
    if (!hkeys) {
        // block keys go to context scratch sized by the batch's full-block count
        uint64_t total = 0;
        if ((e = hipMemcpyAsync(&total, bstart + n, sizeof(uint64_t), hipMemcpyDeviceToHost, st)) !=
                hipSuccess ||
            (e = hipStreamSynchronize(st)) != hipSuccess)
            return e;
        hkeys = static_cast<uint64_t*>(scratch_get(c, kKeySlot, (total + 1) * sizeof(uint64_t), &e));
        if (!hkeys)
            return e;
    }
    if (ev && (e = hipEventRecord(ev[1], st)) != hipSuccess)
        return e;
    if ((e = hash_blocks(c, tokens, offsets, n, bstart, hkeys, out->key)) != hipSuccess)
        return e;
    if (ev && (e = hipEventRecord(ev[2], st)) != hipSuccess)
        return e;
    if ((e = lookup_probe(c, n, out->key, hkeys, bstart, out->cand, out->match, out->flags)) !=
        hipSuccess)
        return e;
    if (ev && (e = hipEventRecord(ev[3], st)) != hipSuccess)
        return e;
    if (c->pipelined) {
        if ((e = hipEventRecord(c->probe_done, st)) != hipSuccess ||
            (e = hipStreamWaitEvent(ss, c->probe_done, 0)) != hipSuccess)
            return e;
    }
    if ((e = select_batch(c, ss, offsets, n, out, loads)) != hipSuccess)
        return e;
    if (c->pipelined && (e = hipEventRecord(c->sel_done, ss)) != hipSuccess)
        return e;
    if (ev)
        e = hipEventRecord(ev[4], ss);
    return e;
}

}  // namespace dm
