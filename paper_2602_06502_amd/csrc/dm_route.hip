// dm_route_batch: batched dual-mapping routing (Sec. 3.2; Sec. A.1.1).
//
//   block_starts   exclusive sum of full blocks per request: where each
//                  request's block keys go; checks the offsets;
//   hash_prefix    both ring keys from the first min(K, full blocks)
//                  blocks (dm_hash.hip);
//   lookup_group   candidates on the two rings, then requests ordered by
//                  their first ring key and grouped by equal ring keys,
//                  with a leader per group (dm_probe.hip);
//   hash_leaders   leaders' full chains and longest cached prefixes;
//   hash_members   every other request's full chain and longest cached
//                  prefix, from its leader's keys and its own probes;
//   select_*       SLO-aware choice in request order, loads updated
//                  (dm_select.hip).
// With timing on, events between the stages give the per-stage times that
// dm_route_stage_ms reports.  With pipelining on, the batch's work runs on
// the context's work stream (after the caller's stream and after the batch
// two back), its serial selection on the selection stream (after the
// batch's record packing and the previous selection), and the output
// epilogue on the output stream; the next batch's hashing and probing thus
// overlap this batch's selection.
#include "dm_internal.h"

namespace dm {
namespace {

constexpr int kKeySlot = kSlotKeys;  // block keys when the caller keeps none

// Clears the batch's malformed-offsets word (a kernel rather than a memset,
// so that a captured graph replays it like the rest of the batch).
__global__ void route_zero_kernel(uint32_t* bad, unsigned long long* ext_count)
{
    *bad = 0;
    if (ext_count)
        *ext_count = 0;
}

}  // namespace

namespace {

uint32_t block_shift_of(const dm_ctx* c)
{
    uint32_t k = 0;
    while ((1u << k) < c->cfg.block_size)
        k++;
    return k;
}

// Block starts [n + 1] and the malformed-offsets word, 256-byte aligned.
uint64_t starts_bytes(uint64_t n) { return ((n + 2) * sizeof(uint64_t) + 255) & ~255ull; }

// The f1 digests the prefix pass keeps for the members pass: K per request,
// when K is small enough that they cost less than a fraction of the tokens
// they replace (always at K <= 16).
uint64_t nh0_bytes(const dm_ctx* c, uint64_t n)
{
    return c->cfg.key_blocks <= 16 ? n * c->cfg.key_blocks * sizeof(uint64_t) : 0;
}

// Routes launches of the helper stages to another stream for one call.
struct StreamSwap {
    dm_ctx* c;
    hipStream_t saved;
    StreamSwap(dm_ctx* ctx, hipStream_t s) : c(ctx), saved(ctx->stream) { c->stream = s; }
    ~StreamSwap() { c->stream = saved; }
};

}  // namespace

void route_scratch_plan(const dm_ctx* c, uint64_t n, uint64_t n_tokens, bool keys_in_scratch,
                        size_t* bytes)
{
    for (int i = 0; i < kScratchSlots; i++)
        bytes[i] = 0;
    // block starts, malformed-offsets word, the first blocks' f1 digests
    bytes[kSlotStarts] = starts_bytes(n) + nh0_bytes(c, n);
    bytes[kSlotProbe] = probe_scratch_bytes(n);       // request order and groups
    bytes[kSlotMembers] = member_scratch_bytes(n);    // members pass records, kept keys
    bytes[kSlotSelect] = select_scratch_bytes(n);     // one set of selection work arrays
    if (keys_in_scratch)                              // block keys
        bytes[kSlotKeys] = ((n_tokens >> block_shift_of(c)) + 1) * sizeof(uint64_t);
    bytes[kSlotSort] = sort_scratch_bytes(n);         // digit counts of the ordering sort
    const uint64_t s1 = scan_scratch_bytes(n), s2 = scan_scratch_bytes(sort_scan_len(n));
    bytes[kSlotScan] = s1 > s2 ? s1 : s2;             // tile sums of both kinds of scan
    if (c->kl.on)  // requests going down the tree; the window record's offsets
        bytes[kSlotRebalance] = 256 + ((n * sizeof(uint32_t) + 255) & ~255ull) +
                                keylen_record_bytes(n);
}

hipError_t route(dm_ctx* c, const int32_t* tokens, uint64_t n_tokens, const int64_t* offsets,
                 uint64_t n, int64_t* loads, const dm_route_out* out)
{
    hipError_t e = hipSuccess;
    const bool pipe = c->pipelined;
    const int par = pipe ? (int)(c->batches & 1) : 0;
    if (pipe) {
        if ((e = hipEventRecord(c->in_ready, c->stream)) != hipSuccess ||
            (e = hipStreamWaitEvent(c->work_stream, c->in_ready, 0)) != hipSuccess)
            return e;
        // outputs and work arrays two batches back may be this batch's
        if (c->batches >= 2 &&
            (e = hipStreamWaitEvent(c->work_stream, c->out_done[par], 0)) != hipSuccess)
            return e;
    }
    StreamSwap swap(c, pipe ? c->work_stream : c->stream);
    hipStream_t st = c->stream;
    hipEvent_t* ev = nullptr;
    if (c->timing) {
        ev = &c->tev[(c->tcount % dm_ctx::kTimingRing) * 5];
        c->tcount++;
    }
    if (ev && (e = hipEventRecord(ev[0], st)) != hipSuccess)
        return e;
    // block starts [n + 1], then the malformed-offsets word, then the f1
    // digests of every request's first min(K, full blocks) blocks
    uint64_t* bstart = static_cast<uint64_t*>(
        scratch_get(c, kSlotStarts, starts_bytes(n) + nh0_bytes(c, n), &e));
    if (!bstart)
        return e;
    uint32_t* bad = reinterpret_cast<uint32_t*>(bstart + n + 1);
    uint64_t* nh0 = nh0_bytes(c, n) ? reinterpret_cast<uint64_t*>(
                                          reinterpret_cast<uint8_t*>(bstart) + starts_bytes(n))
                                    : nullptr;
    // with the hotness tree: the count (first 256 bytes), then the list of
    // requests going down the tree
    unsigned long long* ext_count = nullptr;
    uint32_t* ext_list = nullptr;
    uint64_t* kl_work = nullptr;
    if (c->kl.on) {
        const uint64_t list_bytes = (n * sizeof(uint32_t) + 255) & ~255ull;
        uint8_t* w = static_cast<uint8_t*>(scratch_get(
            c, kSlotRebalance, 256 + list_bytes + keylen_record_bytes(n), &e));
        if (!w)
            return e;
        ext_count = reinterpret_cast<unsigned long long*>(w);
        ext_list = reinterpret_cast<uint32_t*>(w + 256);
        kl_work = reinterpret_cast<uint64_t*>(w + 256 + list_bytes);
    }
    route_zero_kernel<<<1, 1, 0, st>>>(bad, ext_count);
    if ((e = block_starts(c, offsets, n, n_tokens, bstart, bad)) != hipSuccess)
        return e;
    uint64_t* hkeys = out->block_keys;
    // the hotness tree's window records every request's block keys
    const bool write_keys = out->block_keys != nullptr || c->kl.on;
    if (!hkeys) {
        // Requests that pass the offsets check are disjoint ranges of the
        // token array, so they hold at most n_tokens / B full blocks: the
        // scratch is sized without reading the batch's block count back.
        const uint64_t cap = (n_tokens >> block_shift_of(c)) + 1;
        hkeys = static_cast<uint64_t*>(scratch_get(c, kKeySlot, cap * sizeof(uint64_t), &e));
        if (!hkeys)
            return e;
    }
    if (ev && (e = hipEventRecord(ev[1], st)) != hipSuccess)
        return e;
    GroupView gv{};
    if ((e = hash_prefix(c, tokens, offsets, n, bad, out->key, out->key_len, ext_list,
                         ext_count, nh0)) != hipSuccess)
        return e;
    if (c->kl.on && (e = hash_extend(c, tokens, offsets, n, bad, out->key, out->key_len, ext_list,
                                     ext_count)) != hipSuccess)
        return e;
    if ((e = lookup_group(c, n, out->key, bstart, bad, out->cand, out->flags, &gv)) != hipSuccess)
        return e;
    if (ev && (e = hipEventRecord(ev[2], st)) != hipSuccess)
        return e;
    if ((e = hash_leaders(c, tokens, offsets, n, bstart, bad, gv, out->cand, hkeys, out->match)) !=
            hipSuccess ||
        (e = hash_members(c, tokens, offsets, n, bstart, bad, gv, out->cand, hkeys, write_keys,
                          out->match, nh0)) != hipSuccess)
        return e;
    if (c->kl.on) {
        if ((e = keylen_record(c, n, bstart, hkeys, kl_work)) != hipSuccess)
            return e;
        c->kl.win += n;
    }
    if (ev && (e = hipEventRecord(ev[3], st)) != hipSuccess)
        return e;
    if ((e = select_prepare(c, st, offsets, n, out, par)) != hipSuccess)
        return e;
    if (!pipe) {
        if ((e = select_run(c, st, st, nullptr, offsets, n, out, loads, 0)) != hipSuccess)
            return e;
        return ev ? hipEventRecord(ev[4], st) : hipSuccess;
    }
    if ((e = hipEventRecord(c->prep_done, st)) != hipSuccess ||
        (e = hipStreamWaitEvent(c->sel_stream, c->prep_done, 0)) != hipSuccess)
        return e;
    if ((e = select_run(c, c->sel_stream, c->out_stream, c->sel_done, offsets, n, out, loads,
                        par)) != hipSuccess)
        return e;
    if ((e = hipEventRecord(c->out_done[par], c->out_stream)) != hipSuccess)
        return e;
    c->batches++;
    return ev ? hipEventRecord(ev[4], c->out_stream) : hipSuccess;
}

}  // namespace dm
