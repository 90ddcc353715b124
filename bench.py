#!/usr/bin/env python3
"""Benchmark of batched dual-mapping routing on one MI355X.

One step = one dm_route_batch over the large workload: 1,048,576 requests
(lognormal lengths, median 1,024 tokens, cap 16,384; 4,096 Zipf(1.1)
shared-prefix templates; vocab 152,000) against 128 instances x 512 virtual
nodes per ring, block 16, each instance index holding 1,048,576 keys in
2^21 slots.  Inputs are resident in HBM before timing; the loads are reset
to the snapshot before every step (a 2 KB device copy inside the step).

Prints one JSON line: requests routed/s, prompt tokens hashed/s, the HBM
roofline of the hash+match stage (algorithmic bytes / the stage's average
device time measured with HIP events on the stream it runs on; the hash
kernel alone as an extra key), the elastic workload's scale, re-route and
rebalance times (after the timed steps), one row per smaller configuration
(tiny, chat, agent: GPU and oracle throughput, parity), and the CPU oracle
timed on the benchmark's own batch.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, 8 TB/s


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def source_hash(files):
    """Hash of kernel sources: a kernel's memory traffic depends on them alone."""
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2602_06502_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


# Sources of the hash+match stage's kernels (block offsets, hashing, ring
# lookup, request ordering, probing) and of the hash kernel alone.
STAGE_SOURCES = ("dm_internal.h", "dm_route.hip", "dm_scan.hip", "dm_hash.hip", "dm_probe.hip",
                 "dm_sort.hip")
HASH_SOURCES = ("dm_internal.h", "dm_hash.hip")


def load_traffic(name, files):
    """HBM bytes per launch from rocprofv3 FETCH_SIZE/WRITE_SIZE counters, if
    recorded for the current kernel sources."""
    p = os.path.join(ROOT, "profiles", name)
    if not os.path.exists(p):
        return None
    with open(p) as f:
        d = json.load(f)
    if d.get("source_hash") != source_hash(files):
        return None
    return d.get("bytes_per_launch")


# Integer issue peak of the chip: 256 CUs x 4 SIMDs x 16 lanes at 2.4 GHz
# (one 32-bit integer lane-op per lane per clock); a wave-wide VALU
# instruction occupies a SIMD for 4 clocks.
INT_PEAK_TOPS = 256 * 4 * 16 * 2.4e9 / 1e12
VALU_ISSUE_PEAK = 256 * 4 * 2.4e9 / 4


def load_valu(name, files):
    """VALU instruction counts per launch (rocprofv3 SQ_INSTS_* counters), if
    recorded for the current kernel sources."""
    p = os.path.join(ROOT, "profiles", name)
    if not os.path.exists(p):
        return None
    with open(p) as f:
        d = json.load(f)
    return d if d.get("source_hash") == source_hash(files) else None


def host_cpu():
    """(logical CPUs, model name) of the host."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return os.cpu_count(), model


def algorithmic_bytes(off_np, B, match, cand, n):
    """Algorithmic bytes of the hash kernel and of the whole hash+match stage.

    hash kernel: full-block tokens (4 B each), offsets (n + 1) and the two
    8-byte ring keys per request.  hash+match stage: the same plus the other
    per-request outputs (two candidates, two match lengths, flags) and one
    8-byte slot per index probe the first-miss rule needs (match_c blocks plus
    the missing one, per distinct candidate).  Block keys passed between the
    kernels are intermediates and are not counted."""
    import numpy as np
    lens = np.diff(off_np)
    nfull = np.maximum(lens, 0) // B
    ntok = int((nfull * B).sum())
    m1, m2 = match[:n].astype(np.int64), match[n:].astype(np.int64)
    distinct = cand[:n] != cand[n:]
    probes = int((m1 + (m1 < nfull)).sum() + ((m2 + (m2 < nfull)) * distinct).sum())
    hash_bytes = 4 * ntok + 8 * (n + 1) + 16 * n
    stage_bytes = hash_bytes + 17 * n + 8 * probes
    return hash_bytes, stage_bytes, ntok, probes


def walk_steps(cand, match, n, block=None, lanes=64, run_max=3):
    """Depth steps and windows of the selection walk.  Requests are taken in
    blocks of `block` (request order); inside a block a request's level is
    1 + the larger level of the latest earlier request of the block on
    either candidate, except that a request whose latest earlier request on
    both instances is one request of the same pair with the same
    cache-affine candidate (the one with more cached blocks, c1 on equal
    matches) joins that request's run, at its level, while the run holds
    fewer than `run_max` requests.  A level of more than `lanes` requests is
    cut, runs kept whole, into parts of at most `lanes`; every part is one
    depth step.  Windows take consecutive parts and hold two sets of `lanes`
    lanes, the depths alternating between the sets: a window grows while
    both sets' parts fit and its depth stays within 64."""
    if block is None:  # the library's blocks: 2048 requests from 512 Ki requests on
        block = 2048 if n >= 1 << 19 else 1024
    c1, c2 = cand[:n].tolist(), cand[n:].tolist()
    m1, m2 = match[:n].tolist(), match[n:].tolist()
    steps = windows = 0
    for b0 in range(0, n, block):
        last, lv, head, unit, units = {}, {}, {}, {}, {}
        for i in range(b0, min(n, b0 + block)):
            a, o = (c2[i], c1[i]) if m2[i] > m1[i] else (c1[i], c2[i])
            pa, po = last.get(a), last.get(o)
            run = False
            if pa is not None and pa == po and a != o and unit[head[pa]][0] < run_max:
                pab = (c2[pa], c1[pa]) if m2[pa] > m1[pa] else (c1[pa], c2[pa])
                run = pab == (a, o)
            if run:
                head[i], lv[i] = head[pa], lv[pa]
                unit[head[i]][0] += 1
            else:
                lv[i] = 1 + max(lv[pa] if pa is not None else 0, lv[po] if po is not None else 0)
                head[i] = i
                unit[i] = [1]
                units.setdefault(lv[i], []).append(unit[i])
            last[a] = last[o] = i
        parts = []
        for L in range(1, max(units) + 1):
            part = 0
            for sz in (u[0] for u in units[L]):
                if part + sz > lanes:
                    parts.append(part)
                    part = 0
                part += sz
            parts.append(part)
        steps += len(parts)
        # sums of the window's parts at an even (s0) and an odd (s1)
        # distance from its last depth: appending a part swaps them
        s0 = s1 = dep = 0
        for c in parts:
            if dep and (dep == 64 or c + s1 > lanes):
                windows += 1
                s0 = s1 = dep = 0
            s0, s1, dep = c + s1, s0, dep + 1
        windows += 1
    return steps, windows


def cpu_baseline(wl, st, sample):
    """The oracle as it stands, single-threaded, on the first `sample`
    requests of the benchmark's own batch (same index, same initial loads);
    the whole batch by default."""
    import numpy as np

    import oracle
    import oracle.harness as oh
    oracle.build(force=False)
    log("cpu baseline: building oracle state")
    ost = oh.setup(wl, with_batch=False)
    off = st["offsets_np"][:sample + 1]
    tok = st["tokens_np"][:int(off[-1])]
    log(f"cpu baseline: oracle routes {sample:,} requests")
    t0 = time.perf_counter()
    ost["oracle"].route(tok, off, ost["loads0"])
    dt = time.perf_counter() - t0
    ntok = int(((np.diff(off) // wl.route.block) * wl.route.block).sum())
    ncpu, model = host_cpu()
    what = "the whole batch" if sample == wl.n_req else f"the first {sample:,} requests"
    return {"value": sample / dt, "unit": "requests/s", "cores": 1, "kind": "oracle",
            "sample": f"{what} of the {wl.n_req:,}-request benchmark batch (same index and "
                      f"loads), {dt:.1f} s single-threaded",
            "host_logical_cpus": ncpu, "host_cpu_model": model,
            "tokens_hashed_per_s": ntok / dt}


def queues_of(chosen, cand, match, off, B, S, base):
    """Queues of a routed batch: request r waits on its chosen instance with
    its uncached tokens there, the other candidate and its uncached tokens
    there (records in request order)."""
    import numpy as np
    n = len(chosen)
    lens = np.diff(off).astype(np.int64)
    c1, c2 = cand[:n].astype(np.int64), cand[n:].astype(np.int64)
    u1 = lens - B * match[:n].astype(np.int64)
    u2 = lens - B * match[n:].astype(np.int64)
    first = chosen.astype(np.int64) == c1
    here, other = np.where(first, u1, u2), np.where(first, u2, u1)
    alt = np.where(first, c2, c1)
    order = np.argsort(chosen, kind="stable")
    qoff = np.zeros(S + 1, np.int64)
    np.cumsum(np.bincount(chosen, minlength=S), out=qoff[1:])
    return (qoff, order.astype(np.uint64), here[order].astype(np.uint32),
            alt[order].astype(np.uint32), other[order].astype(np.uint32), base)


def config_rows(reps):
    """Configurations 1-3 at their own shapes, each one batch against its
    warmed state: GPU device time of one unpipelined dm_route_batch (HIP
    events around its stages, median over `reps` after one warm-up), the
    oracle on the same batch (one run, single-threaded), and whether every
    output matched.  The agent row adds a rebalancing pass over the batch's
    queues with four seed-chosen instances stalled to 5x the mean work."""
    import numpy as np
    import torch

    import oracle
    import oracle.harness as oh
    import paper_2602_06502_amd.harness as gh
    import workloads
    oracle.build(force=False)
    rows = {}
    specs = [("tiny", workloads.tiny()), ("chat", workloads.chat()), ("agent", workloads.agent())]
    for name, cfg in specs:
        log("config row:", name)
        if name == "tiny":
            g, o = gh.setup(cfg, device="cuda:0"), oh.setup(cfg)
            rc = cfg.route
        else:
            g, o = gh.setup_warm(cfg, device="cuda:0"), oh.setup_warm(cfg)
            rc = cfg.route
        eng = g["eng"]
        n = len(g["offsets_np"]) - 1
        out = eng.alloc_route_out(n)
        dev_ms = []
        for i in range(reps + 1):  # the first call is a warm-up
            L = gh.to_dev(g["loads0"], eng.device)
            eng.set_timing(True)  # restarts the averages: this call alone
            eng.route_into(g["tokens"], g["offsets"], L, out)
            eng.sync()
            if i > 0:
                dev_ms.append(sum(eng.stage_ms()))
        eng.set_timing(False)
        got = {k: v.cpu().numpy() for k, v in out.items()}
        got["loads"] = L.cpu().numpy()
        t0 = time.perf_counter()
        ref = o["oracle"].route(o["tokens"], o["offsets"], o["loads0"])
        odt = time.perf_counter() - t0
        same = all(np.array_equal(got[k], ref[k][:len(got[k])]) for k in
                   ("key", "cand", "match", "chosen", "ttft", "flags", "loads"))
        ntok = int(((np.diff(g["offsets_np"]) // rc.block) * rc.block).sum())
        ms = float(np.median(dev_ms))
        row = {"requests": n, "full_block_tokens": ntok,
               "gpu": {"ms_per_batch": ms, "requests_per_s": n / (ms * 1e-3),
                       "tokens_hashed_per_s": ntok / (ms * 1e-3)},
               "oracle": {"s": odt, "requests_per_s": n / odt, "tokens_hashed_per_s": ntok / odt,
                          "threads": 1},
               "parity": bool(same)}
        if name == "agent":
            S = rc.max_slots
            base = np.zeros(S, np.int64)
            base[:rc.n_inst] = cfg.mu
            hot = workloads.agent_hot_instances(cfg, 0)
            base[hot] += (cfg.hot_factor - 1) * cfg.mu
            q = queues_of(got["chosen"], got["cand"], got["match"], g["offsets_np"], rc.block, S,
                          base)
            qd = [gh.to_dev(x, eng.device) for x in q]
            rms = []
            for i in range(reps + 1):
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                m = eng.rebalance(*qd)
                eng.sync()
                if i > 0:
                    rms.append(1000.0 * (time.perf_counter() - t0))
            cnt = int(m["count"].cpu()[0])
            t0 = time.perf_counter()
            r = o["oracle"].rebalance(*q)
            ort = time.perf_counter() - t0
            rsame = r["status"] == 0 and r["count"] == cnt and all(
                np.array_equal(m[k].cpu().numpy()[:cnt], r[k]) for k in
                ("rec", "src", "dst", "benefit", "ttft_to")) and np.array_equal(
                m["loads"].cpu().numpy(), r["loads"])
            row["rebalance"] = {"records": int(q[0][-1]), "migrations": cnt,
                                "gpu_ms": float(np.median(rms)), "oracle_ms": 1000.0 * ort,
                                "parity": bool(rsame),
                                "note": "host clock per call; queues of the routed batch, "
                                        "four seed-chosen instances stalled to 5x the mean work"}
            # KV save of the routed batch on the chosen instances, LRU-bounded
            nb = int((np.diff(g["offsets_np"]) // rc.block).sum())
            ob = eng.alloc_route_out(n, nb)
            L = gh.to_dev(g["loads0"], eng.device)
            eng.route_into(g["tokens"], g["offsets"], L, ob)
            eng.sync()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            ga = eng.kv_save(g["offsets"], ob["block_keys"], ob["chosen"], 0, cfg.lru_blocks)
            kv_ms = 1000.0 * (time.perf_counter() - t0)
            bk = ob["block_keys"].cpu().numpy()[:nb]
            t0 = time.perf_counter()
            orc, oa, orm = o["oracle"].kv_save(o["offsets"], bk, ob["chosen"].cpu().numpy(), 0,
                                                cfg.lru_blocks)
            kv_ort = time.perf_counter() - t0
            row["kv_save"] = {"blocks": nb, "added": ga[0], "removed": ga[1],
                              "gpu_ms": kv_ms, "oracle_ms": 1000.0 * kv_ort,
                              "parity": bool(orc == 0 and (oa, orm) == ga),
                              "note": "host clock of one dm_kv_save of the routed batch on the "
                                      "chosen instances, LRU bound 200,000 blocks per instance"}
            row["queue_ops"] = queue_ops_row(eng, o["oracle"], g, ob, n, nb, base, cfg)
        rows[name] = row
        del eng, g, o, out
        torch.cuda.empty_cache()
    return rows


def queue_ops_row(eng, orc, g, ob, n, nb, base, cfg):
    """The agent batch's serving state kept on the device: the routed batch
    appended to queues over the stalled base work, re-priced against the
    caches after its KV save, a rebalancing pass over those queues, its
    migration list applied, then 2 ms of service.  Host clock of the second
    of two identical calls (each synchronises), the oracle's beside it,
    and whether the queues matched after every step."""
    import numpy as np
    import torch

    import paper_2602_06502_amd.harness as gh
    d = lambda a: gh.to_dev(a, eng.device)
    S = len(base)
    cpu = {k: v.cpu().numpy() for k, v in ob.items()}
    offs = g["offsets_np"]
    lens = np.diff(offs)
    coff = np.zeros(n + 1, np.int64)
    coff[1:] = np.cumsum(lens // cfg.route.block)
    bk = cpu["block_keys"][:nb]
    empty = (np.zeros(S + 1, np.int64), np.zeros(0, np.uint64), np.zeros(0, np.uint32),
             np.zeros(0, np.uint32), np.zeros(0, np.uint32), base)
    res, same = {}, True

    def step(name, fg, fo):
        nonlocal same
        fg()  # warm-up: the library's scratch grows once
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        qg = fg()
        t1 = time.perf_counter()
        qo = fo()
        t2 = time.perf_counter()
        ok = all(np.array_equal(a.cpu().numpy(), b) for a, b in zip(qg, qo))
        same = same and ok
        res[name] = {"gpu_ms": 1000.0 * (t1 - t0), "oracle_ms": 1000.0 * (t2 - t1),
                     "records": int(qo[0][-1]), "parity": bool(ok)}
        return qg, qo

    qg, qo = step("append", lambda: eng.queue_append(tuple(d(x) for x in empty), g["offsets"], ob, 0),
                  lambda: orc.queue_append(empty, offs, cpu["cand"], cpu["match"], cpu["chosen"], 0))
    dco, dpl = d(coff), d(lens.astype(np.int64))
    qg, qo = step("reprobe", lambda: eng.queue_reprobe(qg, dco, ob["block_keys"][:nb], dpl),
                  lambda: orc.queue_reprobe(qo, coff, bk, lens))
    m = eng.rebalance(*qg)
    eng.sync()
    cnt = int(m["count"].cpu()[0])
    mr, ms_, md = m["rec"][:cnt], m["src"][:cnt], m["dst"][:cnt]
    qg, qo = step("migrate", lambda: eng.queue_migrate(qg, mr, ms_, md),
                  lambda: orc.queue_migrate(qo, mr.cpu().numpy(), ms_.cpu().numpy(),
                                            md.cpu().numpy()))
    units = np.zeros(S, np.int64)
    units[:cfg.route.n_inst] = int(cfg.drain_per_us * 2000)
    qg, qo = step("drain", lambda: eng.queue_drain(qg, d(units)),
                  lambda: orc.queue_drain(qo, units))
    res["migrations"] = cnt
    res["parity"] = bool(same)
    res["note"] = ("host clock per call; queues of the routed batch over the stalled base work, "
                   "re-priced after the batch's KV save, the rebalancing pass's migrations "
                   "applied, 2 ms of service drained")
    return res


def policy_rows(eng, wl, st, L0):
    """The ablation study's selection rules (Sec. 4.3) on the large batch:
    one unpipelined route per rule from the same initial loads; cache hit
    rate (cached prompt tokens of the chosen instances over all prompt
    tokens) and the coefficient of variation of the instances' queued work
    afterwards (Sec. 2.2)."""
    import numpy as np
    import torch
    n = wl.n_req
    lens = np.diff(st["offsets_np"])
    rows = {}
    for pol in ("slo_aware", "cache_affinity", "least_loaded", "min_ttft"):
        eng.set_policy(pol)
        L = L0.clone()
        o = eng.alloc_route_out(n)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        eng.route_into(st["tokens"], st["offsets"], L, o)
        eng.sync()
        ms = 1000.0 * (time.perf_counter() - t0)
        ch = o["chosen"].cpu().numpy()
        cand = o["cand"].cpu().numpy()
        match = o["match"].cpu().numpy()
        m = np.where(ch == cand[:n], match[:n], match[n:]).astype(np.int64)
        fin = L.cpu().numpy()[:wl.route.n_inst].astype(np.float64)
        rows[pol] = {"hit_rate": float((m * wl.route.block).sum() / lens.sum()),
                     "final_load_cv": float(fin.std() / fin.mean()),
                     "fewer_blocks_frac": float((o["flags"].cpu().numpy() & 1).mean()),
                     "ms": ms}
    eng.set_policy("slo_aware")
    rows["note"] = ("one unpipelined dm_route_batch per rule from the same loads and index; "
                    "hit_rate: cached prompt tokens on the chosen instances / prompt tokens; "
                    "final_load_cv: std / mean of the live instances' queued work after the "
                    "batch; fewer_blocks_frac: requests sent to the candidate with fewer cached "
                    "blocks; min_ttft takes the serial selection path; ms: host wall time of "
                    "the call and its sync")
    return rows


def adaptive_leg(eng, wl, st, L0, base_out, base_loads, reps=3):
    """Adaptive hash-key length (Sec. 3.2) on the large batch: each route of
    the batch is one window of the prefix hotness tree, closed after it,
    until the tree stops changing; then the batch is routed with the settled
    tree.  Reported against the fixed-K route of the timed steps: key-length
    spread, the hottest candidate pair's share of requests, the selection
    walk's depth steps, cache hit rate, load CV and times."""
    import numpy as np
    import torch
    n = wl.n_req
    lens = np.diff(st["offsets_np"])

    def stats(o, L):
        ch = o["chosen"].cpu().numpy()
        cand = o["cand"].cpu().numpy()
        match = o["match"].cpu().numpy()
        lo, hi = np.minimum(cand[:n], cand[n:]), np.maximum(cand[:n], cand[n:])
        _, cnt = np.unique(lo.astype(np.int64) * 65536 + hi, return_counts=True)
        m = np.where(ch == cand[:n], match[:n], match[n:]).astype(np.int64)
        fin = L.cpu().numpy()[:wl.route.n_inst].astype(np.float64)
        steps, windows = walk_steps(cand, match, n)
        return {"hottest_pair_share": float(cnt.max() / n), "pairs": int(len(cnt)),
                "select_depth_steps": steps, "select_windows": windows,
                "hit_rate": float((m * wl.route.block).sum() / lens.sum()),
                "final_load_cv": float(fin.std() / fin.mean())}

    base = stats(base_out, base_loads)
    eng.keylen_enable(1 << 16, 1 << 28)
    sizes, close_ms = [], []
    o = eng.alloc_route_out(n, key_len=True)
    for w in range(6):
        L = L0.clone()
        eng.route_into(st["tokens"], st["offsets"], L, o)
        eng.sync()
        t0 = time.perf_counter()
        eng.keylen_window()
        close_ms.append(1000.0 * (time.perf_counter() - t0))
        sizes.append(int(len(eng.keylen_tree())))
        if len(sizes) >= 2 and sizes[-1] == sizes[-2]:
            break
    route_ms = []
    for _ in range(reps):
        L = L0.clone()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        eng.route_into(st["tokens"], st["offsets"], L, o)
        eng.sync()
        route_ms.append(1000.0 * (time.perf_counter() - t0))
        eng.keylen_window()  # each route its own window (the tree has settled)
    kl = o["key_len"].cpu().numpy()[:n]
    ad = stats(o, L)
    eng.keylen_enable(0)
    K = wl.route.key_blocks
    return {"windows_to_settle": len(sizes), "tree_sizes": sizes,
            "key_len": {"K": K, "frac_above_K": float((kl > K).mean()),
                        "p50": float(np.percentile(kl, 50)), "p99": float(np.percentile(kl, 99)),
                        "max": int(kl.max())},
            "fixed_K": base, "adaptive": ad,
            "route_ms": float(np.median(route_ms)), "window_close_ms": float(np.median(close_ms)),
            "note": "each window is one route of the whole batch from the same loads, closed "
                    "after it; route_ms: unpipelined dm_route_batch with the settled tree (the "
                    "window record of every prefix of depth >= K included), host wall clock; "
                    "window_close_ms: dm_keylen_window (sort and count of the record, tree "
                    "rebuild); fixed_K: the timed steps' route"}


def elastic_leg(eng, wl, st, keys, L0, reps):
    """Rows a8/a9 at full size, timed on the host clock around each call (both
    entry points synchronise with the engine's stream before they return):
    dm_scale adds 16 instances and removes 8 (both rings rebuilt, owners of
    2 x n ring keys before and after), one dm_route_batch of the whole batch
    on the scaled cluster, then dm_rebalance over 8 overloaded sources x
    32,768 queued records.  Each scale is undone by the reverse scale before
    the next repetition; the leg ends on the scaled cluster."""
    import numpy as np
    import torch

    import paper_2602_06502_amd.harness as gh
    import workloads

    add, rm = workloads.scale_sets(wl, 16, 8)
    fwd_ms, back_ms = [], []
    for i in range(reps + 1):
        for d, (a, r) in enumerate(((add, rm), (rm, add))):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            res = eng.scale(a.tolist(), r.tolist(), keys)
            eng.sync()
            ms = 1000.0 * (time.perf_counter() - t0)
            if int(res["violations"].cpu()[0]) != 0:
                raise RuntimeError("dm_scale reported keys remapped between unchanged instances")
            if i > 0:
                (fwd_ms if d == 0 else back_ms).append(ms)
    moved = eng.scale(add.tolist(), rm.tolist(), keys)["moved"].cpu().numpy()
    eng.sync()
    n = keys.numel() // 2
    eng.set_pipelining(False)
    route_ms = []
    out = eng.alloc_route_out(n)
    for i in range(reps + 1):
        loads = L0.clone()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        eng.route_into(st["tokens"], st["offsets"], loads, out)
        eng.sync()
        if i > 0:
            route_ms.append(1000.0 * (time.perf_counter() - t0))
    if np.isin(out["cand"].cpu().numpy(), rm).any():
        raise RuntimeError("a removed instance was routed to")
    S, n_live = wl.route.max_slots, wl.route.n_inst - len(rm) + len(add)
    sources = np.sort(np.random.default_rng(3).choice(n_live, size=8, replace=False))
    q = workloads.synthetic_queues(105, S, n_live, sources, 32_768, 2_000, 50_000,
                                   4 * (wl.route.slo_us - 50_000))
    dev = eng.device
    qd = [gh.to_dev(x, dev) for x in (q.qoff, q.rec_id, q.unc_here, q.alt, q.unc_alt, q.base_work)]
    reb_ms, count = [], 0
    for i in range(2 * reps + 2):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        m = eng.rebalance(*qd)
        eng.sync()
        if i > 1:
            reb_ms.append(1000.0 * (time.perf_counter() - t0))
        count = int(m["count"].cpu()[0])
    med = lambda x: float(np.median(x))
    queue_ops = elastic_queue_ops(eng, wl, st, out, qd, m, count)
    return {
        "queue_ops": queue_ops,
        "workload": f"elastic: large state, add ids {int(add[0])}..{int(add[-1])}, remove 8 "
                    f"seeded ids ({n:,} x 2 ring keys); re-route {n:,} requests on "
                    f"{n_live} instances; rebalance {len(q.rec_id):,} records queued on 8 "
                    "overloaded instances",
        "scale_ms": {"median": med(fwd_ms), "min": min(fwd_ms), "reverse_median": med(back_ms),
                     "moved_frac": [float(x) / n for x in moved]},
        "reroute_ms": {"median": med(route_ms), "min": min(route_ms),
                       "requests_per_s": n / (med(route_ms) * 1e-3), "pipelined": False},
        "rebalance_ms": {"median": med(reb_ms), "min": min(reb_ms), "migrations": count,
                         "records": len(q.rec_id)},
        "note": "host wall clock per call, repetitions after one warm-up; the paper reports "
                "2.2-2.5 ms per rebalancing pass on its own machine (context, not a target)",
    }


def elastic_queue_ops(eng, wl, st, out, qd, m, count):
    """The queue operations at the elastic workload's scale: the re-routed
    batch (1,048,576 requests) appended to empty queues, the rebalancing
    pass's migration list applied to its 262,144 queued records, then one
    round of service drained.  Host clock of the second of two identical
    calls (each synchronises), the oracle's operation on the same input
    beside it (one run, single-threaded), and whether the queues matched."""
    import numpy as np
    import torch

    import oracle
    import paper_2602_06502_amd.harness as gh
    o = oracle.Oracle(wl.route.as_dict())
    S = wl.route.max_slots
    d = lambda a: gh.to_dev(a, eng.device)
    res, same = {}, True

    def step(name, fg, fo):
        nonlocal same
        fg()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        g = fg()
        t1 = time.perf_counter()
        r = fo()
        t2 = time.perf_counter()
        ok = all(np.array_equal(a.cpu().numpy(), b) for a, b in zip(g, r))
        same = same and ok
        res[name] = {"gpu_ms": 1000.0 * (t1 - t0), "oracle_ms": 1000.0 * (t2 - t1),
                     "records": int(r[0][-1]), "parity": bool(ok)}
        return g, r

    offs = st["offsets_np"]
    n = len(offs) - 1
    cpu = {k: out[k].cpu().numpy() for k in ("cand", "match", "chosen")}
    empty = (np.zeros(S + 1, np.int64), np.zeros(0, np.uint64), np.zeros(0, np.uint32),
             np.zeros(0, np.uint32), np.zeros(0, np.uint32), np.zeros(S, np.int64))
    step("append", lambda: eng.queue_append(tuple(d(x) for x in empty), st["offsets"], out, 0),
         lambda: o.queue_append(empty, offs, cpu["cand"], cpu["match"], cpu["chosen"], 0))
    qh = tuple(x.cpu().numpy() for x in qd)
    mr, ms_, md = m["rec"][:count], m["src"][:count], m["dst"][:count]
    qg, qo = step("migrate", lambda: eng.queue_migrate(tuple(qd), mr, ms_, md),
                  lambda: o.queue_migrate(qh, mr.cpu().numpy(), ms_.cpu().numpy(),
                                          md.cpu().numpy()))
    units = np.zeros(S, np.int64)
    units[:wl.route.n_inst] = 4 * 2000
    step("drain", lambda: eng.queue_drain(qg, d(units)), lambda: o.queue_drain(qo, units))
    res["parity"] = bool(same)
    res["note"] = ("host clock per call; append: the re-routed batch into empty queues; "
                   "migrate: the rebalancing pass's list on its queues; drain: 8,000 units "
                   "of service per instance")
    return res


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=40)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--n-req", type=int, default=1_048_576)
    ap.add_argument("--cpu-sample", type=int, default=0,
                    help="requests the oracle routes for the CPU baseline (0 = the whole batch)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--config-reps", type=int, default=5)
    ap.add_argument("--no-config-rows", action="store_true",
                    help="skip the tiny / chat / agent rows")
    ap.add_argument("--elastic-reps", type=int, default=5)
    ap.add_argument("--no-elastic", action="store_true",
                    help="skip the scale / re-route / rebalance timings")
    ap.add_argument("--no-adaptive", action="store_true",
                    help="skip the adaptive hash-key length leg")
    ap.add_argument("--no-policies", action="store_true",
                    help="skip the per-rule routes (cache affinity, least loaded, min TTFT)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="after timing, copy 1 GiB device to device once (a plain copy kernel "
                         "of known size, to scale hardware byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the routing path is built and measured on a "
              "single MI355X (see the sharding note in DESIGN.md); run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2602_06502_amd.harness as gh
    import workloads

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    wl = workloads.large(args.n_req)
    log("setup", wl.name, "n_req", wl.n_req)
    t0 = time.perf_counter()
    st = gh.setup(wl, device="cuda:0")
    eng, tokens, offsets = st["eng"], st["tokens"], st["offsets"]
    n = wl.n_req
    log(f"setup done in {time.perf_counter() - t0:.1f} s; tokens {tokens.numel():,}")
    L0 = gh.to_dev(st["loads0"], eng.device)
    # Consecutive batches are pipelined: batch k's selection (one compute
    # unit, in request order) overlaps batch k+1's hashing and probing.
    # Every step routes the same batch from the same load snapshot: each
    # step has its own copy of the initial loads, made before timing, and
    # outputs alternate between two sets.
    n_ref = 3
    loads = [L0.clone() for _ in range(args.warmup + args.steps + n_ref)]
    outs = [eng.alloc_route_out(n), eng.alloc_route_out(n)]
    eng.set_pipelining(True)
    for i in range(args.warmup):
        eng.route_into(tokens, offsets, loads[i], outs[i % 2])
    eng.sync()
    torch.cuda.synchronize()
    eng.set_timing(True)  # stage times averaged over the timed steps
    t0 = time.perf_counter()
    for i in range(args.steps):
        eng.route_into(tokens, offsets, loads[args.warmup + i], outs[i % 2])
    eng.sync()
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    ms_step = 1000.0 * dt / args.steps
    groups_avg, hashm_avg, sel_avg, off_avg = eng.stage_ms()
    out = outs[(args.steps - 1) % 2]
    # the same steps without overlap, for reference
    eng.set_pipelining(False)
    eng.set_timing(True)
    t0 = time.perf_counter()
    for i in range(n_ref):
        eng.route_into(tokens, offsets, loads[args.warmup + args.steps + i], outs[i % 2])
    eng.sync()
    ms_ref = 1000.0 * (time.perf_counter() - t0) / n_ref
    ref_stage = eng.stage_ms()
    if not all(torch.equal(loads[args.warmup + args.steps - 1], x) for x in loads[-n_ref:]):
        raise RuntimeError("pipelined and unpipelined steps ended with different loads")
    match = out["match"].cpu().numpy()
    cand = out["cand"].cpu().numpy()
    hbytes, sbytes, ntok, probes = algorithmic_bytes(st["offsets_np"], wl.route.block, match,
                                                     cand, n)
    achieved = hbytes / (hashm_avg * 1e-3) / 1e9
    stage_gbs = sbytes / ((groups_avg + hashm_avg) * 1e-3) / 1e9
    hash_traffic = load_traffic("traffic_hash_kernel_large.json", HASH_SOURCES)
    valu = load_valu("valu_hash_pass_large.json", HASH_SOURCES)
    stage_traffic = load_traffic("traffic_route_stage_large.json", STAGE_SOURCES)
    final = loads[args.warmup + args.steps - 1].cpu().numpy()[:wl.route.n_inst].astype(np.float64)
    flags = out["flags"].cpu().numpy()
    depth_steps, walk_windows = walk_steps(cand, match, n)
    depth_steps_no_runs, _ = walk_steps(cand, match, n, run_max=1)
    res = {
        "metric": "requests routed/sec and prompt tokens hashed/sec at 1 GPU; % of HBM peak",
        "value": n / (ms_step * 1e-3),
        "unit": "requests/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u64",
        "data": "synthetic",
        "config": {"workload": f"large: {n:,} requests, lognormal lengths (median 1,024, "
                               "sigma 1.0, cap 16,384), 4,096 Zipf(1.1) templates, "
                               "128 instances x 512 vnodes, block 16, K 4, 2^21-slot "
                               "indexes of 1,048,576 keys",
                   "n_req": n, "tokens": int(tokens.numel()), "full_block_tokens": ntok,
                   "instances": wl.route.n_inst, "vnodes": wl.route.vnodes,
                   "block": wl.route.block},
        "tokens_hashed_per_s": ntok / (ms_step * 1e-3),
        "tokens_hashed_per_s_hash_pass": ntok / (hashm_avg * 1e-3),
        "stage_ms": {"keys_groups": groups_avg, "hash_match": hashm_avg, "select": sel_avg,
                     "block_offsets": off_avg,
                     "note": "averaged over the timed steps; keys_groups: prefix hashing, ring "
                             "lookup, ordering and grouping; hash_match: full chains and "
                             "longest cached prefixes of group leaders, then of every other "
                             "request; with pipelining, select runs from the batch's "
                             "hash_match end to its selection end"},
        "pipelined": True,
        "select_bound": {"kernel": "select_fast_kernel", "bound": "latency",
                         "depth_steps": depth_steps, "windows": walk_windows,
                         "depth_steps_without_runs": depth_steps_no_runs,
                         "ns_per_step": ref_stage[2] * 1e6 / depth_steps,
                         "note": "one wave walks windows of up to 2 x 64 requests (one lane "
                                 "set for even depths, one for odd) packed from the "
                                 "dependency levels of 2048-request blocks, runs of up to three "
                                 "same-pair requests sharing a level; each step is an LDS "
                                 "round trip plus the run replay and the decision; time from "
                                 "the unpipelined stage (record packing and levels included)"},
        "unpipelined": {"ms_per_step": ms_ref, "requests_per_s": n / (ms_ref * 1e-3),
                        "steps": n_ref,
                        "stage_ms": {"keys_groups": ref_stage[0], "hash_match": ref_stage[1],
                                     "select": ref_stage[2], "block_offsets": ref_stage[3]}},
        "roofline": {"bound": "hbm",
                     "kernel": "hash+match stage: ring_key_kernel<16>, lookup_kernel, "
                               "radix sort passes, group_head_kernel, "
                               "group scan, group_leader_kernel, "
                               "walk_kernel<16> (leaders, resume), member_record_kernel, "
                               "member_kernel<16>, probe_pending_kernel",
                     "achieved": stage_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": stage_gbs / HBM_PEAK_GBS, "traffic": stage_traffic,
                     "algorithmic_bytes_per_launch": sbytes, "probes": probes,
                     "ms": groups_avg + hashm_avg,
                     "note": "algorithmic bytes of one batch (full-block tokens, offsets, "
                             "per-request outputs, 8 B per index slot the first-miss rule "
                             "inspects) over the stage's device time from HIP events on the "
                             "stream it runs on, averaged over the timed steps"},
        "roofline_hash_match_pass": {"bound": "hbm",
                                     "kernel": "walk_kernel<16> (leaders), "
                                               "member_record_kernel, member_kernel<16>, "
                                               "probe_pending_kernel, walk_kernel<16> (resume)",
                                     "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                     "frac": achieved / HBM_PEAK_GBS, "traffic": hash_traffic,
                                     "algorithmic_bytes_per_launch": hbytes, "ms": hashm_avg},
        "integer_ops": None if valu is None else {
            "kernels": valu["kernels"],
            "int_lane_ops_per_launch": valu["int_lane_ops"],
            "achieved_tops": valu["int_lane_ops"] / (hashm_avg * 1e-3) / 1e12,
            "peak_tops": INT_PEAK_TOPS,
            "frac": valu["int_lane_ops"] / (hashm_avg * 1e-3) / 1e12 / INT_PEAK_TOPS,
            "valu_insts_per_launch": valu["valu_insts"],
            "valu_issue_frac": valu["valu_insts"] / (hashm_avg * 1e-3) / VALU_ISSUE_PEAK,
            "note": "rocprofv3 SQ_INSTS_VALU_INT32 + SQ_INSTS_VALU_INT64 (x 64 lanes) and "
                    "SQ_INSTS_VALU per batch over the hash and match pass "
                    "(profiles/route_large_valu_counters.md), over this run's pass time; "
                    "peak: one 32-bit integer op per lane per clock on 256 CUs x 4 SIMDs x "
                    "16 lanes at 2.4 GHz (64-bit multiplies take several)"},
        "routing_stats": {"slo_switch_frac": float((flags & 1).mean()),
                          "both_over_frac": float(((flags >> 1) & 1).mean()),
                          "hit_blocks_frac": float(
                              np.where(out["chosen"].cpu().numpy() == cand[:n], match[:n],
                                       match[n:]).sum() / max(1, ntok // wl.route.block)),
                          "final_load_cv": float(final.std() / final.mean()),
                          "note": "final_load_cv: coefficient of variation of the instances' "
                                  "queued work after the batch (std / mean over live "
                                  "instances)"},
    }
    if not args.no_policies:
        log("selection rules of the ablation study")
        res["policies"] = policy_rows(eng, wl, st, L0)
    if not args.no_adaptive:
        log("adaptive hash-key length")
        res["adaptive_key_length"] = adaptive_leg(eng, wl, st, L0, out,
                                                  loads[args.warmup + args.steps - 1])
    if not args.no_elastic:
        log("elastic leg: scale, re-route, rebalance")
        res["elastic"] = elastic_leg(eng, wl, st, out["key"], L0, args.elastic_reps)
    if args.calibrate_copy:
        src = torch.ones(1 << 28, dtype=torch.int32, device=eng.device)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        res["calibration_copy_bytes"] = {"read": src.numel() * 4, "write": dst.numel() * 4}
    if not args.no_config_rows:
        log("configuration rows: tiny, chat, agent")
        res["configs"] = config_rows(args.config_reps)
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(wl, st, min(args.cpu_sample or n, n))
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
