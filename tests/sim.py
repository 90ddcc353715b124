"""Serving-state evolution between routed batches, for the multi-batch parity
tests (chat and agent workloads).

The routing path itself works on a snapshot: the index, the loads and the
queues are inputs.  Between batches a serving system changes them: computed
KV blocks are saved into the chosen instance's cache (bounded, least recently
used blocks evicted), queued work drains, queued requests wait for
rebalancing.  This module keeps that state for ONE side (the oracle or the
engine) and updates it from that side's own outputs, so the two sides evolve
independently and every batch compares them.

Nothing here is the routing method: it is the cache and queue bookkeeping of
the serving system around it.
"""
from __future__ import annotations

from typing import Dict, List, Tuple

import numpy as np


class LRUIndex:
    """Per-instance LRU of cached block keys.  A routed request touches its
    chain deepest block first, so ancestors are always more recent than
    descendants and the cache stays prefix-closed.  The cache of an instance
    is always the `cap` most recently touched distinct keys, so a batch's
    effect is computed at its end."""

    def __init__(self, n_slots: int, cap: int):
        self.cap = cap
        self.keys = [np.zeros(0, np.uint64) for _ in range(n_slots)]
        self.time = [np.zeros(0, np.int64) for _ in range(n_slots)]
        self.clock = 0

    def touch(self, inst_of_req: np.ndarray, block_keys: np.ndarray, nfull: np.ndarray
              ) -> Dict[int, Tuple[np.ndarray, np.ndarray]]:
        """Touch every request's chain on its instance, in request order.
        Returns {instance: (added keys, removed keys)}."""
        nfull = nfull.astype(np.int64)
        total = int(nfull.sum())
        starts = np.concatenate([[0], np.cumsum(nfull)[:-1]]).astype(np.int64)
        b = np.arange(total, dtype=np.int64) - np.repeat(starts, nfull)
        # deepest block first: time grows toward the root
        t = self.clock + np.repeat(starts, nfull) + (np.repeat(nfull, nfull) - 1 - b)
        self.clock += total
        inst = np.repeat(inst_of_req.astype(np.int64), nfull)
        grp = np.argsort(inst, kind="stable")
        ig = inst[grp]
        bounds = np.flatnonzero(np.r_[True, ig[1:] != ig[:-1], True])
        out = {}
        for lo, hi in zip(bounds[:-1], bounds[1:]):
            c = int(ig[lo])
            sel = grp[lo:hi]
            k = np.concatenate([self.keys[c], block_keys[sel]])
            tt = np.concatenate([self.time[c], t[sel]])
            # latest touch per key
            order = np.lexsort((-tt, k))
            ks, ts = k[order], tt[order]
            first = np.r_[True, ks[1:] != ks[:-1]]
            ks, ts = ks[first], ts[first]
            if len(ks) > self.cap:
                keep = np.argpartition(-ts, self.cap - 1)[: self.cap]
                ks, ts = ks[keep], ts[keep]
            added = np.setdiff1d(ks, self.keys[c], assume_unique=False)
            removed = np.setdiff1d(self.keys[c], ks, assume_unique=False)
            self.keys[c], self.time[c] = ks, ts
            out[int(c)] = (added.astype(np.uint64), removed.astype(np.uint64))
        return out


class QueueState:
    """Per-instance FIFO queues of routed requests plus base work.  A record
    is (request id, uncached tokens here, the other candidate, uncached
    tokens there)."""

    def __init__(self, n_slots: int, base: np.ndarray):
        self.base = base.astype(np.int64).copy()
        self.q: List[List[Tuple[int, int, int, int]]] = [[] for _ in range(n_slots)]

    def loads(self) -> np.ndarray:
        return np.array([self.base[i] + sum(r[1] for r in self.q[i]) for i in range(len(self.q))],
                        dtype=np.int64)

    def append(self, rec: np.ndarray, chosen: np.ndarray, other: np.ndarray,
               unc_here: np.ndarray, unc_other: np.ndarray) -> None:
        for r, c, o, uh, uo in zip(rec.tolist(), chosen.tolist(), other.tolist(),
                                   unc_here.tolist(), unc_other.tolist()):
            self.q[c].append((r, uh, o, uo))

    def csr(self):
        lens = np.array([len(x) for x in self.q], dtype=np.int64)
        qoff = np.zeros(len(self.q) + 1, dtype=np.int64)
        np.cumsum(lens, out=qoff[1:])
        flat = [r for x in self.q for r in x]
        rec = np.array([r[0] for r in flat], dtype=np.uint64)
        here = np.array([r[1] for r in flat], dtype=np.uint32)
        alt = np.array([r[2] for r in flat], dtype=np.uint32)
        there = np.array([r[3] for r in flat], dtype=np.uint32)
        return qoff, rec, here, alt, there, self.base.copy()

    def migrate(self, rec: np.ndarray, src: np.ndarray, dst: np.ndarray) -> None:
        """Apply a migration list in order: each record leaves its source
        queue (later records move up) and joins the target's tail with its
        pair roles swapped.  Sources never receive migrants in one pass, so
        the order of removals and appends does not interact."""
        gone: Dict[int, set] = {}
        for r, s in zip(rec.tolist(), src.tolist()):
            gone.setdefault(s, set()).add(r)
        taken = {}
        for s, rs in gone.items():
            keep = []
            for x in self.q[s]:
                if x[0] in rs:
                    taken[x[0]] = x
                else:
                    keep.append(x)
            self.q[s] = keep
        for r, s, d in zip(rec.tolist(), src.tolist(), dst.tolist()):
            x = taken.pop(r)
            self.q[d].append((x[0], x[3], s, x[1]))
        assert not taken

    def drain(self, units: np.ndarray) -> None:
        """Serve `units` of work per instance: base work first, then whole
        records from the head; a partly served head keeps the remainder."""
        for i, u in enumerate(units.tolist()):
            take = min(int(self.base[i]), u)
            self.base[i] -= take
            u -= take
            q = self.q[i]
            k = 0
            while k < len(q) and u >= q[k][1]:
                u -= q[k][1]
                k += 1
            del q[:k]
            if q and u > 0:
                r = q[0]
                q[0] = (r[0], r[1] - u, r[2], r[3])


def drain_loads(loads: np.ndarray, live: np.ndarray, units: float) -> np.ndarray:
    """Queued work after `units` of service on every live instance."""
    out = loads.copy()
    out[live] = np.maximum(0, out[live] - int(units))
    return out


# ---------------------------------------------------------------------------
# Multi-batch drivers.  `side` routes and keeps an index and (agent) runs
# rebalance passes: route(tok, off, loads) -> outputs incl. block_keys and
# loads; insert(inst, keys); erase(inst, keys); rebalance(csr) -> migrations.
# Each driver yields (stage, batch, outputs) so two sides can be compared
# step by step.
# ---------------------------------------------------------------------------

_CACHE: Dict = {}


def _cached(key, make):
    """Inputs shared by the two sides of a comparison are generated once."""
    if key not in _CACHE:
        while len(_CACHE) >= 6:
            _CACHE.pop(next(iter(_CACHE)))
        _CACHE[key] = make()
    return _CACHE[key]


def _apply_lru(side, lru: LRUIndex, inst: np.ndarray, out, off: np.ndarray, block: int) -> None:
    if getattr(side, "kv_on_side", False):
        # the side saves the batch itself (dm_kv_save / or_kv_save); the
        # clock advances as the model's would
        side.kv_save(off, out, inst, lru.clock, lru.cap)
        lru.clock += int((np.maximum(np.diff(off), 0) // block).sum())
        return
    upd = lru.touch(inst, out["block_keys"], np.maximum(np.diff(off), 0) // block)
    for c, (added, removed) in sorted(upd.items()):
        if len(removed):
            side.erase(c, removed)
        if len(added):
            side.insert(c, added)


def _uncached(out, off: np.ndarray, block: int):
    n = len(off) - 1
    lens = np.diff(off).astype(np.int64)
    u1 = lens - block * out["match"][:n].astype(np.int64)
    u2 = lens - block * out["match"][n:].astype(np.int64)
    return u1, u2


def run_chat(side, cfg, n_batches: int):
    import workloads
    rc = cfg.route
    S, B = rc.max_slots, rc.block
    live = np.arange(rc.n_inst)
    lru = LRUIndex(S, cfg.lru_blocks)
    # warm-up population, routed from zero loads; its chains fill the caches
    warm = _cached(("chat-stream", cfg, 1), lambda: workloads.ChatStream(cfg, 1))
    Lw = np.zeros(S, np.int64)
    unc_sum, unc_n = 0, 0
    for lo in range(0, warm.n, cfg.batch):
        tok, off = _cached(("chat", cfg, 1, lo), lambda: warm.batch(lo, lo + cfg.batch))
        out = side.route(tok, off, Lw)
        yield "warm", lo // cfg.batch, out
        Lw = out["loads"]
        u1, u2 = _uncached(out, off, B)
        n = len(off) - 1
        unc_sum += int(np.where(out["chosen"] == out["cand"][:n], u1, u2).sum())
        unc_n += n
        _apply_lru(side, lru, out["chosen"], out, off, B)
    # Poisson arrivals at the rate that offers `utilisation` of the drain
    mean_gap = (unc_sum / max(unc_n, 1)) / (cfg.utilisation * rc.n_inst * cfg.drain_per_us)
    gaps = workloads.arrival_gaps(cfg.seed, n_batches, cfg.batch, mean_gap)
    stream = _cached(("chat-stream", cfg, 0), lambda: workloads.ChatStream(cfg, 0))
    L = workloads.batch_initial_loads(cfg.seed, S, cfg.load_hi)
    for b in range(n_batches):
        tok, off = _cached(("chat", cfg, 0, b),
                           lambda: stream.batch(b * cfg.batch, (b + 1) * cfg.batch))
        if len(off) < 2:
            break
        out = side.route(tok, off, L)
        yield "route", b, out
        _apply_lru(side, lru, out["chosen"], out, off, B)
        L = drain_loads(out["loads"], live, cfg.drain_per_us * gaps[b])


def agent_base_work(cfg, mu: int) -> np.ndarray:
    base = np.zeros(cfg.route.max_slots, np.int64)
    base[: cfg.route.n_inst] = mu
    return base


def _close_window(side, stage, b):
    """With the prefix hotness tree on, every routed batch is one window."""
    if getattr(side, "keylen", False):
        side.window()
        return ("window", b, {"tree": side.tree()})
    return None


def run_agent(side, cfg, mu: int, n_batches: int, warm: bool = True):
    import workloads
    rc = cfg.route
    S, B = rc.max_slots, rc.block
    lru = LRUIndex(S, cfg.lru_blocks)
    unc_sum, unc_n = 0, 0
    if warm:
        Lw = np.zeros(S, np.int64)
        for w in range(0, cfg.n_warm, cfg.batch):
            n = min(cfg.batch, cfg.n_warm - w)
            tok, off = _cached(("agent", cfg, 1, w),
                               lambda: workloads.agent_batch(cfg, w // cfg.batch, n, warm=True))
            out = side.route(tok, off, Lw)
            yield "warm", w // cfg.batch, out
            win = _close_window(side, "warm", w // cfg.batch)
            if win:
                yield win
            Lw = out["loads"]
            u1, u2 = _uncached(out, off, B)
            unc_sum += int(np.where(out["chosen"] == out["cand"][:n], u1, u2).sum())
            unc_n += n
            _apply_lru(side, lru, out["chosen"], out, off, B)
    mean_gap = (unc_sum / max(unc_n, 1)) / (cfg.utilisation * rc.n_inst * cfg.drain_per_us)
    gaps = workloads.arrival_gaps(cfg.seed, n_batches, cfg.batch, mean_gap)
    # the side keeps the queues itself (dm_queue_* / or_queue_*), or this
    # module's model does
    qs = side.queues(S, agent_base_work(cfg, mu)) if getattr(side, "queues_on_side", False) \
        else QueueState(S, agent_base_work(cfg, mu))
    for b in range(n_batches):
        tok, off = _cached(("agent", cfg, 0, b), lambda: workloads.agent_batch(cfg, b, cfg.batch))
        n = len(off) - 1
        out = side.route(tok, off, qs.loads())
        yield "route", b, out
        win = _close_window(side, "route", b)
        if win:
            yield win
        c1, c2 = out["cand"][:n].astype(np.int64), out["cand"][n:].astype(np.int64)
        ch = out["chosen"].astype(np.int64)
        u1, u2 = _uncached(out, off, B)
        first = ch == c1
        rec = np.arange(b * cfg.batch, b * cfg.batch + n, dtype=np.uint64)
        if getattr(side, "queues_on_side", False):
            qs.append_routed(off, b * cfg.batch)
        else:
            qs.append(rec, ch, np.where(first, c2, c1), np.where(first, u1, u2),
                      np.where(first, u2, u1))
        # a stall the router did not see (e.g. decode-bound instances,
        # Sec. A.7): a few instances' queued work jumps to hot_factor x mu
        hot = workloads.agent_hot_instances(cfg, b)
        qs.base[hot] += (cfg.hot_factor - 1) * mu
        if getattr(side, "reprobe", False):
            # queued records re-priced against the caches as they are now
            qs.reprobe()
        queued = qs.count() if getattr(side, "queues_on_side", False) else sum(len(x) for x in qs.q)
        mg = side.rebalance(qs.csr())
        mg["queued"] = queued
        yield "rebalance", b, mg
        qs.migrate(mg["rec"], mg["src"], mg["dst"])
        # the request's blocks are computed where it is finally served
        served = ch.copy()
        mine = (mg["rec"] >= b * cfg.batch) & (mg["rec"] < b * cfg.batch + n)
        served[(mg["rec"][mine] - b * cfg.batch).astype(np.int64)] = mg["dst"][mine]
        _apply_lru(side, lru, served, out, off, B)
        units = np.zeros(S, np.int64)
        units[: rc.n_inst] = int(cfg.drain_per_us * gaps[b])
        qs.drain(units)
