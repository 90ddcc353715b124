"""Workload set-up on the CPU oracle -- TEST INFRASTRUCTURE ONLY.

Builds a workload's starting state with the oracle's own functions and the
seeded generators in `workloads` (rings for ids 0..n_inst-1; cached block
sets from routed prior requests, or from template chains on their first
candidate -- and on a coin flip their second -- topped up with random keys;
initial loads), mirroring the steps the GPU-side set-up takes with the
engine.
"""
from __future__ import annotations

from typing import Dict

import numpy as np

import workloads

from . import Oracle


def oracle_for(wl: workloads.Workload, n_live=None) -> Oracle:
    o = Oracle(wl.route.as_dict())
    rc = o.build_rings(range(wl.route.n_inst if n_live is None else n_live))
    assert rc == 0, rc
    return o


def insert_blocks(o: Oracle, keys: np.ndarray, per_block_inst: np.ndarray) -> None:
    for c in np.unique(per_block_inst):
        o.index_insert(int(c), keys[per_block_inst == c])


def prefill_from_prior(o: Oracle, wl: workloads.Workload) -> None:
    if wl.n_prior == 0:
        return
    tok, off = workloads.prompts(wl, wl.n_prior, sub=1)
    out = o.route(tok, off, np.zeros(wl.route.max_slots, np.int64), block_keys=True)
    nfull = np.diff(off) // wl.route.block
    insert_blocks(o, out["block_keys"], np.repeat(out["chosen"], nfull))


def prefill_templates(o: Oracle, wl: workloads.Workload) -> None:
    ttok, toff = workloads.templates(wl)
    out = o.route(ttok, toff, np.zeros(wl.route.max_slots, np.int64), block_keys=True)
    nt = wl.n_templates
    nfull = np.diff(toff) // wl.route.block
    c1 = np.repeat(out["cand"][:nt], nfull)
    c2 = np.repeat(out["cand"][nt:], nfull)
    coin = np.repeat(workloads.coin_flips(wl, nt).astype(bool), nfull)
    insert_blocks(o, out["block_keys"], c1)
    insert_blocks(o, out["block_keys"][coin], c2[coin])
    if wl.filler_per_inst:
        for c in range(wl.route.n_inst):
            have = o.index_size(c)
            fk = workloads.filler_keys(wl, c, wl.filler_per_inst - have)
            if len(fk):
                o.index_insert(c, fk)


def setup(wl: workloads.Workload, with_batch: bool = True) -> Dict:
    o = oracle_for(wl)
    if wl.filler_per_inst:
        prefill_templates(o, wl)
    else:
        prefill_from_prior(o, wl)
    res = dict(oracle=o, loads0=workloads.initial_loads(wl, wl.route.max_slots))
    if with_batch:
        res["tokens"], res["offsets"] = workloads.prompts(wl, wl.n_req, sub=0)
    return res


def setup_warm(cfg) -> Dict:
    """The oracle's counterpart of the engine-side warm start of a chat or
    agent workload: warm-up batches routed in order from zero queued work,
    each batch's chains inserted into its chosen instance; then the first
    measured batch and its queued work."""
    rc = cfg.route
    o = Oracle(rc.as_dict())
    assert o.build_rings(range(rc.n_inst)) == 0
    Lw = np.zeros(rc.max_slots, np.int64)
    for tok, off in workloads.warmup_batches(cfg):
        out = o.route(tok, off, Lw, block_keys=True)
        Lw = out["loads"]
        insert_blocks(o, out["block_keys"], np.repeat(out["chosen"], np.diff(off) // rc.block))
    tok, off, L0 = workloads.measured_batch(cfg)
    return dict(oracle=o, tokens=tok, offsets=off, loads0=L0)
