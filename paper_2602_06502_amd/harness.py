"""Workload set-up on the GPU engine for tests and the benchmark.

Builds the cluster state a workload starts from using only the engine's C
ABI (through the binding) and the seeded generators in `workloads`:
  - rings for ids 0..n_inst-1;
  - cached block sets: for the tiny and random workloads, prior requests are
    routed over an empty index with zero loads and each routed chain is
    inserted into its chosen instance; for the large workload every
    template's chain goes into its first candidate (and, on a coin flip, its
    second), then each instance is topped up with random keys to
    filler_per_inst keys;
  - initial loads.
"""
from __future__ import annotations

from typing import Dict, Optional

import numpy as np

import workloads

from . import DualMap


def _torch():
    import torch
    return torch


def to_dev(a: np.ndarray, device):
    torch = _torch()
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


def engine_for(wl: workloads.Workload, device="cuda:0", n_live: Optional[int] = None) -> DualMap:
    cfg = wl.route.as_dict()
    eng = DualMap(cfg, device=device)
    eng.build_rings(range(wl.route.n_inst if n_live is None else n_live))
    return eng


def insert_blocks(eng: DualMap, keys, per_block_inst) -> None:
    """Insert block key k into the index of instance per_block_inst[k]."""
    torch = _torch()
    k64 = keys[:per_block_inst.numel()].view(torch.int64)
    for c in torch.unique(per_block_inst).tolist():
        sel = k64[per_block_inst == c].contiguous().view(torch.uint64)
        eng.index_insert(int(c), sel)


def full_blocks(eng: DualMap, offsets):
    torch = _torch()
    return ((offsets[1:] - offsets[:-1]).clamp(min=0) // eng.block).to(torch.int64)


def prefill_from_prior(eng: DualMap, wl: workloads.Workload) -> None:
    """Route the workload's prior requests over the current index with zero
    loads and cache each chain on its chosen instance."""
    torch = _torch()
    if wl.n_prior == 0:
        return
    tok, off = workloads.prompts(wl, wl.n_prior, sub=1)
    tok_d, off_d = to_dev(tok, eng.device), to_dev(off, eng.device)
    zero = torch.zeros(eng.max_slots, dtype=torch.int64, device=eng.device)
    out = eng.route(tok_d, off_d, zero, block_keys=True)
    per_block = torch.repeat_interleave(out["chosen"].to(torch.int64), full_blocks(eng, off_d))
    insert_blocks(eng, out["block_keys"], per_block)
    eng.sync()


def prefill_templates(eng: DualMap, wl: workloads.Workload) -> None:
    """Template chains into candidate 1 (and candidate 2 on a coin flip),
    then random keys up to filler_per_inst keys per live instance."""
    torch = _torch()
    ttok, toff = workloads.templates(wl)
    tok_d, off_d = to_dev(ttok, eng.device), to_dev(toff, eng.device)
    zero = torch.zeros(eng.max_slots, dtype=torch.int64, device=eng.device)
    out = eng.route(tok_d, off_d, zero, block_keys=True)
    nt = wl.n_templates
    nfull = full_blocks(eng, off_d)
    c1 = torch.repeat_interleave(out["cand"][:nt].to(torch.int64), nfull)
    c2 = torch.repeat_interleave(out["cand"][nt:].to(torch.int64), nfull)
    coin = torch.repeat_interleave(to_dev(workloads.coin_flips(wl, nt).astype(np.int64),
                                          eng.device), nfull).bool()
    insert_blocks(eng, out["block_keys"], c1)
    k64 = out["block_keys"].view(torch.int64)
    insert_blocks(eng, k64[coin].contiguous().view(torch.uint64), c2[coin])
    eng.sync()
    if wl.filler_per_inst:
        for c in range(wl.route.n_inst):
            have = eng.index_size(c)
            fk = workloads.filler_keys(wl, c, wl.filler_per_inst - have)
            if len(fk):
                eng.index_insert(c, to_dev(fk, eng.device))
        eng.sync()


def setup(wl: workloads.Workload, device="cuda:0") -> Dict:
    """Engine with the workload's starting state, its measured batch on the
    device and its initial loads."""
    eng = engine_for(wl, device)
    if wl.filler_per_inst:
        prefill_templates(eng, wl)
    else:
        prefill_from_prior(eng, wl)
    tok, off = workloads.prompts(wl, wl.n_req, sub=0)
    loads0 = workloads.initial_loads(wl, wl.route.max_slots)
    return dict(eng=eng, tokens=to_dev(tok, eng.device), offsets=to_dev(off, eng.device),
                loads0=loads0, tokens_np=tok, offsets_np=off)


def setup_warm(cfg, device="cuda:0") -> Dict:
    """Engine for a chat or agent workload after its warm-up: the warm-up
    batches routed in order from zero queued work (loads carried from batch
    to batch), each batch's chains cached on its chosen instance.  The
    warm-up stays under the per-instance cache bound, so no block is
    evicted.  Returns the engine and the first measured batch (device and
    host copies) with its queued work."""
    torch = _torch()
    rc = cfg.route
    eng = DualMap(rc.as_dict(), device=device)
    eng.build_rings(list(range(rc.n_inst)))
    Lw = torch.zeros(eng.max_slots, dtype=torch.int64, device=eng.device)
    for tok, off in workloads.warmup_batches(cfg):
        off_d = to_dev(off, eng.device)
        out = eng.route(to_dev(tok, eng.device), off_d, Lw, block_keys=True)
        per_block = torch.repeat_interleave(out["chosen"].to(torch.int64), full_blocks(eng, off_d))
        insert_blocks(eng, out["block_keys"], per_block)
    eng.sync()
    tok, off, L0 = workloads.measured_batch(cfg)
    return dict(eng=eng, tokens=to_dev(tok, eng.device), offsets=to_dev(off, eng.device),
                loads0=L0, tokens_np=tok, offsets_np=off)
