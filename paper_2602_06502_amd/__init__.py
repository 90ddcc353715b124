"""Python binding of the DualMap routing engine (libdualmap.so, gfx950).

Argument marshalling only: every step of routing, rebalancing and scaling
runs in the HIP kernels behind the C ABI declared in include/dualmap.h.
PyTorch supplies device memory and the stream.  The module refuses to load
if the library has not been built (run __graft_entry__.build() or
python -m paper_2602_06502_amd._build); there is no CPU fallback.

Functions with the C names (dm_create, dm_build_rings, dm_index_insert,
dm_route_batch, dm_rebalance, dm_scale, ...) take raw device pointers; the
DualMap class wraps them for torch tensors.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Dict, Optional, Sequence

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libdualmap.so")

DM_OK, DM_EINVAL, DM_ENOMEM, DM_EFULL, DM_ESTATE, DM_EDEVICE = range(6)
_NAMES = {0: "DM_OK", 1: "DM_EINVAL", 2: "DM_ENOMEM", 3: "DM_EFULL", 4: "DM_ESTATE",
          5: "DM_EDEVICE"}

EXPORTS = ("dm_create", "dm_destroy", "dm_build_rings", "dm_ring_export", "dm_index_insert",
           "dm_index_erase", "dm_index_clear", "dm_index_size", "dm_route_batch",
           "dm_route_batch_noalloc",
           "dm_rebalance", "dm_scale", "dm_set_timing", "dm_route_stage_ms",
           "dm_kv_save", "dm_queue_append", "dm_queue_migrate", "dm_queue_drain", "dm_queue_reprobe",
           "dm_set_pipelining", "dm_set_policy", "dm_keylen_enable",
           "dm_keylen_window",
           "dm_keylen_export", "dm_sync", "dm_last_error")


class DMError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{_NAMES.get(status, status)}: {msg}")
        self.status = status


class dm_config(C.Structure):
    _fields_ = [("block_size", C.c_uint32), ("key_blocks", C.c_uint32),
                ("seed", C.c_uint64 * 2), ("vnodes", C.c_uint32), ("max_slots", C.c_uint32),
                ("index_log2_slots", C.c_uint32), ("reserved", C.c_uint32),
                ("ttft_base_us", C.c_int64), ("ttft_per_token_us", C.c_int64),
                ("queue_div", C.c_int64), ("slo_us", C.c_int64)]


class dm_route_out(C.Structure):
    _fields_ = [("key", C.c_void_p), ("cand", C.c_void_p), ("match", C.c_void_p),
                ("chosen", C.c_void_p), ("ttft_us", C.c_void_p), ("flags", C.c_void_p),
                ("block_keys", C.c_void_p), ("key_len", C.c_void_p)]


class dm_queues(C.Structure):
    _fields_ = [("qoff", C.c_void_p), ("rec_id", C.c_void_p), ("unc_here", C.c_void_p),
                ("alt", C.c_void_p), ("unc_alt", C.c_void_p), ("base_work", C.c_void_p),
                ("prefill_interval", C.c_void_p), ("decode_threshold_us", C.c_int64)]


class dm_queue_out(C.Structure):
    _fields_ = [("qoff", C.c_void_p), ("rec_id", C.c_void_p), ("unc_here", C.c_void_p),
                ("alt", C.c_void_p), ("unc_alt", C.c_void_p), ("base_work", C.c_void_p),
                ("cap", C.c_uint64)]


class dm_migrations(C.Structure):
    _fields_ = [("rec_id", C.c_void_p), ("from_", C.c_void_p), ("to", C.c_void_p),
                ("benefit_us", C.c_void_p), ("ttft_to_us", C.c_void_p), ("count", C.c_void_p)]


_lib = None


def load_library(path: str = LIB_PATH):
    """Load libdualmap.so (raises if it is missing: no fallback exists)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"libdualmap.so not built at {path}; run __graft_entry__.build()")
    L = C.CDLL(path)
    P, u32, u64, i32 = C.c_void_p, C.c_uint32, C.c_uint64, C.c_int
    sig = {
        "dm_create": (i32, [P, P, P]),
        "dm_destroy": (None, [P]),
        "dm_build_rings": (i32, [P, P, u32]),
        "dm_ring_export": (i32, [P, i32, P, P, u64, P]),
        "dm_index_insert": (i32, [P, u32, P, u64]),
        "dm_index_erase": (i32, [P, u32, P, u64]),
        "dm_index_clear": (i32, [P, u32]),
        "dm_index_size": (i32, [P, u32, P]),
        "dm_route_batch": (i32, [P, P, u64, P, u64, P, P]),
        "dm_route_batch_noalloc": (i32, [P, P, u64, P, u64, P, P]),
        "dm_rebalance": (i32, [P, P, P, P, u64]),
        "dm_scale": (i32, [P, P, u32, P, u32, P, u64, P, P, P, P]),
        "dm_set_timing": (i32, [P, i32]),
        "dm_route_stage_ms": (i32, [P, P, i32]),
        "dm_set_pipelining": (i32, [P, i32]),
        "dm_set_policy": (i32, [P, i32]),
        "dm_kv_save": (i32, [P, P, u64, P, P, u64, u64, P, P]),
        "dm_queue_append": (i32, [P, P, P, u64, P, u64, P]),
        "dm_queue_migrate": (i32, [P, P, P, P, P, u64, P]),
        "dm_queue_drain": (i32, [P, P, P, P]),
        "dm_queue_reprobe": (i32, [P, P, P, P, u64, P, u64, P]),
        "dm_keylen_enable": (i32, [P, u64, u64]),
        "dm_keylen_window": (i32, [P]),
        "dm_keylen_export": (i32, [P, P, u64, P]),
        "dm_sync": (i32, [P]),
        "dm_last_error": (C.c_char_p, [P]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


def __getattr__(name):
    # dm_* names resolve to the C functions
    if name in EXPORTS:
        return getattr(load_library(), name)
    raise AttributeError(name)


def make_config(cfg: Dict) -> dm_config:
    c = dm_config()
    c.block_size = cfg["block"]
    c.key_blocks = cfg["key_blocks"]
    c.seed[0], c.seed[1] = cfg["seeds"]
    c.vnodes = cfg["vnodes"]
    c.max_slots = cfg["max_slots"]
    c.index_log2_slots = cfg.get("index_log2_slots", 16)
    c.reserved = 0
    c.ttft_base_us = cfg.get("ttft_base_us", 2000)
    c.ttft_per_token_us = cfg.get("ttft_per_token_us", 3)
    c.queue_div = cfg.get("queue_div", 4)
    c.slo_us = cfg.get("slo_us", 400_000)
    return c


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


class DualMap:
    """A routing engine context on one GPU (torch tensors in and out)."""

    def __init__(self, cfg: Dict, device=None, stream=None):
        import torch
        self.torch = torch
        self.lib = load_library()
        self.device = torch.device("cuda", torch.cuda.current_device() if device is None
                                   else torch.device(device).index or 0)
        self.cfg = dict(cfg)
        self.max_slots = cfg["max_slots"]
        self.block = cfg["block"]
        with torch.cuda.device(self.device):
            self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
            h = C.c_void_p()
            st = self.lib.dm_create(C.byref(make_config(cfg)), C.c_void_p(self.stream.cuda_stream),
                                    C.byref(h))
        if st != DM_OK:
            raise DMError(st, "dm_create rejected the configuration %r" % (cfg,))
        self._h = h

    def close(self):
        if getattr(self, "_h", None):
            self.lib.dm_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- helpers ----------------------------------------------------------
    def _check(self, st: int, what: str):
        if st != DM_OK:
            raise DMError(st, f"{what}: {self.lib.dm_last_error(self._h).decode()}")

    def _dev(self, t, dtype, name):
        torch = self.torch
        if not isinstance(t, torch.Tensor) or t.device != self.device or t.dtype != dtype \
                or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous {dtype} tensor on {self.device}")
        return t

    def _empty(self, n, dtype):
        return self.torch.empty(max(int(n), 0), dtype=dtype, device=self.device)

    # -- C ABI mirrors --------------------------------------------------------
    def set_timing(self, on: bool) -> None:
        self._check(self.lib.dm_set_timing(self._h, 1 if on else 0), "dm_set_timing")

    def set_pipelining(self, on: bool) -> None:
        """Overlap each batch's selection with the next batch's hashing and
        probing (see dm_set_pipelining): consecutive batches need distinct
        output buffers, and results are final after sync()."""
        self._check(self.lib.dm_set_pipelining(self._h, 1 if on else 0), "dm_set_pipelining")

    POLICIES = {"slo_aware": 0, "cache_affinity": 1, "least_loaded": 2, "min_ttft": 3}

    def set_policy(self, policy) -> None:
        """Selection rule of later batches (see dm_set_policy): a name of
        POLICIES or its number."""
        p = self.POLICIES[policy] if isinstance(policy, str) else int(policy)
        self._check(self.lib.dm_set_policy(self._h, p), "dm_set_policy")

    def stage_ms(self):
        """(hash, lookup+match, selection, block offsets) ms, averaged over the
        batches routed since timing was turned on (the last 64 at most)."""
        ms = (C.c_float * 4)()
        self._check(self.lib.dm_route_stage_ms(self._h, ms, 4), "dm_route_stage_ms")
        return tuple(float(x) for x in ms)

    def sync(self) -> None:
        self._check(self.lib.dm_sync(self._h), "dm_sync")

    def build_rings(self, ids: Sequence[int]) -> None:
        arr = (C.c_uint32 * len(ids))(*[int(i) for i in ids])
        self._check(self.lib.dm_build_rings(self._h, arr, len(ids)), "dm_build_rings")

    def ring(self, s: int):
        import numpy as np
        n = C.c_uint64()
        self._check(self.lib.dm_ring_export(self._h, s, None, None, 0, C.byref(n)), "dm_ring_export")
        pos = np.zeros(n.value, np.uint64)
        ids = np.zeros(n.value, np.uint32)
        self._check(self.lib.dm_ring_export(self._h, s, pos.ctypes.data_as(C.c_void_p),
                                            ids.ctypes.data_as(C.c_void_p), n.value, C.byref(n)),
                    "dm_ring_export")
        return pos, ids

    def index_insert(self, inst: int, keys) -> None:
        keys = self._dev(keys, self.torch.uint64, "keys")
        self._check(self.lib.dm_index_insert(self._h, inst, _ptr(keys), keys.numel()),
                    "dm_index_insert")

    def index_erase(self, inst: int, keys) -> None:
        keys = self._dev(keys, self.torch.uint64, "keys")
        self._check(self.lib.dm_index_erase(self._h, inst, _ptr(keys), keys.numel()),
                    "dm_index_erase")

    def index_clear(self, inst: int) -> None:
        self._check(self.lib.dm_index_clear(self._h, inst), "dm_index_clear")

    def index_size(self, inst: int) -> int:
        n = C.c_uint64()
        self._check(self.lib.dm_index_size(self._h, inst, C.byref(n)), "dm_index_size")
        return int(n.value)

    def route_into(self, tokens, offsets, loads, out: Dict, noalloc: bool = False) -> None:
        """dm_route_batch into preallocated outputs; with noalloc,
        dm_route_batch_noalloc (work arrays from the library's static area)."""
        n = offsets.numel() - 1
        ro = dm_route_out(_ptr(out["key"]), _ptr(out["cand"]), _ptr(out["match"]),
                          _ptr(out["chosen"]), _ptr(out["ttft"]), _ptr(out["flags"]),
                          _ptr(out.get("block_keys")), _ptr(out.get("key_len")))
        fn = self.lib.dm_route_batch_noalloc if noalloc else self.lib.dm_route_batch
        name = "dm_route_batch_noalloc" if noalloc else "dm_route_batch"
        self._check(fn(self._h, _ptr(tokens), tokens.numel(), _ptr(offsets), n, _ptr(loads),
                       C.byref(ro)), name)

    def alloc_route_out(self, n: int, n_blocks: Optional[int] = None,
                        key_len: bool = False) -> Dict:
        t = self.torch
        out = dict(key=self._empty(2 * n, t.uint64), cand=self._empty(2 * n, t.uint32),
                   match=self._empty(2 * n, t.uint32), chosen=self._empty(n, t.uint32),
                   ttft=self._empty(n, t.int64), flags=self._empty(n, t.uint8))
        if n_blocks is not None:
            out["block_keys"] = self._empty(max(n_blocks, 1), t.uint64)
        if key_len:
            out["key_len"] = self._empty(max(n, 1), t.uint32)
        return out

    def kv_save(self, offsets, block_keys, inst, clock: int, cap: int):
        """Save a served batch's blocks with LRU eviction (see dm_kv_save);
        returns (keys added, keys removed)."""
        t = self.torch
        offsets = self._dev(offsets, t.int64, "offsets")
        block_keys = self._dev(block_keys, t.uint64, "block_keys")
        inst = self._dev(inst, t.uint32, "inst")
        a, r = C.c_uint64(), C.c_uint64()
        self._check(self.lib.dm_kv_save(self._h, _ptr(offsets), offsets.numel() - 1,
                                        _ptr(block_keys), _ptr(inst), int(clock), int(cap),
                                        C.byref(a), C.byref(r)), "dm_kv_save")
        return int(a.value), int(r.value)

    # -- queued requests on the device: tuples (qoff, rec_id, unc_here, alt,
    # unc_alt, base_work) of device tensors
    def _qin(self, q):
        t = self.torch
        qoff, rec, here, alt, there, base = q
        return (self._dev(qoff, t.int64, "qoff"), self._dev(rec, t.uint64, "rec_id"),
                self._dev(here, t.uint32, "unc_here"), self._dev(alt, t.uint32, "alt"),
                self._dev(there, t.uint32, "unc_alt"), self._dev(base, t.int64, "base_work"))

    def _qnew(self, cap: int):
        t = self.torch
        c = max(int(cap), 1)
        return (self._empty(self.max_slots + 1, t.int64), self._empty(c, t.uint64),
                self._empty(c, t.uint32), self._empty(c, t.uint32), self._empty(c, t.uint32),
                self._empty(self.max_slots, t.int64))

    @staticmethod
    def _qstructs(qi, qo, cap):
        qs = dm_queues(*[_ptr(x) for x in qi], None, 0)
        qd = dm_queue_out(*[_ptr(x) for x in qo], int(cap))
        return qs, qd

    def _qtrim(self, qo):
        n = int(qo[0][-1].item())
        return (qo[0], qo[1][:n], qo[2][:n], qo[3][:n], qo[4][:n], qo[5])

    def queue_append(self, q, offsets, routed: Dict, rec_base: int):
        """A routed batch joins the queues (see dm_queue_append)."""
        qi = self._qin(q)
        offsets = self._dev(offsets, self.torch.int64, "offsets")
        n = offsets.numel() - 1
        cap = qi[1].numel() + n
        qo = self._qnew(cap)
        qs, qd = self._qstructs(qi, qo, cap)
        ro = dm_route_out(_ptr(routed["key"]), _ptr(routed["cand"]), _ptr(routed["match"]),
                          _ptr(routed["chosen"]), _ptr(routed["ttft"]), _ptr(routed["flags"]),
                          None, None)
        self._check(self.lib.dm_queue_append(self._h, C.byref(qs), _ptr(offsets), n,
                                             C.byref(ro), int(rec_base), C.byref(qd)),
                    "dm_queue_append")
        return self._qtrim(qo)

    def queue_migrate(self, q, rec_id, src, dst):
        """A migration list applied to the queues (see dm_queue_migrate)."""
        t = self.torch
        qi = self._qin(q)
        rec_id = self._dev(rec_id, t.uint64, "rec_id")
        src = self._dev(src, t.uint32, "from")
        dst = self._dev(dst, t.uint32, "to")
        cap = qi[1].numel()
        qo = self._qnew(cap)
        qs, qd = self._qstructs(qi, qo, cap)
        self._check(self.lib.dm_queue_migrate(self._h, C.byref(qs), _ptr(rec_id), _ptr(src),
                                              _ptr(dst), rec_id.numel(), C.byref(qd)),
                    "dm_queue_migrate")
        return self._qtrim(qo)

    def queue_drain(self, q, units):
        """units[i] of service per instance (see dm_queue_drain)."""
        qi = self._qin(q)
        units = self._dev(units, self.torch.int64, "units")
        cap = qi[1].numel()
        qo = self._qnew(cap)
        qs, qd = self._qstructs(qi, qo, cap)
        self._check(self.lib.dm_queue_drain(self._h, C.byref(qs), _ptr(units), C.byref(qd)),
                    "dm_queue_drain")
        return self._qtrim(qo)

    def queue_reprobe(self, q, chain_off, chain_keys, prompt_len):
        """Queued records re-priced against the current caches (see
        dm_queue_reprobe): record id r's chain chain_keys[chain_off[r]:
        chain_off[r+1]], its prompt prompt_len[r] tokens."""
        t = self.torch
        qi = self._qin(q)
        chain_off = self._dev(chain_off, t.int64, "chain_off")
        chain_keys = self._dev(chain_keys, t.uint64, "chain_keys")
        prompt_len = self._dev(prompt_len, t.int64, "prompt_len")
        if chain_off.numel() != prompt_len.numel() + 1:
            raise ValueError("chain_off needs one entry more than prompt_len")
        cap = qi[1].numel()
        qo = self._qnew(cap)
        qs, qd = self._qstructs(qi, qo, cap)
        self._check(self.lib.dm_queue_reprobe(self._h, C.byref(qs), _ptr(chain_off),
                                              _ptr(chain_keys), chain_keys.numel(),
                                              _ptr(prompt_len), prompt_len.numel(), C.byref(qd)),
                    "dm_queue_reprobe")
        return self._qtrim(qo)

    def keylen_enable(self, max_nodes: int, max_window_blocks: int = 1 << 24) -> None:
        """Adaptive hash-key length (see dm_keylen_enable): an empty prefix
        hotness tree with room for max_nodes extended prefixes and a window
        record of max_window_blocks prefixes; max_nodes = 0 turns it off."""
        self._check(self.lib.dm_keylen_enable(self._h, int(max_nodes), int(max_window_blocks)),
                    "dm_keylen_enable")

    def keylen_window(self) -> None:
        """Close the hotness window: hot leaves extend, cold nodes shrink."""
        self._check(self.lib.dm_keylen_window(self._h), "dm_keylen_window")

    def keylen_tree(self):
        """The extended prefixes (canonical f1 keys), ascending, as numpy."""
        import numpy as np
        n = C.c_uint64()
        self._check(self.lib.dm_keylen_export(self._h, None, 0, C.byref(n)), "dm_keylen_export")
        a = np.zeros(max(int(n.value), 1), np.uint64)
        self._check(self.lib.dm_keylen_export(self._h, a.ctypes.data_as(C.c_void_p), len(a),
                                              C.byref(n)), "dm_keylen_export")
        return a[:int(n.value)]

    def route(self, tokens, offsets, loads, block_keys: bool = False) -> Dict:
        """Route a batch; loads (int64 [max_slots]) are updated in place."""
        t = self.torch
        tokens = self._dev(tokens, t.int32, "tokens")
        offsets = self._dev(offsets, t.int64, "offsets")
        loads = self._dev(loads, t.int64, "loads")
        if loads.numel() != self.max_slots:
            raise ValueError("loads must have max_slots entries")
        n = offsets.numel() - 1
        nb = None
        if block_keys:
            nb = int(((offsets[1:] - offsets[:-1]).clamp(min=0) // self.block).sum().item())
        out = self.alloc_route_out(n, nb, key_len=True)
        self.route_into(tokens, offsets, loads, out)
        return out

    def rebalance(self, qoff, rec_id, unc_here, alt, unc_alt, base_work, cap: Optional[int] = None,
                  prefill_interval=None, decode_threshold_us: int = 3_000_000):
        t = self.torch
        qoff = self._dev(qoff, t.int64, "qoff")
        rec_id = self._dev(rec_id, t.uint64, "rec_id")
        unc_here = self._dev(unc_here, t.uint32, "unc_here")
        alt = self._dev(alt, t.uint32, "alt")
        unc_alt = self._dev(unc_alt, t.uint32, "unc_alt")
        base_work = self._dev(base_work, t.int64, "base_work")
        if qoff.numel() != self.max_slots + 1 or base_work.numel() != self.max_slots:
            raise ValueError("qoff needs max_slots + 1 entries and base_work max_slots")
        if prefill_interval is not None:
            prefill_interval = self._dev(prefill_interval, t.int64, "prefill_interval")
            if prefill_interval.numel() != self.max_slots:
                raise ValueError("prefill_interval needs max_slots entries")
        cap = rec_id.numel() if cap is None else cap
        m = dict(rec=self._empty(max(cap, 1), t.uint64), src=self._empty(max(cap, 1), t.uint32),
                 dst=self._empty(max(cap, 1), t.uint32), benefit=self._empty(max(cap, 1), t.int64),
                 ttft_to=self._empty(max(cap, 1), t.int64), count=self._empty(1, t.uint64))
        loads = self._empty(self.max_slots, t.int64)
        q = dm_queues(_ptr(qoff), _ptr(rec_id), _ptr(unc_here), _ptr(alt), _ptr(unc_alt),
                      _ptr(base_work),
                      _ptr(prefill_interval), int(decode_threshold_us))
        mg = dm_migrations(_ptr(m["rec"]), _ptr(m["src"]), _ptr(m["dst"]), _ptr(m["benefit"]),
                           _ptr(m["ttft_to"]), _ptr(m["count"]))
        self._check(self.lib.dm_rebalance(self._h, C.byref(q), _ptr(loads), C.byref(mg), cap),
                    "dm_rebalance")
        m["loads"] = loads
        return m

    def scale(self, add: Sequence[int], rm: Sequence[int], keys) -> Dict:
        t = self.torch
        keys = self._dev(keys, t.uint64, "keys")
        n = keys.numel() // 2
        a = (C.c_uint32 * max(len(add), 1))(*[int(i) for i in add])
        r = (C.c_uint32 * max(len(rm), 1))(*[int(i) for i in rm])
        out = dict(old=self._empty(2 * n, t.uint32), new=self._empty(2 * n, t.uint32),
                   moved=self._empty(2, t.uint64), violations=self._empty(1, t.uint64))
        self._check(self.lib.dm_scale(self._h, a, len(add), r, len(rm), _ptr(keys), n,
                                      _ptr(out["old"]), _ptr(out["new"]), _ptr(out["moved"]),
                                      _ptr(out["violations"])), "dm_scale")
        return out
