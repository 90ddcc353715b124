"""CPU oracle of DualMap's routing path -- TEST INFRASTRUCTURE ONLY.

Python handle over the plain single-threaded C oracle in dm_oracle.c.  Only
the tests, the package smoke check and the benchmark's CPU-baseline leg may
import this module; the product path (the HIP library and its binding) never
does, and shares no code with it.

build() compiles dm_oracle.c with gcc into liboracle.so next to it.  A
process that sets DM_ORACLE_LIB loads the build at that path instead (the
sanitizer tests use it for an instrumented build of the same source).
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from typing import Dict, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "dm_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

OK, EINVAL, ENOMEM, EFULL, ESTATE = 0, 1, 2, 3, 4


def build(force: bool = True) -> str:
    """Compile the oracle (gcc -O2, single-threaded)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-shared", "-fPIC",
                               "-o", tmp, _SRC])
        os.replace(tmp, _LIB)
    return _LIB


class _Cfg(C.Structure):
    _fields_ = [("block_size", C.c_uint32), ("key_blocks", C.c_uint32),
                ("seed", C.c_uint64 * 2), ("vnodes", C.c_uint32), ("max_slots", C.c_uint32),
                ("ttft_base_us", C.c_int64), ("ttft_per_token_us", C.c_int64),
                ("queue_div", C.c_int64), ("slo_us", C.c_int64)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        path = os.environ.get("DM_ORACLE_LIB")
        if not path:
            path = _LIB
            if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
                build(force=False)
        L = C.CDLL(path)
        P = C.c_void_p
        u64, u32, i64, i32 = C.c_uint64, C.c_uint32, C.c_int64, C.c_int
        sig = {
            "or_mix64": (u64, [u64]),
            "or_params": (None, [u64, u32, P, P, P]),
            "or_nh": (u64, [P, P, u32]),
            "or_chain": (u64, [P, i32, P, i64, P]),
            "or_ring_key": (u64, [P, i32, P, i64]),
            "or_vpos": (u64, [P, i32, u32, u32]),
            "or_owner_sorted": (u32, [P, P, u64, u64]),
            "or_owner": (u32, [P, i32, u64]),
            "or_sort_u64": (i32, [P, u64]),
            "or_create": (P, [P]),
            "or_destroy": (None, [P]),
            "or_build_rings": (i32, [P, P, u32]),
            "or_ring_copy": (u64, [P, i32, P, P]),
            "or_canon": (u64, [u64]),
            "or_index_contains": (i32, [P, u32, u64]),
            "or_index_insert": (i32, [P, u32, P, u64]),
            "or_index_erase": (i32, [P, u32, P, u64]),
            "or_index_clear": (i32, [P, u32]),
            "or_index_size": (u64, [P, u32]),
            "or_ttft": (i64, [P, i64, i64]),
            "or_candidates": (i32, [P, u64, u64, P, P]),
            "or_select": (u32, [P, u32, u32, u64, u64, i64, P, P, P]),
            "or_route": (i32, [P, P, P, u64, P, P, P, P, P, P, P, P, P]),
            "or_set_policy": (i32, [P, i32]),
            "or_kv_save": (i32, [P, P, u64, P, P, u64, u64, P, P]),
            "or_queue_append": (i32, [P, P, P, P, P, P, u64, P, P, P, P, u64, P, P, P, P, P]),
            "or_queue_migrate": (i32, [P, P, P, P, P, P, u64, P, P, P, P, P, P, P, P]),
            "or_queue_drain": (i32, [P, P, P, P, P, P, P, P, P, P, P, P, P, P]),
            "or_queue_reprobe": (i32, [P, P, P, P, u64, P, P, P, P, P]),
            "or_keylen_enable": (i32, [P, u64]),
            "or_keylen_window": (i32, [P]),
            "or_keylen_export": (i32, [P, P, u64, P]),
            "or_ring_key_at": (u64, [P, i32, P, u64]),
            "or_rebalance": (i32, [P, P, P, P, P, P, P, P, i64, P, P, P, P, P, P, u64, P]),
            "or_scale": (i32, [P, P, u32, P, u32, P, u64, P, P, P, P]),
            "or_n_live": (u32, [P]),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def mix64(z: int) -> int:
    return int(lib().or_mix64(z & 0xFFFFFFFFFFFFFFFF))


def params(seed: int, block: int):
    """(key words uint32[B], multiplier, chain start) of one hash function."""
    kk = np.zeros(block, dtype=np.uint32)
    m, h = C.c_uint64(), C.c_uint64()
    lib().or_params(seed, block, _p(kk), C.byref(m), C.byref(h))
    return kk, int(m.value), int(h.value)


def nh(tokens: np.ndarray, kk: np.ndarray) -> int:
    t = np.ascontiguousarray(tokens, dtype=np.int32)
    k = np.ascontiguousarray(kk, dtype=np.uint32)
    return int(lib().or_nh(_p(t), _p(k), len(t)))


def owner_sorted(pos: np.ndarray, ids: np.ndarray, x: int) -> int:
    pos = np.ascontiguousarray(pos, dtype=np.uint64)
    ids = np.ascontiguousarray(ids, dtype=np.uint32)
    return int(lib().or_owner_sorted(_p(pos), _p(ids), len(pos), x))


def sort_u64(a: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(a, dtype=np.uint64).copy()
    rc = lib().or_sort_u64(_p(b), len(b))
    assert rc == OK
    return b


def canon(k: int) -> int:
    return int(lib().or_canon(k))


class Oracle:
    """Oracle state: configuration, hash parameters, live set, both rings and
    each instance's cached block-key set."""

    def __init__(self, cfg: Dict):
        c = _Cfg()
        c.block_size = cfg["block"]
        c.key_blocks = cfg["key_blocks"]
        c.seed[0], c.seed[1] = cfg["seeds"]
        c.vnodes = cfg["vnodes"]
        c.max_slots = cfg["max_slots"]
        c.ttft_base_us = cfg.get("ttft_base_us", 2000)
        c.ttft_per_token_us = cfg.get("ttft_per_token_us", 3)
        c.queue_div = cfg.get("queue_div", 4)
        c.slo_us = cfg.get("slo_us", 400_000)
        self.cfg = dict(cfg)
        self.max_slots = cfg["max_slots"]
        self.block = cfg["block"]
        self._h = lib().or_create(C.byref(c))
        if not self._h:
            raise ValueError("oracle: invalid configuration %r" % (cfg,))

    def __del__(self):
        h = getattr(self, "_h", None)
        if h:
            lib().or_destroy(h)
            self._h = None

    # -- state ------------------------------------------------------------
    POLICIES = {"slo_aware": 0, "cache_affinity": 1, "least_loaded": 2, "min_ttft": 3}

    def set_policy(self, policy) -> int:
        """Selection rule for later routes: a name of POLICIES or its number."""
        p = self.POLICIES.get(policy, policy) if isinstance(policy, str) else int(policy)
        return lib().or_set_policy(self._h, p)

    def kv_save(self, offsets, block_keys, inst, clock: int, cap: int):
        """Save the batch's blocks on the serving instances with LRU eviction
        (or_kv_save); returns (status, keys added, keys removed)."""
        o = np.ascontiguousarray(offsets, np.int64)
        bk = np.ascontiguousarray(block_keys, np.uint64)
        ins = np.ascontiguousarray(inst, np.uint32)
        a, r = C.c_uint64(), C.c_uint64()
        rc = lib().or_kv_save(self._h, _p(o), len(o) - 1, _p(bk), _p(ins), int(clock), int(cap),
                              C.byref(a), C.byref(r))
        return rc, int(a.value), int(r.value)

    # -- queued requests (CSR tuples: qoff, rec_id, unc_here, alt, unc_alt, base_work)
    @staticmethod
    def _q(q):
        qoff, rec, here, alt, there, base = q
        return (np.ascontiguousarray(qoff, np.int64), np.ascontiguousarray(rec, np.uint64),
                np.ascontiguousarray(here, np.uint32), np.ascontiguousarray(alt, np.uint32),
                np.ascontiguousarray(there, np.uint32), np.ascontiguousarray(base, np.int64))

    def _qout(self, n):
        return (np.zeros(self.max_slots + 1, np.int64), np.zeros(max(n, 1), np.uint64),
                np.zeros(max(n, 1), np.uint32), np.zeros(max(n, 1), np.uint32),
                np.zeros(max(n, 1), np.uint32))

    def queue_append(self, q, offsets, cand, match, chosen, rec_base: int):
        """A routed batch joins the queues (or_queue_append)."""
        qoff, rec, here, alt, there, base = self._q(q)
        off = np.ascontiguousarray(offsets, np.int64)
        nb = len(off) - 1
        cand = np.ascontiguousarray(cand, np.uint32)
        match = np.ascontiguousarray(match, np.uint32)
        chosen = np.ascontiguousarray(chosen, np.uint32)
        o = self._qout(int(qoff[-1]) + nb)
        rc = lib().or_queue_append(self._h, _p(qoff), _p(rec), _p(here), _p(alt), _p(there), nb,
                                   _p(off), _p(cand), _p(match), _p(chosen), int(rec_base),
                                   *[_p(x) for x in o])
        if rc != OK:
            raise RuntimeError("or_queue_append failed with status %d" % rc)
        n2 = int(o[0][-1])
        return (o[0], o[1][:n2], o[2][:n2], o[3][:n2], o[4][:n2], base.copy())

    def queue_migrate(self, q, mrec, msrc, mdst):
        """A migration list applied to the queues (or_queue_migrate)."""
        qoff, rec, here, alt, there, base = self._q(q)
        mrec = np.ascontiguousarray(mrec, np.uint64)
        msrc = np.ascontiguousarray(msrc, np.uint32)
        mdst = np.ascontiguousarray(mdst, np.uint32)
        o = self._qout(int(qoff[-1]))
        rc = lib().or_queue_migrate(self._h, _p(qoff), _p(rec), _p(here), _p(alt), _p(there),
                                    len(mrec), _p(mrec), _p(msrc), _p(mdst), *[_p(x) for x in o])
        if rc != OK:
            raise RuntimeError("or_queue_migrate failed with status %d" % rc)
        n2 = int(o[0][-1])
        return (o[0], o[1][:n2], o[2][:n2], o[3][:n2], o[4][:n2], base.copy())

    def queue_reprobe(self, q, coff, keys, plen):
        """Queued records re-priced against the current caches
        (or_queue_reprobe): record id r's chain keys[coff[r]:coff[r+1]], its
        prompt plen[r] tokens."""
        qoff, rec, here, alt, there, base = self._q(q)
        coff = np.ascontiguousarray(coff, np.int64)
        keys = np.ascontiguousarray(keys, np.uint64)
        plen = np.ascontiguousarray(plen, np.int64)
        n = max(len(rec), 1)
        here2, there2 = np.zeros(n, np.uint32), np.zeros(n, np.uint32)
        rc = lib().or_queue_reprobe(self._h, _p(qoff), _p(rec), _p(alt), len(plen), _p(coff),
                                    _p(keys), _p(plen), _p(here2), _p(there2))
        if rc != OK:
            raise RuntimeError("or_queue_reprobe failed with status %d" % rc)
        Q = len(rec)
        return (qoff.copy(), rec.copy(), here2[:Q], alt.copy(), there2[:Q], base.copy())

    def queue_drain(self, q, units):
        """units[i] of service on every instance (or_queue_drain)."""
        qoff, rec, here, alt, there, base = self._q(q)
        units = np.ascontiguousarray(units, np.int64)
        o = self._qout(int(qoff[-1]))
        base2 = np.zeros_like(base)
        rc = lib().or_queue_drain(self._h, _p(qoff), _p(rec), _p(here), _p(alt), _p(there),
                                  _p(base), _p(units), *[_p(x) for x in o], _p(base2))
        if rc != OK:
            raise RuntimeError("or_queue_drain failed with status %d" % rc)
        n2 = int(o[0][-1])
        return (o[0], o[1][:n2], o[2][:n2], o[3][:n2], o[4][:n2], base2)

    def keylen_enable(self, max_nodes: int) -> int:
        """Adaptive hash-key length: an empty prefix hotness tree with room for
        max_nodes extended prefixes (0 turns it off)."""
        return lib().or_keylen_enable(self._h, int(max_nodes))

    def keylen_window(self) -> int:
        """Close the current window: hot leaves extend, cold nodes shrink."""
        return lib().or_keylen_window(self._h)

    def keylen_tree(self) -> np.ndarray:
        """The extended prefixes (canon f1 keys of their last blocks), ascending."""
        n = C.c_uint64()
        lib().or_keylen_export(self._h, None, 0, C.byref(n))
        a = np.zeros(max(int(n.value), 1), np.uint64)
        lib().or_keylen_export(self._h, _p(a), len(a), C.byref(n))
        return a[:int(n.value)]

    def ring_key_at(self, s: int, tokens: np.ndarray, kr: int) -> int:
        t = np.ascontiguousarray(tokens, dtype=np.int32)
        return int(lib().or_ring_key_at(self._h, s, _p(t), int(kr)))

    def build_rings(self, ids: Sequence[int]) -> int:
        a = np.ascontiguousarray(ids, dtype=np.uint32)
        return lib().or_build_rings(self._h, _p(a), len(a))

    def ring(self, s: int):
        n = lib().or_ring_copy(self._h, s, None, None)
        pos = np.zeros(n, dtype=np.uint64)
        ids = np.zeros(n, dtype=np.uint32)
        lib().or_ring_copy(self._h, s, _p(pos), _p(ids))
        return pos, ids

    def n_live(self) -> int:
        return int(lib().or_n_live(self._h))

    def index_insert(self, inst: int, keys: np.ndarray) -> int:
        k = np.ascontiguousarray(keys, dtype=np.uint64)
        return lib().or_index_insert(self._h, inst, _p(k), len(k))

    def index_erase(self, inst: int, keys: np.ndarray) -> int:
        k = np.ascontiguousarray(keys, dtype=np.uint64)
        return lib().or_index_erase(self._h, inst, _p(k), len(k))

    def index_clear(self, inst: int) -> int:
        return lib().or_index_clear(self._h, inst)

    def index_size(self, inst: int) -> int:
        return int(lib().or_index_size(self._h, inst))

    def index_contains(self, inst: int, key: int) -> bool:
        return bool(lib().or_index_contains(self._h, inst, key))

    # -- single-request pieces ----------------------------------------------
    def chain(self, s: int, tokens: np.ndarray) -> np.ndarray:
        t = np.ascontiguousarray(tokens, dtype=np.int32)
        out = np.zeros(len(t) // self.block, dtype=np.uint64)
        n = lib().or_chain(self._h, s, _p(t), len(t), _p(out))
        return out[:n]

    def ring_key(self, s: int, tokens: np.ndarray) -> int:
        t = np.ascontiguousarray(tokens, dtype=np.int32)
        return int(lib().or_ring_key(self._h, s, _p(t), len(t)))

    def vpos(self, s: int, inst: int, v: int) -> int:
        return int(lib().or_vpos(self._h, s, inst, v))

    def owner(self, s: int, x: int) -> int:
        return int(lib().or_owner(self._h, s, x))

    def candidates(self, x1: int, x2: int):
        c1, c2 = C.c_uint32(), C.c_uint32()
        fix = lib().or_candidates(self._h, x1, x2, C.byref(c1), C.byref(c2))
        return int(c1.value), int(c2.value), bool(fix)

    def ttft(self, uncached: int, load: int) -> int:
        return int(lib().or_ttft(self._h, uncached, load))

    def select(self, c1, c2, m1, m2, length, loads: np.ndarray, flags: int = 0):
        L = np.ascontiguousarray(loads, dtype=np.int64)
        t = C.c_int64()
        f = C.c_uint8(flags)
        ch = lib().or_select(self._h, c1, c2, m1, m2, length, _p(L), C.byref(t), C.byref(f))
        return int(ch), int(t.value), int(f.value)

    # -- batch operations ---------------------------------------------------
    def route(self, tokens: np.ndarray, offsets: np.ndarray, loads: np.ndarray,
              block_keys: bool = False) -> Dict[str, np.ndarray]:
        """Route a batch; returns the outputs and the updated loads (the input
        array is not modified)."""
        t = np.ascontiguousarray(tokens, dtype=np.int32)
        o = np.ascontiguousarray(offsets, dtype=np.int64)
        n = len(o) - 1
        L = np.array(loads, dtype=np.int64, copy=True)
        out = dict(key=np.zeros(2 * n, np.uint64), cand=np.zeros(2 * n, np.uint32),
                   match=np.zeros(2 * n, np.uint32), chosen=np.zeros(n, np.uint32),
                   ttft=np.zeros(n, np.int64), flags=np.zeros(n, np.uint8),
                   key_len=np.zeros(n, np.uint32))
        bk = None
        if block_keys:
            nfull = np.diff(o) // self.block
            bk = np.zeros(int(nfull.sum()), np.uint64)
        rc = lib().or_route(self._h, _p(t), _p(o), n, _p(L), _p(out["key"]), _p(out["cand"]),
                            _p(out["match"]), _p(out["chosen"]), _p(out["ttft"]),
                            _p(out["flags"]), _p(bk), _p(out["key_len"]))
        if rc != OK:
            raise RuntimeError("or_route failed with status %d" % rc)
        out["loads"] = L
        if bk is not None:
            out["block_keys"] = bk
        return out

    def rebalance(self, qoff, rec_id, unc_here, alt, unc_alt, base_work, cap: Optional[int] = None,
                  prefill_interval=None, decode_threshold_us: int = 3_000_000):
        qoff = np.ascontiguousarray(qoff, np.int64)
        pint = None if prefill_interval is None else np.ascontiguousarray(prefill_interval, np.int64)
        rec_id = np.ascontiguousarray(rec_id, np.uint64)
        unc_here = np.ascontiguousarray(unc_here, np.uint32)
        alt = np.ascontiguousarray(alt, np.uint32)
        unc_alt = np.ascontiguousarray(unc_alt, np.uint32)
        base_work = np.ascontiguousarray(base_work, np.int64)
        Q = len(rec_id)
        cap = Q if cap is None else cap
        loads = np.zeros(self.max_slots, np.int64)
        m = dict(rec=np.zeros(max(cap, 1), np.uint64), src=np.zeros(max(cap, 1), np.uint32),
                 dst=np.zeros(max(cap, 1), np.uint32), benefit=np.zeros(max(cap, 1), np.int64),
                 ttft_to=np.zeros(max(cap, 1), np.int64))
        cnt = C.c_uint64()
        rc = lib().or_rebalance(self._h, _p(qoff), _p(rec_id), _p(unc_here), _p(alt), _p(unc_alt),
                                _p(base_work), _p(pint) if pint is not None else None,
                                int(decode_threshold_us), _p(loads), _p(m["rec"]), _p(m["src"]),
                                _p(m["dst"]),
                                _p(m["benefit"]), _p(m["ttft_to"]), cap, C.byref(cnt))
        n = int(cnt.value)
        out = {k: v[:min(n, cap)] for k, v in m.items()}
        out["count"] = n
        out["loads"] = loads
        out["status"] = rc
        return out

    def scale(self, add, rm, keys: np.ndarray):
        add = np.ascontiguousarray(add, np.uint32)
        rm = np.ascontiguousarray(rm, np.uint32)
        keys = np.ascontiguousarray(keys, np.uint64)
        n = len(keys) // 2
        old = np.zeros(2 * n, np.uint32)
        new = np.zeros(2 * n, np.uint32)
        moved = np.zeros(2, np.uint64)
        viol = C.c_uint64()
        rc = lib().or_scale(self._h, _p(add), len(add), _p(rm), len(rm), _p(keys), n,
                            _p(old), _p(new), _p(moved), C.byref(viol))
        return dict(status=rc, old=old, new=new, moved=moved, violations=int(viol.value))
