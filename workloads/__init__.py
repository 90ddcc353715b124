"""Seeded synthetic inputs for the DualMap routing path.

This module holds none of the method's arithmetic: it draws token streams,
prompt lengths, template choices, loads, coin flips, random key streams and
queue records with the shapes and distributions of the workloads the routing
path is measured on, and nothing else.  Both the HIP path (tests, benchmark)
and the CPU oracle take their inputs from here; every state that needs the
method's arithmetic (cached block sets built from routed prompts, candidate
pairs, loads after routing) is built by each side with its own code.

The paper measures on two Mooncake traces (Conversation and Tool&Agent,
Table 1 and Sec. A.2.1); those traces are not available, so the generators
below stand in for them: template-plus-suffix prompts with Zipf-distributed
template popularity reproduce the shared-prefix structure, multi-turn
sessions reproduce the conversation structure.

Random streams: numpy's PCG64 seeded by SeedSequence([workload_seed, stream]),
one stream per component, so each component is reproducible on its own.
"""
from __future__ import annotations

import ctypes as C
import dataclasses
import math
import os
import subprocess
from typing import Dict, Optional, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_FG_SRC = os.path.join(_HERE, "_fastgen.c")
_FG_LIB = os.path.join(_HERE, "libfastgen.so")
_fg = None


def build(force: bool = True) -> str:
    """Compile the token-fill helper (gcc, OpenMP)."""
    if force or not os.path.exists(_FG_LIB) or os.path.getmtime(_FG_LIB) < os.path.getmtime(_FG_SRC):
        tmp = _FG_LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O3", "-fopenmp", "-shared", "-fPIC", "-o", tmp, _FG_SRC])
        os.replace(tmp, _FG_LIB)
    return _FG_LIB


def _fastgen():
    global _fg
    if _fg is None:
        build(force=False)
        L = C.CDLL(_FG_LIB)
        L.fg_uniform_tokens.argtypes = [C.c_void_p, C.c_int64, C.c_uint32, C.c_uint64]
        L.fg_uniform_tokens.restype = None
        L.fg_copy_prefixes.argtypes = [C.c_void_p] * 6 + [C.c_int64]
        L.fg_copy_prefixes.restype = None
        _fg = L
    return _fg


def _vp(a: np.ndarray):
    return a.ctypes.data_as(C.c_void_p)

# Stream ids: one independent random stream per generated component.
_S_TEMPLATE_LEN, _S_TEMPLATE_TOK, _S_REQ_LEN, _S_REQ_TPL, _S_REQ_TOK = 1, 2, 3, 4, 5
_S_LOADS, _S_COINS, _S_FILLER, _S_PRIOR, _S_SCALE, _S_QUEUE = 6, 7, 8, 9, 10, 11


def _rng(seed: int, stream: int, sub: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, stream, sub])))


@dataclasses.dataclass(frozen=True)
class RouteConfig:
    """Routing parameters of one workload (passed to both implementations)."""

    name: str
    n_inst: int               # live instances at start (ids 0..n_inst-1)
    vnodes: int               # virtual nodes per instance on each ring
    block: int                # tokens per KV block
    key_blocks: int           # ring key covers the first key_blocks full blocks
    seeds: Tuple[int, int]    # seeds of the two hash functions
    max_slots: int            # instance-id space
    index_log2_slots: int     # per-instance device table: 2**k slots
    ttft_base_us: int = 2000
    ttft_per_token_us: int = 3
    queue_div: int = 4
    slo_us: int = 400_000

    def as_dict(self) -> Dict:
        return dataclasses.asdict(self)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    route: RouteConfig
    seed: int
    n_req: int
    vocab: int
    # prompt lengths
    len_kind: str             # "uniform" | "lognormal"
    len_a: float              # uniform: low;  lognormal: median
    len_b: float              # uniform: high; lognormal: sigma
    len_cap: int
    # shared-prefix templates
    n_templates: int
    tlen_lo: int
    tlen_hi: int
    zipf_s: float
    load_hi: int = 50_000     # initial per-instance load ~ U[0, load_hi]
    n_prior: int = 0          # prior requests whose chains pre-fill the index
    filler_per_inst: int = 0  # random keys topping each instance index up to this size
    suffix_lo: int = 0        # template prompts: random tail ~ U[suffix_lo, suffix_hi]
    suffix_hi: int = 0        #   (0, 0 = prompt length drawn from len_kind instead)


def tiny(slo_us: int = 400_000) -> Workload:
    """8 instances x 64 vnodes, 1,024 requests of U[256,768] tokens over 64
    Zipf(1.0) templates of U[128,512] tokens, vocab 32,000, block 16; the index
    is pre-filled by routing 256 prior requests."""
    rc = RouteConfig("tiny", 8, 64, 16, 4, (1, 2), 8, 14, slo_us=slo_us)
    return Workload("tiny" if slo_us == 400_000 else "tiny-tight", rc, 101, 1024, 32_000,
                    "uniform", 256, 768, 768, 64, 128, 512, 1.0, n_prior=256)


def large(n_req: int = 1_048_576) -> Workload:
    """128 instances x 512 vnodes, 1,048,576 requests with lognormal lengths
    (median 1,024, sigma 1.0, cap 16,384), 4,096 Zipf(1.1) templates of
    U[128,2048] tokens, vocab 152,000, block 16; each instance index holds
    1,048,576 keys in 2**21 slots."""
    rc = RouteConfig("large", 128, 512, 16, 4, (1, 2), 256, 21)
    return Workload("large" if n_req == 1_048_576 else f"large-{n_req}", rc, 104, n_req, 152_000,
                    "lognormal", 1024.0, 1.0, 16_384, 4096, 128, 2048, 1.1,
                    filler_per_inst=1_048_576)


def small_random(seed: int, n_inst: int, vnodes: int, block: int, n_req: int,
                 key_blocks: Optional[int] = None, slo_us: int = 400_000) -> Workload:
    """Small randomized configuration for property and parity sweeps; lengths
    include 0, shorter than a block and exact multiples of the block."""
    kb = key_blocks if key_blocks is not None else max(1, 64 // block)
    rc = RouteConfig(f"rand{seed}", n_inst, vnodes, block, kb, (1 + seed, 2 + seed),
                     max(n_inst, 1) + 3, 12, slo_us=slo_us)
    return Workload(f"rand{seed}", rc, 1000 + seed, n_req, 50,
                    "uniform", 0, 6 * block, 6 * block, 6, 1, 4 * block, 1.0, n_prior=n_req // 2)


# --------------------------------------------------------------------------
# Building blocks
# --------------------------------------------------------------------------

def zipf_ranks(rng: np.random.Generator, n_items: int, s: float, size: int) -> np.ndarray:
    """Item indices 0..n_items-1 with P(k) proportional to (k+1)^-s, via the CDF
    and a 53-bit uniform."""
    w = np.arange(1, n_items + 1, dtype=np.float64) ** (-s)
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    u = rng.random(size)
    idx = np.searchsorted(cdf, u, side="right")
    return np.minimum(idx, n_items - 1).astype(np.int64)


def uniform_tokens(rng: np.random.Generator, vocab: int, size: int) -> np.ndarray:
    """size tokens uniform in [0, vocab), from chunked PCG32 streams seeded by
    one draw of rng."""
    out = np.empty(size, dtype=np.int32)
    if size:
        _fastgen().fg_uniform_tokens(_vp(out), size, vocab, int(rng.integers(0, 2**63)))
    return out


def templates(wl: Workload) -> Tuple[np.ndarray, np.ndarray]:
    """Template token CSR: (tokens int32, offsets int64)."""
    lens = _rng(wl.seed, _S_TEMPLATE_LEN).integers(wl.tlen_lo, wl.tlen_hi + 1, size=wl.n_templates)
    off = np.zeros(wl.n_templates + 1, dtype=np.int64)
    np.cumsum(lens, out=off[1:])
    tok = uniform_tokens(_rng(wl.seed, _S_TEMPLATE_TOK), wl.vocab, int(off[-1]))
    return tok, off


def _lengths(wl: Workload, rng: np.random.Generator, n: int) -> np.ndarray:
    if wl.len_kind == "uniform":
        return rng.integers(int(wl.len_a), int(wl.len_b) + 1, size=n).astype(np.int64)
    z = rng.standard_normal(n)
    lens = np.rint(np.exp(math.log(wl.len_a) + wl.len_b * z))
    return np.minimum(lens, wl.len_cap).astype(np.int64)


def prompts(wl: Workload, n: int, sub: int = 0, chunk: int = 1 << 16) -> Tuple[np.ndarray, np.ndarray]:
    """n prompts: each is the first min(len, T_len) tokens of a Zipf-chosen
    template followed by uniform random tokens up to len.  Returns the token
    CSR (int32 tokens, int64 offsets).  `sub` selects an independent batch
    (0 = measured batch, 1 = prior requests)."""
    ttok, toff = templates(wl)
    tlen = np.diff(toff)
    lens = _lengths(wl, _rng(wl.seed, _S_REQ_LEN, sub), n)
    tpl = zipf_ranks(_rng(wl.seed, _S_REQ_TPL, sub), wl.n_templates, wl.zipf_s, n)
    off = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(lens, out=off[1:])
    total = int(off[-1])
    # random tokens everywhere, then each prompt's shared part overwritten
    # with its template's prefix
    tok = uniform_tokens(_rng(wl.seed, _S_REQ_TOK, sub), wl.vocab, total)
    shared = np.ascontiguousarray(np.minimum(lens, tlen[tpl]), dtype=np.int64)
    _fastgen().fg_copy_prefixes(_vp(tok), _vp(off), _vp(np.ascontiguousarray(tpl)), _vp(shared),
                                _vp(ttok), _vp(toff), n)
    del chunk
    return tok, off


def initial_loads(wl: Workload, n_slots: int) -> np.ndarray:
    """Per-slot pending work U[0, load_hi] (int64)."""
    return _rng(wl.seed, _S_LOADS).integers(0, wl.load_hi + 1, size=n_slots).astype(np.int64)


def coin_flips(wl: Workload, n: int) -> np.ndarray:
    """n fair coins (uint8 0/1)."""
    return _rng(wl.seed, _S_COINS).integers(0, 2, size=n).astype(np.uint8)


def filler_keys(wl: Workload, inst: int, count: int) -> np.ndarray:
    """The first `count` values of instance inst's random 64-bit key stream."""
    if count <= 0:
        return np.zeros(0, dtype=np.uint64)
    return _rng(wl.seed, _S_FILLER, inst).integers(0, 2**64, size=count, dtype=np.uint64)


def scale_sets(wl: Workload, n_add: int, n_rm: int) -> Tuple[np.ndarray, np.ndarray]:
    """Elastic step: add ids n_inst..n_inst+n_add-1, remove n_rm seed-chosen
    ids from 0..n_inst-1."""
    add = np.arange(wl.route.n_inst, wl.route.n_inst + n_add, dtype=np.uint32)
    rm = np.sort(_rng(wl.seed, _S_SCALE).choice(wl.route.n_inst, size=n_rm, replace=False))
    return add, rm.astype(np.uint32)


@dataclasses.dataclass
class Queues:
    """Per-instance pending-request queues in CSR form (head first)."""

    qoff: np.ndarray       # int64 [n_slots + 1]
    rec_id: np.ndarray     # uint64 [Q]
    unc_here: np.ndarray   # uint32 [Q]
    alt: np.ndarray        # uint32 [Q]
    unc_alt: np.ndarray    # uint32 [Q]
    base_work: np.ndarray  # int64 [n_slots]


def synthetic_queues(seed: int, n_slots: int, n_live: int, sources: np.ndarray, per_source: int,
                     unc_hi: int, cold_hi: int, base_src: int = 0) -> Queues:
    """Queues on the given source instances (ids < n_live), each holding
    per_source records whose alternative is a uniformly drawn other live
    instance; uncached tokens ~ U[0, unc_hi] on the alternative and the
    smaller of two such draws on the queue's own instance (it holds more of
    the prefix).  Sources start with base work base_src; the other instances
    get base work U[0, cold_hi] and empty queues."""
    rng = _rng(seed, _S_QUEUE)
    lens = np.zeros(n_slots, dtype=np.int64)
    lens[sources] = per_source
    qoff = np.zeros(n_slots + 1, dtype=np.int64)
    np.cumsum(lens, out=qoff[1:])
    Q = int(qoff[-1])
    owner = np.repeat(np.arange(n_slots), lens)
    alt = rng.integers(0, n_live - 1, size=Q)
    alt = np.where(alt >= owner, alt + 1, alt).astype(np.uint32)
    a = rng.integers(0, unc_hi + 1, size=Q)
    b = rng.integers(0, unc_hi + 1, size=Q)
    here = np.minimum(a, b).astype(np.uint32)
    other = rng.integers(0, unc_hi + 1, size=Q).astype(np.uint32)
    rec = rng.permutation(np.arange(Q, dtype=np.uint64) * 7 + 3).astype(np.uint64)
    base = rng.integers(0, cold_hi + 1, size=n_slots).astype(np.int64)
    base[sources] = base_src
    return Queues(qoff, rec, here, alt, other, base)


# --------------------------------------------------------------------------
# Multi-batch workloads: conversation sessions and agent system prompts.
# They stand in for the Mooncake Conversation and Tool&Agent traces
# (Table 1, Sec. A.2.1): the first reproduces multi-turn prefix reuse, the
# second a few very hot, long shared system prompts.
# --------------------------------------------------------------------------

_S_SESSION_BUDGET, _S_SESSION_TURNS, _S_SESSION_TOK, _S_ARRIVAL = 12, 13, 14, 15
_S_GAPS, _S_AGENT_TPL, _S_AGENT_TAIL, _S_AGENT_TOK, _S_AGENT_HOT = 16, 17, 18, 19, 20


@dataclasses.dataclass(frozen=True)
class Chat:
    """Multi-turn chat: sessions of 1..max_turns user turns; a turn's prompt is
    the first history_cap tokens of the session's earlier turns followed by
    the new turn; sessions arrive by Zipf popularity among those with turns
    left.  A disjoint population of warm_sessions sessions supplies the
    warm-up requests that fill the LRU-bounded indexes."""

    route: RouteConfig
    seed: int = 102
    vocab: int = 128_000
    n_sessions: int = 8192
    warm_sessions: int = 2048
    max_turns: int = 16
    turn_lo: int = 64
    turn_hi: int = 512
    history_cap: int = 8192
    zipf_s: float = 0.9
    n_req: int = 65_536
    n_warm: int = 16_384
    batch: int = 4096
    lru_blocks: int = 200_000
    load_hi: int = 50_000
    drain_per_us: int = 4
    utilisation: float = 0.9


def chat(n_req: int = 65_536, n_warm: int = 16_384) -> Chat:
    """16 instances x 128 vnodes, block 16, K 4, vocab 128,000; 8,192 sessions
    (2,048 more for warm-up), turns U[64,512] tokens, history cap 8,192,
    Zipf 0.9; batches of 4,096; LRU of 200,000 blocks per instance in 2^19-slot
    tables."""
    rc = RouteConfig("chat", 16, 128, 16, 4, (1, 2), 16, 19)
    return Chat(rc, n_req=n_req, n_warm=n_warm)


class ChatStream:
    """Arrivals of one session population (0 = measured, 1 = warm-up) and the
    prompts they carry."""

    def __init__(self, cfg: Chat, population: int):
        self.cfg = cfg
        S = cfg.n_sessions if population == 0 else cfg.warm_sessions
        n = cfg.n_req if population == 0 else cfg.n_warm
        self.pop = population
        self.budget = _rng(cfg.seed, _S_SESSION_BUDGET, population).integers(
            1, cfg.max_turns + 1, size=S)
        self.turn_len = _rng(cfg.seed, _S_SESSION_TURNS, population).integers(
            cfg.turn_lo, cfg.turn_hi + 1, size=(S, cfg.max_turns)).astype(np.int64)
        self.session, self.turn = self._arrivals(S, min(n, int(self.budget.sum())))
        self.n = len(self.session)
        self._tok: Dict[int, np.ndarray] = {}

    def _arrivals(self, S: int, n: int) -> Tuple[np.ndarray, np.ndarray]:
        """Zipf draws over sessions; a draw of a session with no turns left is
        drawn again (rejection), which samples Zipf restricted to the sessions
        with turns left."""
        rng = _rng(self.cfg.seed, _S_ARRIVAL, self.pop)
        used = np.zeros(S, dtype=np.int64)
        parts = []
        got = 0
        while got < n:
            d = zipf_ranks(rng, S, self.cfg.zipf_s, 1 << 20)
            order = np.argsort(d, kind="stable")
            ds = d[order]
            starts = np.r_[0, np.flatnonzero(np.diff(ds)) + 1]
            occ_sorted = np.arange(len(ds)) - np.repeat(starts, np.diff(np.r_[starts, len(ds)]))
            occ = np.empty_like(occ_sorted)
            occ[order] = occ_sorted
            acc = d[(used[d] + occ) < self.budget[d]][: n - got]
            np.add.at(used, acc, 1)
            parts.append(acc)
            got += len(acc)
        ses = np.concatenate(parts) if parts else np.zeros(0, dtype=np.int64)
        # turn index of each arrival = earlier arrivals of its session
        order = np.argsort(ses, kind="stable")
        ss = ses[order]
        starts = np.r_[0, np.flatnonzero(np.diff(ss)) + 1] if len(ss) else np.zeros(0, np.int64)
        occ_sorted = np.arange(len(ss)) - np.repeat(starts, np.diff(np.r_[starts, len(ss)]))
        turn = np.empty_like(occ_sorted)
        turn[order] = occ_sorted
        return ses.astype(np.int64), turn.astype(np.int64)

    def _session_tokens(self, s: int) -> np.ndarray:
        t = self._tok.get(s)
        if t is None:
            total = int(self.turn_len[s, : self.budget[s]].sum())
            t = uniform_tokens(_rng(self.cfg.seed, _S_SESSION_TOK, self.pop * (1 << 20) + s),
                               self.cfg.vocab, total)
            self._tok[s] = t
        return t

    def batch(self, lo: int, hi: int) -> Tuple[np.ndarray, np.ndarray]:
        """Prompts of arrivals lo..hi-1 as a token CSR."""
        parts = []
        for i in range(lo, min(hi, self.n)):
            s, t = int(self.session[i]), int(self.turn[i])
            tok = self._session_tokens(s)
            cum = np.concatenate([[0], np.cumsum(self.turn_len[s, : t + 1])])
            hist = tok[: min(int(cum[t]), self.cfg.history_cap)]
            parts.append(np.concatenate([hist, tok[cum[t]: cum[t + 1]]]))
        off = np.zeros(len(parts) + 1, dtype=np.int64)
        np.cumsum([len(p) for p in parts], out=off[1:])
        tok = np.concatenate(parts).astype(np.int32) if parts else np.zeros(0, np.int32)
        return tok, off


@dataclasses.dataclass(frozen=True)
class Agent:
    """Agent/tool workload: a few long system prompts with Zipf popularity and
    a random tail per request; queued work skewed onto hot_inst instances."""

    route: RouteConfig
    seed: int = 103
    vocab: int = 128_000
    n_templates: int = 32
    tlen_lo: int = 2048
    tlen_hi: int = 8192
    zipf_s: float = 1.3
    tail_lo: int = 128
    tail_hi: int = 1024
    n_req: int = 262_144
    n_warm: int = 16_384
    batch: int = 16_384
    lru_blocks: int = 200_000
    hot_inst: int = 4
    hot_factor: int = 5
    drain_per_us: int = 4
    utilisation: float = 0.9
    # Base queued work per instance.  5 mu / 4 crosses the SLO at 320,000;
    # calibrated to 480,000 so that, with the prefix hotness tree on and one
    # window per batch, at least 10% of the queued records migrate over the
    # 16 rebalancing passes (10.2%; 4.5% with a fixed key length).
    mu: int = 480_000


def agent(n_req: int = 262_144, n_warm: int = 16_384, batch: int = 16_384) -> Agent:
    """32 instances x 256 vnodes, block 32, K 2, vocab 128,000; 32 system
    prompts of U[2,048, 8,192] tokens, Zipf 1.3, tails U[128, 1,024]; batches
    of 16,384; LRU of 200,000 blocks per instance in 2^19-slot tables."""
    rc = RouteConfig("agent", 32, 256, 32, 2, (1, 2), 32, 19)
    return Agent(rc, n_req=n_req, n_warm=n_warm, batch=batch)


def agent_templates(cfg: Agent) -> Tuple[np.ndarray, np.ndarray]:
    lens = _rng(cfg.seed, _S_TEMPLATE_LEN).integers(cfg.tlen_lo, cfg.tlen_hi + 1,
                                                    size=cfg.n_templates)
    off = np.zeros(cfg.n_templates + 1, dtype=np.int64)
    np.cumsum(lens, out=off[1:])
    return uniform_tokens(_rng(cfg.seed, _S_TEMPLATE_TOK), cfg.vocab, int(off[-1])), off


def agent_batch(cfg: Agent, index: int, n: int, warm: bool = False) -> Tuple[np.ndarray, np.ndarray]:
    """n prompts of batch `index` (warm-up batches draw from other streams):
    a Zipf-chosen system prompt followed by a uniform random tail."""
    sub = index + (1 << 16 if warm else 0)
    ttok, toff = agent_templates(cfg)
    tpl = zipf_ranks(_rng(cfg.seed, _S_AGENT_TPL, sub), cfg.n_templates, cfg.zipf_s, n)
    tail = _rng(cfg.seed, _S_AGENT_TAIL, sub).integers(cfg.tail_lo, cfg.tail_hi + 1, size=n)
    tlen = np.diff(toff)[tpl]
    lens = tlen + tail
    off = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(lens, out=off[1:])
    tok = uniform_tokens(_rng(cfg.seed, _S_AGENT_TOK, sub), cfg.vocab, int(off[-1]))
    _fastgen().fg_copy_prefixes(_vp(tok), _vp(off), _vp(np.ascontiguousarray(tpl)),
                                _vp(np.ascontiguousarray(tlen, dtype=np.int64)), _vp(ttok),
                                _vp(toff), n)
    return tok, off


def agent_hot_instances(cfg: Agent, batch: int = 0) -> np.ndarray:
    """The seed-chosen instances whose queued work jumps to hot_factor times
    the mean before batch `batch`'s rebalancing pass."""
    return np.sort(_rng(cfg.seed, _S_AGENT_HOT, batch).choice(cfg.route.n_inst, size=cfg.hot_inst,
                                                              replace=False)).astype(np.int64)


def arrival_gaps(seed: int, n_batches: int, batch: int, mean_gap_us: float) -> np.ndarray:
    """Duration of each batch's arrivals (microseconds): the sum of `batch`
    exponential gaps of mean mean_gap_us (Poisson arrivals)."""
    rng = _rng(seed, _S_GAPS)
    return rng.gamma(batch, mean_gap_us, size=n_batches)


def batch_initial_loads(seed: int, n_slots: int, hi: int) -> np.ndarray:
    """Per-slot queued work U[0, hi] for the multi-batch workloads."""
    return _rng(seed, _S_LOADS).integers(0, hi + 1, size=n_slots).astype(np.int64)


# --------------------------------------------------------------------------
# One measured batch of a multi-batch workload, after its warm-up (for the
# per-configuration rows of the benchmark).
# --------------------------------------------------------------------------

def warmup_batches(cfg):
    """The warm-up requests of a chat or agent workload as a list of token
    CSRs, one per batch of cfg.batch requests."""
    out = []
    if isinstance(cfg, Chat):
        st = ChatStream(cfg, 1)
        for lo in range(0, st.n, cfg.batch):
            out.append(st.batch(lo, lo + cfg.batch))
    else:
        for w in range(0, cfg.n_warm, cfg.batch):
            out.append(agent_batch(cfg, w // cfg.batch, min(cfg.batch, cfg.n_warm - w), warm=True))
    return out


def measured_batch(cfg, b: int = 0):
    """Batch b of the measured requests of a chat or agent workload, and the
    queued work per slot it is routed against when it is the first batch
    (chat: U[0, load_hi]; agent: mu on every live instance)."""
    S = cfg.route.max_slots
    if isinstance(cfg, Chat):
        tok, off = ChatStream(cfg, 0).batch(b * cfg.batch, (b + 1) * cfg.batch)
        return tok, off, batch_initial_loads(cfg.seed, S, cfg.load_hi)
    tok, off = agent_batch(cfg, b, cfg.batch)
    L = np.zeros(S, np.int64)
    L[: cfg.route.n_inst] = cfg.mu
    return tok, off, L
