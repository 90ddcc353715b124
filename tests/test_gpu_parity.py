"""HIP engine vs CPU oracle, element by element, through the C ABI.

Every case builds its starting state on each side with that side's own code
(paper_2602_06502_amd.harness for the engine, oracle.harness for the
oracle) from the same seeded inputs, then compares all outputs bit for bit:
ring arrays, ring keys, candidates, match lengths, chosen instances, TTFTs,
flags, updated loads, block keys, migration lists and remap results.
"""
import sys

import numpy as np
import pytest

import oracle
import oracle.harness as oh
import workloads

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2602_06502_amd as pk
    pk.load_library()  # fails loudly if the library is missing
    oracle.build(force=False)
    yield


def _h():
    import paper_2602_06502_amd.harness as gh
    return gh


def cpu(t):
    return t.cpu().numpy()


def compare_route(g, o, n, with_bk=False):
    for k in ("key", "cand", "match", "chosen", "ttft", "flags"):
        a, b = cpu(g[k]), o[k]
        if not np.array_equal(a, b):
            bad = np.nonzero(a != b)[0]
            raise AssertionError(f"{k}: {len(bad)} mismatches, first at {bad[:5]}: "
                                 f"gpu {a[bad[:5]]} oracle {b[bad[:5]]}")
    if with_bk:
        assert np.array_equal(cpu(g["block_keys"])[:len(o["block_keys"])], o["block_keys"])
    if "key_len" in g:
        assert np.array_equal(cpu(g["key_len"])[:n], o["key_len"]), "key_len"


def run_pair(wl, block_keys=True, n_live=None):
    gh = _h()
    _say("setup", wl.name, wl.route)
    eng = gh.engine_for(wl, n_live=n_live)
    o = oh.oracle_for(wl, n_live=n_live)
    if wl.filler_per_inst:
        gh.prefill_templates(eng, wl)
        oh.prefill_templates(o, wl)
    else:
        gh.prefill_from_prior(eng, wl)
        oh.prefill_from_prior(o, wl)
    tok, off = workloads.prompts(wl, wl.n_req, sub=0)
    L0 = workloads.initial_loads(wl, wl.route.max_slots)
    _say("route", wl.name, "n", wl.n_req, "tokens", len(tok))
    Ld = gh.to_dev(L0, eng.device)
    g = eng.route(gh.to_dev(tok, eng.device), gh.to_dev(off, eng.device), Ld, block_keys=block_keys)
    eng.sync()
    r = o.route(tok, off, L0, block_keys=block_keys)
    compare_route(g, r, wl.n_req, with_bk=block_keys)
    assert np.array_equal(cpu(Ld), r["loads"])
    return eng, o, g, r, tok, off


def test_rings_match_oracle():
    for wl in (workloads.tiny(), workloads.small_random(3, 5, 7, 16, 10)):
        gh = _h()
        eng = gh.engine_for(wl)
        o = oh.oracle_for(wl)
        for s in (0, 1):
            gp, gi = eng.ring(s)
            op, oi = o.ring(s)
            assert np.array_equal(gp, op) and np.array_equal(gi, oi)


def test_tiny_parity():
    eng, o, g, r, tok, off = run_pair(workloads.tiny())
    # Tiny never reaches the SLO knee (every TTFT << 400 ms)
    assert (r["flags"] & 1).sum() == 0
    assert (r["match"] > 0).mean() > 0.2


def test_tiny_tight_parity():
    eng, o, g, r, tok, off = run_pair(workloads.tiny(slo_us=20_000))
    f = r["flags"]
    assert (f & 1).sum() > 0 and (f & 2).sum() > 0  # both SLO branches taken


@pytest.mark.parametrize("seed,n_inst,vnodes,block", [
    (0, 1, 4, 16), (1, 2, 1, 4), (2, 3, 16, 8), (3, 9, 5, 32), (4, 7, 16, 64), (5, 4, 2, 16),
    (6, 5, 9, 4), (7, 8, 16, 16),
])
def test_random_small_parity(seed, n_inst, vnodes, block):
    wl = workloads.small_random(seed, n_inst, vnodes, block, 300 + 37 * seed,
                                slo_us=3_000 if seed % 2 else 400_000)
    run_pair(wl)


def _pair_with_loads(wl, L0, policy=None):
    gh = _h()
    eng = gh.engine_for(wl)
    o = oh.oracle_for(wl)
    if policy is not None:
        eng.set_policy(policy)
        assert o.set_policy(policy) == oracle.OK
    gh.prefill_from_prior(eng, wl)
    oh.prefill_from_prior(o, wl)
    tok, off = workloads.prompts(wl, wl.n_req, sub=0)
    Ld = gh.to_dev(L0, eng.device)
    g = eng.route(gh.to_dev(tok, eng.device), gh.to_dev(off, eng.device), Ld, block_keys=True)
    eng.sync()
    r = o.route(tok, off, L0, block_keys=True)
    compare_route(g, r, wl.n_req, with_bk=True)
    assert np.array_equal(cpu(Ld), r["loads"])
    return r


@pytest.mark.parametrize("n_inst,top", [(8, 0), (150, 0), (200, 0), (8, 1), (150, 1)])
def test_selection_wide_loads_parity(n_inst, top):
    """Loads spread beyond 2^30 take the windowed selection on 64-bit loads;
    a spread beyond 2^62 (top=1) takes the serial 64-bit selection."""
    wl = workloads.small_random(31, n_inst, 3, 16, 700, slo_us=6_000_000_000)
    L0 = workloads.initial_loads(wl, wl.route.max_slots)
    L0[::3] += 1 << 40
    L0[1] = (1 << 62) - (1 << 50) if not top else (1 << 62) + (1 << 50)
    _say("wide loads", n_inst, top)
    r = _pair_with_loads(wl, L0)
    assert (r["flags"] & 1).sum() + (r["flags"] & 4).sum() > 0


@pytest.mark.parametrize("n_inst,wide", [(1, False), (2, False), (2, True), (3, True)])
def test_deep_windows_across_blocks_parity(n_inst, wide):
    """One to three instances over several 1024-request blocks: every level
    holds one pair (one to three requests), so windows alternate many small
    depths between their two lane sets and reach the 64-depth cap (four
    passes of the 16-step block); wide: loads beyond 2^30 (64-bit walk)."""
    wl = workloads.small_random(41 + n_inst, n_inst, 3, 16, 2600, slo_us=400_000)
    L0 = workloads.initial_loads(wl, wl.route.max_slots)
    if wide:
        L0[::2] += 1 << 40
    _say("deep windows", n_inst, wide)
    _pair_with_loads(wl, L0)


@pytest.mark.parametrize("policy", ["cache_affinity", "least_loaded", "min_ttft"])
@pytest.mark.parametrize("n_inst,wide", [(8, 0), (200, 0), (150, 1), (300, 0), (8, 2)])
def test_policy_selection_parity(policy, n_inst, wide):
    """The single-criterion rules of the ablation study (Sec. 4.3) on every
    selection path: the windowed walk on 32-bit loads (8 and 200 instances)
    and on 64-bit loads (spread beyond 2^30), the serial path with loads in
    registers (spread beyond 2^62) and in LDS (300 instances).  The
    minimum-TTFT rule always runs serially."""
    wl = workloads.small_random(61 + n_inst, n_inst, 3, 16, 700,
                                slo_us=6_000_000_000 if wide else 20_000)
    L0 = workloads.initial_loads(wl, wl.route.max_slots)
    if wide:
        L0[::3] += 1 << 40
        L0[1] = (1 << 62) - (1 << 50) if wide == 1 else (1 << 62) + (1 << 50)
    _say("policy", policy, n_inst, wide)
    r = _pair_with_loads(wl, L0, policy)
    fewer = (r["flags"] & 1) != 0
    if policy == "cache_affinity":
        assert not fewer.any()
    else:
        assert fewer.any()


def test_policy_changes_between_pipelined_batches():
    """The rule is taken when a batch is routed: pipelined batches under
    different rules, each against the oracle under the same rule in order."""
    gh = _h()
    wl = workloads.tiny(slo_us=20_000)
    eng, o = gh.engine_for(wl), oh.oracle_for(wl)
    gh.prefill_from_prior(eng, wl)
    oh.prefill_from_prior(o, wl)
    tok, off = workloads.prompts(wl, wl.n_req, sub=0)
    L0 = workloads.initial_loads(wl, wl.route.max_slots)
    Ld = gh.to_dev(L0, eng.device)
    td, od = gh.to_dev(tok, eng.device), gh.to_dev(off, eng.device)
    eng.set_pipelining(True)
    outs = []
    seq = ["least_loaded", "slo_aware", "min_ttft", "cache_affinity", "slo_aware"]
    for pol in seq:
        eng.set_policy(pol)
        outs.append(eng.route(td, od, Ld))
    eng.sync()
    eng.set_pipelining(False)
    L = L0.copy()
    for pol, g in zip(seq, outs):
        assert o.set_policy(pol) == oracle.OK
        r = o.route(tok, off, L)
        compare_route(g, r, wl.n_req)
        L = r["loads"]
    assert np.array_equal(cpu(Ld), L)
    o.set_policy("slo_aware")


def test_policy_rejects_unknown_rule():
    gh = _h()
    import paper_2602_06502_amd as pk
    eng = gh.engine_for(workloads.tiny())
    for bad in (-1, 4, 99):
        with pytest.raises(pk.DMError) as ei:
            eng.set_policy(bad)
        assert ei.value.status == pk.DM_EINVAL


# ---------------------------------------------------------------------------
# Adaptive hash-key length (prefix hotness tree)
# ---------------------------------------------------------------------------

def _hot_batches(seed, B, K, n_batches, tlen_blocks=(1, 40), n_tpl=8, zipf=1.3):
    """Batches of prompts over Zipf-popular templates (whole templates or
    cut past depth K, then a random tail): hot templates extend their keys
    window by window, long ones past a 64-block chunk."""
    rng = np.random.default_rng(seed)
    tpl = [rng.integers(0, 1 << 20, size=B * int(rng.integers(K + tlen_blocks[0], K + tlen_blocks[1])),
                        dtype=np.int32) for _ in range(n_tpl)]
    w = 1.0 / np.arange(1, n_tpl + 1) ** zipf
    w /= w.sum()
    out = []
    for _ in range(n_batches):
        ps = []
        for _ in range(int(rng.integers(200, 700))):
            if rng.random() < 0.15:
                ps.append(rng.integers(0, 1 << 20, size=int(rng.integers(0, 8 * B)), dtype=np.int32))
                continue
            t = tpl[int(rng.choice(n_tpl, p=w))]
            cut = int(rng.integers(K * B, len(t) + 1))
            ps.append(np.concatenate([t[:cut], rng.integers(0, 1 << 20, size=int(rng.integers(0, 4 * B)),
                                                            dtype=np.int32)]))
        off = np.zeros(len(ps) + 1, np.int64)
        off[1:] = np.cumsum([len(p) for p in ps])
        out.append((np.concatenate(ps) if ps else np.zeros(0, np.int32), off))
    return out


@pytest.mark.parametrize("B,K,n_inst,pipelined", [(16, 4, 8, False), (4, 60, 12, True),
                                                  (32, 2, 32, False), (64, 3, 10, True),
                                                  (8, 1, 16, False)])
def test_keylen_windows_parity(B, K, n_inst, pipelined):
    """Every batch one window: key lengths, ring keys and all routing outputs
    per batch, and the tree after every window, against the oracle.  With
    K = 60 the paths cross the extension walk's 64-block chunk boundary as
    the tree deepens; short and empty prompts sit below the roots."""
    gh = _h()
    wl = workloads.small_random(71 + B, n_inst, 8, B, 64, slo_us=30_000, key_blocks=K)
    eng, o = gh.engine_for(wl), oh.oracle_for(wl)
    eng.keylen_enable(4096, 1 << 20)
    assert o.keylen_enable(4096) == oracle.OK
    if pipelined:
        eng.set_pipelining(True)
    L0 = workloads.initial_loads(wl, wl.route.max_slots)
    Ld = gh.to_dev(L0, eng.device)
    L = L0.copy()
    deepest = 0
    batches = _hot_batches(5 + B, B, K, 14, tlen_blocks=(1, 90))
    for i, (tok, off) in enumerate(batches):
        _say("keylen window", B, K, n_inst, i, "requests", len(off) - 1)
        g = eng.route(gh.to_dev(tok, eng.device), gh.to_dev(off, eng.device), Ld)
        eng.keylen_window()
        r = o.route(tok, off, L)
        assert o.keylen_window() == oracle.OK
        L = r["loads"]
        compare_route(g, r, len(off) - 1)
        assert np.array_equal(eng.keylen_tree(), o.keylen_tree()), f"tree after window {i}"
        deepest = max(deepest, int(r["key_len"].max()))
    assert np.array_equal(cpu(Ld), L)
    assert deepest > K + 1, deepest
    if K + 14 > 64:
        assert deepest > 64, deepest
    eng.set_pipelining(False)


def test_keylen_window_spans_batches_and_errors():
    """Windows of several batches (pipelined), the record and tree limits,
    and the tree turned off."""
    gh = _h()
    import paper_2602_06502_amd as pk
    B, K = 16, 2
    wl = workloads.small_random(81, 6, 8, B, 64, slo_us=30_000, key_blocks=K)
    eng, o = gh.engine_for(wl), oh.oracle_for(wl)
    batches = _hot_batches(9, B, K, 9)
    L0 = workloads.initial_loads(wl, wl.route.max_slots)
    with pytest.raises(pk.DMError) as ei:
        eng.keylen_window()
    assert ei.value.status == pk.DM_ESTATE
    eng.keylen_enable(1024, 1 << 20)
    o.keylen_enable(1024)
    eng.set_pipelining(True)
    Ld, L = gh.to_dev(L0, eng.device), L0.copy()
    for i, (tok, off) in enumerate(batches):
        n = len(off) - 1
        _say("keylen multi-batch window", i, "requests", n)
        g = eng.route(gh.to_dev(tok, eng.device), gh.to_dev(off, eng.device), Ld)
        r = o.route(tok, off, L)
        L = r["loads"]
        if i % 3 == 2:  # three batches per window
            eng.keylen_window()
            assert o.keylen_window() == oracle.OK
            assert np.array_equal(eng.keylen_tree(), o.keylen_tree()), i
        eng.sync()
        compare_route(g, r, n)
    eng.set_pipelining(False)
    assert np.array_equal(cpu(Ld), L)
    assert len(o.keylen_tree()) > 0
    # a tree too small for the next window's hot prefixes: DM_EFULL, unchanged
    eng.keylen_enable(2, 1 << 20)
    assert o.keylen_enable(2) == oracle.OK
    for tok, off in batches[:2]:
        eng.route(gh.to_dev(tok, eng.device), gh.to_dev(off, eng.device), Ld)
        o.route(tok, off, L)
    assert o.keylen_window() == oracle.EFULL
    with pytest.raises(pk.DMError) as ei:
        eng.keylen_window()
    assert ei.value.status == pk.DM_EFULL
    assert len(eng.keylen_tree()) == 0 == len(o.keylen_tree())
    # prefixes past the record's room: reported by dm_sync, and the close
    # leaves the tree unchanged
    eng.keylen_enable(64, 16)
    td, od = gh.to_dev(batches[0][0], eng.device), gh.to_dev(batches[0][1], eng.device)
    eng.route(td, od, Ld)
    with pytest.raises(pk.DMError) as ei:
        eng.sync()
    assert ei.value.status == pk.DM_EFULL
    with pytest.raises(pk.DMError) as ei:
        eng.keylen_window()
    assert ei.value.status == pk.DM_EFULL
    assert len(eng.keylen_tree()) == 0
    eng.keylen_enable(0)
    with pytest.raises(pk.DMError):
        eng.keylen_tree()


def test_keylen_close_without_hot_roots_and_after_overflow():
    """Window closes that keep nothing (distinct random prompts: no root is
    carried by W / n requests; prompts shorter than K blocks: no record
    entries) after a window that built a tree, and a normal window after
    one whose record overflowed: the trees against the oracle's."""
    gh = _h()
    import paper_2602_06502_amd as pk
    B, K = 16, 2
    wl = workloads.small_random(83, 6, 8, B, 64, key_blocks=K)
    eng, o = gh.engine_for(wl), oh.oracle_for(wl)
    L = workloads.initial_loads(wl, wl.route.max_slots)
    d = lambda a: gh.to_dev(a, eng.device)
    rng = np.random.default_rng(17)

    def window(tok, off):
        eng.route(d(tok), d(off), d(L))
        o.route(tok, off, L)
        eng.keylen_window()
        assert o.keylen_window() == oracle.OK
        t = eng.keylen_tree()
        assert np.array_equal(t, o.keylen_tree())
        return t

    def random_batch(n, lo, hi):
        lens = rng.integers(lo, hi, size=n)
        off = np.zeros(n + 1, np.int64)
        off[1:] = np.cumsum(lens)
        return rng.integers(0, 1 << 20, size=int(off[-1])).astype(np.int32), off

    eng.keylen_enable(1024, 1 << 20)
    o.keylen_enable(1024)
    hot = _hot_batches(19, B, K, 2)
    assert len(window(*hot[0])) > 0
    _say("keylen: a window of distinct prompts")
    assert len(window(*random_batch(500, 4 * B, 30 * B))) == 0
    assert len(window(*hot[1])) > 0
    _say("keylen: a window of prompts shorter than K blocks")
    assert len(window(*random_batch(300, 0, K * B))) == 0
    # a window whose record overflows (the close fails, the tree and the
    # window start over), then a window that fits, on the same context
    tok1, off1 = hot[1]
    m = 40
    small = (tok1[:off1[m]], off1[:m + 1])
    cap = int(np.maximum(np.diff(small[1]) // B - K + 1, 0).sum())
    eng.keylen_enable(1024, cap)
    assert o.keylen_enable(1024) == oracle.OK
    tok, off = hot[0]
    eng.route(d(tok), d(off), d(L))
    with pytest.raises(pk.DMError) as ei:
        eng.sync()
    assert ei.value.status == pk.DM_EFULL
    with pytest.raises(pk.DMError):
        eng.keylen_window()
    _say("keylen: a window after an overflowed one, record of", cap)
    assert len(window(*small)) > 0


# ---------------------------------------------------------------------------
# KV save with LRU eviction
# ---------------------------------------------------------------------------

def test_kv_save_parity_and_errors():
    """Batches over hot templates routed, then saved on the chosen
    instances with a small cap (evictions every batch), each side on its
    own state: added and removed counts, index sizes and the next batch's
    routing (which reads the caches) against the oracle; then bad inputs."""
    gh = _h()
    import paper_2602_06502_amd as pk
    B, K = 16, 2
    wl = workloads.small_random(95, 8, 8, B, 64, slo_us=30_000, key_blocks=K)
    eng, o = gh.engine_for(wl), oh.oracle_for(wl)
    L = workloads.initial_loads(wl, wl.route.max_slots)
    clock, cap = 0, 300
    for i, (tok, off) in enumerate(_hot_batches(96, B, K, 8, tlen_blocks=(1, 30))):
        _say("kv save batch", i, "requests", len(off) - 1)
        Ld = gh.to_dev(L, eng.device)
        g = eng.route(gh.to_dev(tok, eng.device), gh.to_dev(off, eng.device), Ld, block_keys=True)
        eng.sync()
        r = o.route(tok, off, L, block_keys=True)
        compare_route(g, r, len(off) - 1, with_bk=True)
        L = r["loads"]
        ga = eng.kv_save(gh.to_dev(off, eng.device), g["block_keys"], g["chosen"], clock, cap)
        rc, a, rm = o.kv_save(off, r["block_keys"], r["chosen"], clock, cap)
        assert rc == oracle.OK and ga == (a, rm), (ga, a, rm)
        clock += int((np.diff(off) // B).sum())
        for c in range(wl.route.n_inst):
            assert eng.index_size(c) == o.index_size(c) <= cap
    assert rm > 0
    tok, off = _hot_batches(96, B, K, 1)[0]
    bad_inst = gh.to_dev(np.full(len(off) - 1, wl.route.max_slots, np.uint32), eng.device)
    nb = int((np.diff(off) // B).sum())
    keys = gh.to_dev(np.arange(max(nb, 1), dtype=np.uint64), eng.device)
    with pytest.raises(pk.DMError) as ei:
        eng.kv_save(gh.to_dev(off, eng.device), keys, bad_inst, clock, cap)
    assert ei.value.status == pk.DM_EINVAL
    with pytest.raises(pk.DMError) as ei:
        eng.kv_save(gh.to_dev(off, eng.device), keys, gh.to_dev(np.zeros(len(off) - 1, np.uint32),
                                                               eng.device), clock, 1 << 20)
    assert ei.value.status == pk.DM_EINVAL
    # clearing an instance drops its saved keys from the record too
    eng.index_clear(0)
    o.index_clear(0)
    assert eng.index_size(0) == 0 == o.index_size(0)


def _q_eq(g, o, what):
    names = ("qoff", "rec_id", "unc_here", "alt", "unc_alt", "base_work")
    for name, a, b in zip(names, g, o):
        a = cpu(a)
        assert a.shape == b.shape and np.array_equal(a, b), f"{what}: {name}"


@pytest.mark.parametrize("seed,n_inst,batch", [(0, 6, 40), (1, 60, 3000), (2, 200, 9000)])
def test_queue_operations_parity(seed, n_inst, batch):
    """Routed batches appended, random migration lists applied and random
    service drained, on the device queues and on the oracle's, compared
    after every operation; the batches span several blocks of the kernels,
    include empty prompts, an empty batch and an empty migration list."""
    gh = _h()
    B = 16
    wl = workloads.small_random(97 + seed, n_inst, 4, B, 8)
    eng, o = gh.engine_for(wl), oh.oracle_for(wl)
    S = wl.route.max_slots
    d = lambda a: gh.to_dev(a, eng.device)
    rng = np.random.default_rng(400 + seed)
    base = rng.integers(0, 5000, size=S).astype(np.int64)
    qo = (np.zeros(S + 1, np.int64), np.zeros(0, np.uint64), np.zeros(0, np.uint32),
          np.zeros(0, np.uint32), np.zeros(0, np.uint32), base)
    qg = tuple(d(x) for x in qo)
    rec_base = 0
    for step in range(6):
        nb = 0 if step == 2 else int(rng.integers(1, batch))
        _say("queue ops step", step, "batch", nb, "queued", int(qo[0][-1]))
        lens = rng.integers(0, 40 * B, size=nb)
        lens[rng.random(nb) < 0.05] = 0
        off = np.zeros(nb + 1, np.int64)
        off[1:] = np.cumsum(lens)
        c1 = rng.integers(0, n_inst, size=nb)
        c2 = (c1 + rng.integers(1, n_inst, size=nb)) % n_inst
        cand = np.concatenate([c1, c2]).astype(np.uint32)
        match = np.concatenate([rng.integers(0, 1 + lens // B), rng.integers(0, 1 + lens // B)])
        match = match.astype(np.uint32)
        chosen = np.where(rng.random(nb) < 0.5, c1, c2).astype(np.uint32)
        routed = {"key": None, "ttft": None, "flags": None,
                  "cand": d(cand), "match": d(match), "chosen": d(chosen)}
        qg = eng.queue_append(qg, d(off), routed, rec_base)
        qo = o.queue_append(qo, off, cand, match, chosen, rec_base)
        _q_eq(qg, qo, "append")
        rec_base += nb
        Q = int(qo[0][-1])
        k = 0 if step == 3 else min(Q, int(rng.integers(0, max(2, Q // 4))))
        pick = rng.choice(Q, size=k, replace=False) if k else np.zeros(0, np.int64)
        owner = np.searchsorted(qo[0], np.arange(Q), side="right") - 1
        mrec, msrc, mdst = qo[1][pick], owner[pick].astype(np.uint32), qo[3][pick]
        qg = eng.queue_migrate(qg, d(mrec), d(msrc), d(mdst))
        qo = o.queue_migrate(qo, mrec, msrc, mdst)
        _q_eq(qg, qo, "migrate")
        units = rng.integers(0, 20_000, size=S).astype(np.int64)
        units[rng.random(S) < 0.2] = 0
        qg = eng.queue_drain(qg, d(units))
        qo = o.queue_drain(qo, units)
        _q_eq(qg, qo, "drain")


def test_queue_operations_errors():
    """Bad inputs are rejected, nothing written: a chosen id out of range, a
    migration of a record that is not on its source, a record listed twice,
    negative service."""
    gh = _h()
    import paper_2602_06502_amd as pk
    wl = workloads.small_random(99, 6, 4, 16, 8)
    eng = gh.engine_for(wl)
    S = wl.route.max_slots
    d = lambda a: gh.to_dev(a, eng.device)
    q = (d(np.array([0] + [2] * S, np.int64)), d(np.array([5, 6], np.uint64)),
         d(np.array([3, 4], np.uint32)), d(np.array([1, 1], np.uint32)),
         d(np.array([7, 8], np.uint32)), d(np.zeros(S, np.int64)))
    off = np.array([0, 16], np.int64)
    routed = {"key": None, "ttft": None, "flags": None, "cand": d(np.array([0, 1], np.uint32)),
              "match": d(np.zeros(2, np.uint32)), "chosen": d(np.array([S], np.uint32))}
    cases = [
        lambda: eng.queue_append(q, d(off), routed, 10),
        lambda: eng.queue_migrate(q, d(np.array([5], np.uint64)), d(np.array([1], np.uint32)),
                                  d(np.array([2], np.uint32))),
        lambda: eng.queue_migrate(q, d(np.array([5, 5], np.uint64)),
                                  d(np.array([0, 0], np.uint32)), d(np.array([1, 1], np.uint32))),
        lambda: eng.queue_migrate(q, d(np.array([5], np.uint64)), d(np.array([0], np.uint32)),
                                  d(np.array([S], np.uint32))),
        lambda: eng.queue_drain(q, d(np.full(S, -1, np.int64))),
    ]
    for i, f in enumerate(cases):
        _say("queue error case", i)
        with pytest.raises(pk.DMError) as ei:
            f()
        assert ei.value.status == pk.DM_EINVAL, i
    # the valid forms of the same calls go through
    g = eng.queue_migrate(q, d(np.array([6], np.uint64)), d(np.array([0], np.uint32)),
                          d(np.array([1], np.uint32)))
    assert cpu(g[0]).tolist()[:3] == [0, 1, 2] and cpu(g[1]).tolist() == [5, 6]
    assert cpu(g[2]).tolist() == [3, 8] and cpu(g[3]).tolist() == [1, 0]


def test_queue_reprobe_parity_and_errors():
    """Queues built from routed batches over long hot templates (chains past
    several 64-block chunks); between batches the served chains are saved on
    the chosen instances and some on the alternatives, so queued records'
    cached prefixes change; the re-probed queues against the oracle's after
    every batch and after a migration; then bad chain stores."""
    gh = _h()
    import paper_2602_06502_amd as pk
    B, K = 16, 2
    wl = workloads.small_random(98, 8, 8, B, 8, key_blocks=K)
    eng, o = gh.engine_for(wl), oh.oracle_for(wl)
    S = wl.route.max_slots
    d = lambda a: gh.to_dev(a, eng.device)
    rng = np.random.default_rng(77)
    L = workloads.initial_loads(wl, S)
    qo = (np.zeros(S + 1, np.int64), np.zeros(0, np.uint64), np.zeros(0, np.uint32),
          np.zeros(0, np.uint32), np.zeros(0, np.uint32), np.zeros(S, np.int64))
    qg = tuple(d(x) for x in qo)
    coff, keys, plen = [0], [], []
    for i, (tok, off) in enumerate(_hot_batches(98, B, K, 4, tlen_blocks=(1, 200))):
        n = len(off) - 1
        _say("reprobe batch", i, "requests", n)
        g = eng.route(d(tok), d(off), d(L), block_keys=True)
        eng.sync()
        r = o.route(tok, off, L, block_keys=True)
        compare_route(g, r, n, with_bk=True)
        L = r["loads"]
        rb = len(plen)
        qg = eng.queue_append(qg, d(off), g, rb)
        qo = o.queue_append(qo, off, r["cand"], r["match"], r["chosen"], rb)
        _q_eq(qg, qo, "append")
        lens = np.diff(off)
        nf = lens // B
        coff += (coff[-1] + np.cumsum(nf)).tolist()
        keys.append(r["block_keys"])
        plen += lens.tolist()
        bo = np.concatenate([[0], np.cumsum(nf)])
        # served chains saved on the chosen instance, a third also on the other
        other = np.where(r["chosen"] == r["cand"][:n], r["cand"][n:], r["cand"][:n])
        extra = rng.random(n) < 0.33
        for c in range(S):
            for sel in (r["chosen"] == c, (other == c) & extra):
                ks = [r["block_keys"][bo[j]:bo[j + 1]] for j in np.nonzero(sel)[0]]
                if ks:
                    kk = np.concatenate(ks)
                    eng.index_insert(c, d(kk))
                    o.index_insert(c, kk)
        K_all = np.concatenate(keys)
        co, pl = np.array(coff, np.int64), np.array(plen, np.int64)
        qg = eng.queue_reprobe(qg, d(co), d(K_all), d(pl))
        qo = o.queue_reprobe(qo, co, K_all, pl)
        _q_eq(qg, qo, "reprobe")
        Q = int(qo[0][-1])
        pick = rng.choice(Q, size=Q // 5, replace=False)
        owner = np.searchsorted(qo[0], np.arange(Q), side="right") - 1
        mrec, msrc, mdst = qo[1][pick], owner[pick].astype(np.uint32), qo[3][pick]
        qg = eng.queue_migrate(qg, d(mrec), d(msrc), d(mdst))
        qo = o.queue_migrate(qo, mrec, msrc, mdst)
        qg = eng.queue_reprobe(qg, d(co), d(K_all), d(pl))
        qo = o.queue_reprobe(qo, co, K_all, pl)
        _q_eq(qg, qo, "reprobe after migrate")
    assert max(np.diff(co)) > 128
    bad = [
        (co[:-1], pl[:-1]),                       # the last id has no chain
        (co, np.where(np.diff(co) > 0, B * np.diff(co) - 1, pl)),  # chains longer than prompts
        (co + 1, pl),                             # the last chain runs past the keys
    ]
    for j, (c2, p2) in enumerate(bad):
        _say("reprobe error case", j)
        with pytest.raises(pk.DMError) as ei:
            eng.queue_reprobe(qg, d(np.asarray(c2, np.int64)), d(K_all),
                              d(np.asarray(p2, np.int64)))
        assert ei.value.status == pk.DM_EINVAL, j


def test_kv_save_runs_and_lower_cap_parity():
    """KV saves whose batches send one key many times to one instance (long
    runs of equal keys), record entries touched again, and a lowered cap on
    a later save that sends some instances nothing: counts and index sizes
    against the oracle after every save, then a route that reads the
    caches."""
    gh = _h()
    B, K = 16, 2
    wl = workloads.small_random(91, 6, 8, B, 8, key_blocks=K)
    eng, o = gh.engine_for(wl), oh.oracle_for(wl)
    S = wl.route.max_slots
    d = lambda a: gh.to_dev(a, eng.device)
    rng = np.random.default_rng(5)
    clock = 0
    for step, (cap, n_inst) in enumerate([(0, 6), (400, 6), (400, 2), (150, 1), (0, 3)]):
        tok, off = _hot_batches(200 + step, B, K, 1, tlen_blocks=(1, 60), n_tpl=3, zipf=2.0)[0]
        n = len(off) - 1
        bk = o.route(tok, off, workloads.initial_loads(wl, S), block_keys=True)["block_keys"]
        inst = rng.integers(0, n_inst, size=n).astype(np.uint32)
        _say("kv save step", step, "cap", cap, "instances", n_inst, "requests", n)
        ga = eng.kv_save(d(off), d(bk), d(inst), clock, cap)
        rc, a, rm = o.kv_save(off, bk, inst, clock, cap)
        assert rc == oracle.OK and ga == (a, rm), (step, ga, a, rm)
        clock += int((np.diff(off) // B).sum())
        for c in range(S):
            assert eng.index_size(c) == o.index_size(c), (step, c)
    tok, off = _hot_batches(299, B, K, 1, tlen_blocks=(1, 60), n_tpl=3, zipf=2.0)[0]
    L = workloads.initial_loads(wl, S)
    g = eng.route(d(tok), d(off), d(L), block_keys=True)
    eng.sync()
    compare_route(g, o.route(tok, off, L, block_keys=True), len(off) - 1, with_bk=True)


def _disjoint_pair_prompts(o, rng, n_pool):
    """Random prompts whose candidate pairs are pairwise disjoint (greedy
    over a pool), found with the oracle's ring keys and candidates."""
    used, out = set(), []
    for _ in range(n_pool):
        p = rng.integers(0, 1 << 20, size=int(rng.integers(8, 160)), dtype=np.int32)
        c1, c2, _ = o.candidates(o.ring_key(0, p), o.ring_key(1, p))
        if c1 == c2 or c1 in used or c2 in used:
            continue
        used |= {c1, c2}
        out.append(p)
    return out


@pytest.mark.parametrize("wide,big", [(False, False), (True, False), (False, True)])
def test_levels_above_64_requests_parity(wide, big):
    """Levels of more than 64 requests: prompts with pairwise disjoint
    candidate pairs over 200 instances, each sent twice in a row in three
    rounds, so that consecutive same-pair requests form runs (of three, then
    of three again) and a dependency level holds far more than 64 requests.
    The packing cuts each such level into parts of at most 64 requests, one
    depth each, and must keep every run whole.  Random prompts follow,
    across the next request block.  wide: loads spread beyond 2^30 (64-bit
    walk).  big: the same 1,100 requests repeated past 512 Ki requests, so
    that the selection takes its blocks of 2048 requests."""
    gh = _h()
    wl = workloads.small_random(33, 200, 3, 16, 64, slo_us=5_000)
    eng, o = gh.engine_for(wl), oh.oracle_for(wl)
    rng = np.random.default_rng(33)
    uniq = _disjoint_pair_prompts(o, rng, 4000)
    assert len(uniq) >= 40, len(uniq)
    seq = []
    for _ in range(3):
        for p in uniq:
            seq += [p, p]
    assert 2 * len(uniq) > 64
    # each side caches the prompts' chains where a prior routing of them
    # (zero loads) sends them, so that matches differ between candidates
    uoff = np.zeros(len(uniq) + 1, np.int64)
    uoff[1:] = np.cumsum([len(p) for p in uniq])
    utok = np.concatenate(uniq).astype(np.int32)
    zero = np.zeros(wl.route.max_slots, np.int64)
    pr = o.route(utok, uoff, zero, block_keys=True)
    oh.insert_blocks(o, pr["block_keys"], np.repeat(pr["chosen"], np.diff(uoff) // wl.route.block))
    uoff_d = gh.to_dev(uoff, eng.device)
    pg = eng.route(gh.to_dev(utok, eng.device), uoff_d, gh.to_dev(zero, eng.device),
                   block_keys=True)
    gh.insert_blocks(eng, pg["block_keys"],
                     torch.repeat_interleave(pg["chosen"].to(torch.int64), gh.full_blocks(eng, uoff_d)))
    eng.sync()
    for _ in range(1100 - len(seq)):
        seq.append(rng.integers(0, 1 << 20, size=int(rng.integers(0, 120)), dtype=np.int32))
    if big:
        seq = seq * -(-600_000 // len(seq))
    off = np.zeros(len(seq) + 1, np.int64)
    off[1:] = np.cumsum([len(p) for p in seq])
    tok = np.concatenate(seq).astype(np.int32)
    L0 = workloads.initial_loads(wl, wl.route.max_slots)
    if wide:
        L0[::3] += 1 << 40
    _say("levels above 64", len(uniq), "pairs", len(seq), "requests", "wide" if wide else "")
    Ld = gh.to_dev(L0, eng.device)
    g = eng.route(gh.to_dev(tok, eng.device), gh.to_dev(off, eng.device), Ld)
    eng.sync()
    r = o.route(tok, off, L0)
    compare_route(g, r, len(seq))
    assert np.array_equal(cpu(Ld), r["loads"])
    # the affine-candidate rule ran, with SLO switches among its decisions
    assert ((r["flags"] >> 2) & 1).sum() < len(seq) and (r["flags"] & 1).sum() > 0


def test_selection_many_instances_parity():
    """More live instances than the register banks hold (LDS selection)."""
    wl = workloads.small_random(32, 300, 2, 16, 900, slo_us=30_000)
    L0 = workloads.initial_loads(wl, wl.route.max_slots)
    _say("300 instances")
    _pair_with_loads(wl, L0)


def test_sparse_live_ids_parity():
    # ids 0..n-1 not all live: fixup must take the next live id
    wl = workloads.small_random(11, 6, 3, 16, 400)
    gh = _h()
    eng = gh.DualMap(wl.route.as_dict(), device="cuda:0")
    o = oracle.Oracle(wl.route.as_dict())
    ids = [0, 2, 5, 8]
    eng.build_rings(ids)
    o.build_rings(ids)
    tok, off = workloads.prompts(wl, wl.n_req)
    L0 = workloads.initial_loads(wl, wl.route.max_slots)
    Ld = gh.to_dev(L0, eng.device)
    g = eng.route(gh.to_dev(tok, eng.device), gh.to_dev(off, eng.device), Ld)
    eng.sync()
    r = o.route(tok, off, L0)
    compare_route(g, r, wl.n_req)
    assert (r["flags"] & 8).sum() > 0
    assert set(np.unique(r["cand"]).tolist()) <= set(ids)


def test_long_prompts_cross_chunks():
    """Prompts spanning many 64-block chunks, with cached prefixes ending
    inside, at and across chunk boundaries (ragged tails included)."""
    gh = _h()
    B = 16
    cfg = dict(block=B, key_blocks=4, seeds=(7, 9), vnodes=8, max_slots=4, index_log2_slots=14)
    eng = gh.DualMap(cfg, device="cuda:0")
    o = oracle.Oracle(cfg)
    eng.build_rings([0, 1, 2, 3])
    o.build_rings([0, 1, 2, 3])
    rng = np.random.default_rng(5)
    base = rng.integers(0, 1000, size=B * 300).astype(np.int32)
    # cache the first 200 blocks of `base` on every instance
    keys = o.chain(0, base[:200 * B])
    for c in range(4):
        eng.index_insert(c, gh.to_dev(keys, eng.device))
        o.index_insert(c, keys)
    prompts = []
    for cut in (0, 1, 63, 64, 65, 127, 128, 129, 199, 200, 250):
        for extra in (0, 5, B * 70 + 3):
            p = np.concatenate([base[:cut * B], rng.integers(2000, 3000, size=extra).astype(np.int32)])
            prompts.append(p)
    off = np.zeros(len(prompts) + 1, np.int64)
    off[1:] = np.cumsum([len(p) for p in prompts])
    tok = np.concatenate(prompts)
    L0 = rng.integers(0, 1000, size=4).astype(np.int64)
    Ld = gh.to_dev(L0, eng.device)
    g = eng.route(gh.to_dev(tok, eng.device), gh.to_dev(off, eng.device), Ld, block_keys=True)
    eng.sync()
    r = o.route(tok, off, L0, block_keys=True)
    compare_route(g, r, len(prompts), with_bk=True)
    assert np.array_equal(cpu(Ld), r["loads"])


def test_edge_cases_and_errors():
    gh = _h()
    import paper_2602_06502_amd as pk
    cfg = dict(block=16, key_blocks=4, seeds=(1, 2), vnodes=4, max_slots=4, index_log2_slots=10)
    eng = gh.DualMap(cfg, device="cuda:0")
    dev = eng.device
    L = torch.zeros(4, dtype=torch.int64, device=dev)
    # routing before rings exist
    with pytest.raises(pk.DMError) as ei:
        eng.route(torch.zeros(4, dtype=torch.int32, device=dev),
                  torch.tensor([0, 4], dtype=torch.int64, device=dev), L)
    assert ei.value.status == pk.DM_ESTATE
    with pytest.raises(pk.DMError):
        eng.build_rings([])
    with pytest.raises(pk.DMError):
        eng.build_rings([1, 1])
    with pytest.raises(pk.DMError):
        eng.build_rings([9])
    eng.build_rings([0, 1, 2, 3])
    o = oracle.Oracle(cfg)
    o.build_rings([0, 1, 2, 3])
    # n = 0 is a no-op
    out = eng.route(torch.zeros(1, dtype=torch.int32, device=dev),
                    torch.zeros(1, dtype=torch.int64, device=dev), L)
    eng.sync()
    # empty and sub-block prompts
    off = np.array([0, 0, 5, 5, 21, 37], np.int64)
    tok = np.arange(37, dtype=np.int32)
    g = eng.route(gh.to_dev(tok, dev), gh.to_dev(off, dev), L)
    eng.sync()
    r = o.route(tok, off, np.zeros(4, np.int64))
    compare_route(g, r, 5)
    # malformed offsets are reported by dm_sync (the batch is not read past
    # them): decreasing, negative, past the token array, and overlapping
    # prompts that are each in range
    for bad, ntok in (([0, 8, 4], 8), ([-16, 0, 8], 8), ([0, 8, 24], 16), ([0, 64, 0, 64], 64)):
        _say("malformed offsets", bad, "tokens", ntok)
        eng.route(torch.zeros(64, dtype=torch.int32, device=dev)[:ntok],
                  torch.tensor(bad, dtype=torch.int64, device=dev), L, block_keys=True)
        with pytest.raises(pk.DMError) as ei:
            eng.sync()
        assert ei.value.status == pk.DM_EINVAL
        eng.sync()  # cleared
    # the same token array with valid offsets routes normally afterwards
    L = torch.zeros(4, dtype=torch.int64, device=dev)
    g = eng.route(gh.to_dev(tok, dev), gh.to_dev(off, dev), L)
    eng.sync()
    compare_route(g, r, 5)
    assert np.array_equal(cpu(L), r["loads"])
    # misaligned pointer rejected on the host
    lib = pk.load_library()
    import ctypes as C
    buf = torch.zeros(64, dtype=torch.int64, device=dev)
    ro = pk.dm_route_out(buf.data_ptr() + 4, buf.data_ptr(), buf.data_ptr(), buf.data_ptr(),
                         buf.data_ptr(), buf.data_ptr(), None)
    st = lib.dm_route_batch(eng._h, buf.data_ptr(), 128, buf.data_ptr(), 2, L.data_ptr(),
                            C.byref(ro))
    assert st == pk.DM_EINVAL
    st = lib.dm_route_batch(eng._h, None, 128, buf.data_ptr(), 2, L.data_ptr(), C.byref(ro))
    assert st == pk.DM_EINVAL
    # a batch past the 32-bit selection slots is rejected before any work
    ok = pk.dm_route_out(buf.data_ptr(), buf.data_ptr(), buf.data_ptr(), buf.data_ptr(),
                         buf.data_ptr(), buf.data_ptr(), None)
    st = lib.dm_route_batch(eng._h, buf.data_ptr(), 128, buf.data_ptr(), 1_908_874_241,
                            L.data_ptr(), C.byref(ok))
    assert st == pk.DM_EINVAL
    eng.sync()


def test_batch_sizes_around_chunks_and_blocks_parity():
    """Batch sizes at and around the selection's 64-request chunks and
    1024-request blocks (partial chunks, partial blocks, one request past a
    block), each a prefix of the same prompt stream, routed from the same
    index and loads on both sides."""
    gh = _h()
    wl = workloads.small_random(41, 12, 4, 16, 3000, slo_us=20_000)
    eng, o = gh.engine_for(wl), oh.oracle_for(wl)
    gh.prefill_from_prior(eng, wl)
    oh.prefill_from_prior(o, wl)
    tok, off = workloads.prompts(wl, wl.n_req, sub=0)
    L0 = workloads.initial_loads(wl, wl.route.max_slots)
    tok_d = gh.to_dev(tok, eng.device)
    for k in (1, 2, 63, 64, 65, 127, 1023, 1024, 1025, 2047, 2049, 3000):
        _say("batch size", k)
        Ld = gh.to_dev(L0, eng.device)
        g = eng.route(tok_d, gh.to_dev(off[:k + 1], eng.device), Ld)
        eng.sync()
        r = o.route(tok[:off[k]], off[:k + 1], L0)
        compare_route(g, r, k)
        assert np.array_equal(cpu(Ld), r["loads"]), k


def test_batch_beyond_one_request_per_wave_parity():
    """More requests than the hashing passes' grid has waves (4 Mi): waves
    then take several requests each (the members pass loads the next
    request's record and first chunk ahead).  A 3,000-prompt stream, cut to
    at most 40 tokens, repeated past 4 Mi requests, so groups are large and
    members share their leader's prefix."""
    gh = _h()
    wl = workloads.small_random(43, 8, 4, 16, 3000)
    eng, o = gh.engine_for(wl), oh.oracle_for(wl)
    gh.prefill_from_prior(eng, wl)
    oh.prefill_from_prior(o, wl)
    tok, off = workloads.prompts(wl, wl.n_req, sub=0)
    lens = np.minimum(np.diff(off), 40)
    base = np.concatenate([tok[off[i]:off[i] + lens[i]] for i in range(len(lens))])
    n = (1 << 22) + 1234
    reps = -(-n // len(lens))
    L_all = np.tile(lens, reps)[:n]
    off_big = np.zeros(n + 1, np.int64)
    off_big[1:] = np.cumsum(L_all)
    tok_big = np.tile(base, reps)[:off_big[-1]]
    L0 = workloads.initial_loads(wl, wl.route.max_slots)
    _say("route", n, "requests", len(tok_big), "tokens")
    Ld = gh.to_dev(L0, eng.device)
    g = eng.route(gh.to_dev(tok_big, eng.device), gh.to_dev(off_big, eng.device), Ld,
                  block_keys=True)
    eng.sync()
    r = o.route(tok_big, off_big, L0, block_keys=True)
    compare_route(g, r, n, with_bk=True)
    assert np.array_equal(cpu(Ld), r["loads"])


def test_index_ops_and_capacity():
    gh = _h()
    import paper_2602_06502_amd as pk
    cfg = dict(block=16, key_blocks=4, seeds=(1, 2), vnodes=4, max_slots=3, index_log2_slots=8)
    eng = gh.DualMap(cfg, device="cuda:0")
    dev = eng.device
    rng = np.random.default_rng(1)
    keys = rng.integers(0, 2**64, size=100, dtype=np.uint64)
    keys[:3] = [0, 1, 1 << 63]
    dup = np.concatenate([keys, keys[:50]])
    eng.index_insert(0, gh.to_dev(dup, dev))
    eng.sync()
    assert eng.index_size(0) == len({oracle.canon(int(k)) for k in keys})
    eng.index_erase(0, gh.to_dev(keys[10:20], dev))
    eng.sync()
    left = {oracle.canon(int(k)) for k in keys} - {oracle.canon(int(k)) for k in keys[10:20]}
    assert eng.index_size(0) == len(left)
    eng.index_clear(0)
    eng.sync()
    assert eng.index_size(0) == 0
    # capacity: 2^8 slots hold at most 128 keys
    many = rng.integers(2, 2**64, size=200, dtype=np.uint64)
    eng.index_insert(1, gh.to_dev(many[:128], dev))
    eng.sync()
    assert eng.index_size(1) == 128
    eng.index_insert(1, gh.to_dev(many[128:], dev))
    with pytest.raises(pk.DMError) as ei:
        eng.sync()
    assert ei.value.status == pk.DM_EFULL
    assert eng.index_size(1) == 128


def test_index_capacity_within_one_batch():
    """One insert batch that crosses the load limit stores exactly up to the
    limit and reports DM_EFULL; a batch that fits (many duplicates, up to
    exactly the limit) is stored whole with no error, however its threads
    race for the last slots; a rebuild after erasures never holds more than
    the limit.  2^8 slots hold at most 128 keys."""
    gh = _h()
    import paper_2602_06502_amd as pk
    cfg = dict(block=16, key_blocks=4, seeds=(1, 2), vnodes=4, max_slots=4, index_log2_slots=8)
    eng = gh.DualMap(cfg, device="cuda:0")
    d = lambda a: gh.to_dev(a, eng.device)
    rng = np.random.default_rng(5)

    def full_error():
        with pytest.raises(pk.DMError) as ei:
            eng.sync()
        assert ei.value.status == pk.DM_EFULL

    # 200 distinct keys in one batch
    many = rng.integers(2, 2**64, size=200, dtype=np.uint64)
    _say("index: one batch of 200 distinct keys")
    eng.index_insert(0, d(many))
    full_error()
    assert eng.index_size(0) == 128
    # exactly 128 distinct keys, each four times, shuffled: fits, no error
    k128 = rng.integers(2, 2**64, size=128, dtype=np.uint64)
    _say("index: 128 distinct keys x 4 in one batch")
    eng.index_insert(1, d(rng.permutation(np.tile(k128, 4))))
    eng.sync()
    assert eng.index_size(1) == 128
    # 127 distinct keys x 3, then one new key x 60 with the old ones again
    k127 = rng.integers(2, 2**64, size=128, dtype=np.uint64)
    eng.index_insert(2, d(rng.permutation(np.tile(k127[:127], 3))))
    eng.sync()
    assert eng.index_size(2) == 127
    eng.index_insert(2, d(rng.permutation(np.concatenate([np.repeat(k127[127:], 60), k127[:127]]))))
    eng.sync()
    assert eng.index_size(2) == 128
    eng.index_insert(2, d(rng.integers(2, 2**64, size=3, dtype=np.uint64)))
    full_error()
    assert eng.index_size(2) == 128
    # erase 28 of the full table, then 40 fresh keys: the rebuild keeps 100
    # live keys and stores 28 more
    eng.index_erase(0, d(many[:200]))  # erases exactly the stored ones
    eng.sync()
    assert eng.index_size(0) == 0
    eng.index_insert(0, d(many[:128]))
    eng.sync()
    assert eng.index_size(0) == 128
    eng.index_erase(0, d(many[:28]))
    eng.sync()
    assert eng.index_size(0) == 100
    fresh = rng.integers(2, 2**64, size=40, dtype=np.uint64)
    _say("index: rebuild after erasures, then past the limit")
    eng.index_insert(0, d(fresh))
    full_error()
    assert eng.index_size(0) == 128


def test_index_churn_rebuilds_erased_slots():
    """Erased slots never take new keys, so churn would fill a table with
    them; an insert that would pass the load limit while erased slots exist
    rebuilds the table first.  2^8 slots hold at most 128 keys."""
    gh = _h()
    cfg = dict(block=16, key_blocks=4, seeds=(1, 2), vnodes=4, max_slots=2, index_log2_slots=8)
    eng = gh.DualMap(cfg, device="cuda:0")
    d = lambda a: gh.to_dev(a, eng.device)
    rng = np.random.default_rng(11)
    keys = rng.integers(2, 2**64, size=180, dtype=np.uint64)
    assert len(set(keys.tolist())) == 180
    eng.index_insert(0, d(keys[:100]))
    eng.index_erase(0, d(keys[:60]))
    eng.index_insert(0, d(keys[100:]))  # 100 occupied + 80 > 128: rebuilt, 40 + 80 live
    eng.sync()
    assert eng.index_size(0) == 120
    eng.index_erase(0, d(keys[:60]))  # absent keys: nothing changes
    eng.sync()
    assert eng.index_size(0) == 120
    eng.index_erase(0, d(keys[60:]))  # all 120 present
    eng.sync()
    assert eng.index_size(0) == 0
    # many rounds of churn, each inserting 100 fresh keys and erasing them
    for r in range(20):
        k = rng.integers(2, 2**64, size=100, dtype=np.uint64)
        eng.index_insert(1, d(k))
        eng.sync()
        assert eng.index_size(1) == 100, r
        eng.index_erase(1, d(k))
        eng.sync()
        assert eng.index_size(1) == 0, r


def test_index_erase_then_match_parity():
    """Erased blocks break a cached prefix at the erased block."""
    gh = _h()
    wl = workloads.tiny()
    eng = gh.engine_for(wl)
    o = oh.oracle_for(wl)
    gh.prefill_from_prior(eng, wl)
    oh.prefill_from_prior(o, wl)
    ttok, toff = workloads.templates(wl)
    some = o.chain(0, ttok[toff[0]:toff[1]])[3:6]
    for c in range(8):
        eng.index_erase(c, gh.to_dev(some, eng.device))
        o.index_erase(c, some)
    tok, off = workloads.prompts(wl, wl.n_req)
    L0 = workloads.initial_loads(wl, 8)
    Ld = gh.to_dev(L0, eng.device)
    g = eng.route(gh.to_dev(tok, eng.device), gh.to_dev(off, eng.device), Ld)
    eng.sync()
    r = o.route(tok, off, L0)
    compare_route(g, r, wl.n_req)
    for c in range(8):
        assert eng.index_size(c) == o.index_size(c)


# ---------------------------------------------------------------------------
# Rebalance
# ---------------------------------------------------------------------------

def compare_rebalance(eng, o, q, cap=None, interval=None, thresh=3_000_000):
    gh = _h()
    dev = eng.device
    g = eng.rebalance(gh.to_dev(q.qoff, dev), gh.to_dev(q.rec_id, dev), gh.to_dev(q.unc_here, dev),
                      gh.to_dev(q.alt, dev), gh.to_dev(q.unc_alt, dev), gh.to_dev(q.base_work, dev),
                      cap=cap, prefill_interval=None if interval is None else gh.to_dev(interval, dev),
                      decode_threshold_us=thresh)
    status = 0
    try:
        eng.sync()
    except Exception as e:  # DM_EFULL when cap is exceeded
        status = e.status
    r = o.rebalance(q.qoff, q.rec_id, q.unc_here, q.alt, q.unc_alt, q.base_work, cap=cap,
                    prefill_interval=interval, decode_threshold_us=thresh)
    assert status == r["status"]
    n = int(cpu(g["count"])[0])
    assert n == r["count"]
    m = min(n, len(r["rec"]))
    for k in ("rec", "src", "dst", "benefit", "ttft_to"):
        assert np.array_equal(cpu(g[k])[:m], r[k][:m]), k
    assert np.array_equal(cpu(g["loads"]), r["loads"])
    return r


@pytest.mark.parametrize("seed", range(6))
def test_rebalance_synthetic_parity(seed):
    gh = _h()
    S, n_live = 16, 12
    cfg = dict(block=16, key_blocks=4, seeds=(1, 2), vnodes=4, max_slots=S, index_log2_slots=8,
               slo_us=60_000 + 20_000 * seed)
    eng = gh.DualMap(cfg, device="cuda:0")
    o = oracle.Oracle(cfg)
    rng = np.random.default_rng(seed)
    src = np.sort(rng.choice(n_live, size=1 + seed % 4, replace=False))
    # sources start 10 ms under the SLO so the tail of each queue is over it
    q = workloads.synthetic_queues(seed, S, n_live, src, 300 + 500 * seed, 400, 150_000,
                                   4 * (cfg["slo_us"] - 10_000))
    _say("rebalance synthetic", seed, "records", len(q.rec_id))
    r = compare_rebalance(eng, o, q)
    assert r["count"] > 0


def test_rebalance_cap_and_empty():
    gh = _h()
    S = 8
    cfg = dict(block=16, key_blocks=4, seeds=(1, 2), vnodes=4, max_slots=S, index_log2_slots=8,
               slo_us=50_000)
    eng = gh.DualMap(cfg, device="cuda:0")
    o = oracle.Oracle(cfg)
    q = workloads.synthetic_queues(3, S, S, np.array([1, 5]), 400, 300, 100_000, 4 * 40_000)
    r = compare_rebalance(eng, o, q)
    assert r["count"] > 2
    compare_rebalance(eng, o, q, cap=2)
    # no records at all
    empty = workloads.Queues(np.zeros(S + 1, np.int64), np.zeros(0, np.uint64),
                             np.zeros(0, np.uint32), np.zeros(0, np.uint32), np.zeros(0, np.uint32),
                             np.arange(S, dtype=np.int64))
    r = compare_rebalance(eng, o, empty)
    assert r["count"] == 0


def test_rebalance_long_queues_many_targets_parity():
    """One source whose queue is longer than a commit workgroup holds in
    registers (40,000 records), one that fits unevenly (20,000), and 1,500
    live instances, so each source has more (source, target) segments than
    the workgroup has threads.  Sources start 100 ms under the SLO with small
    uncached counts, so the queues meet the SLO after part of the accepted
    records leave and the stop rule truncates."""
    gh = _h()
    S, n_live = 2048, 1500
    cfg = dict(block=16, key_blocks=4, seeds=(1, 2), vnodes=4, max_slots=S, index_log2_slots=8,
               slo_us=400_000)
    eng = gh.DualMap(cfg, device="cuda:0")
    o = oracle.Oracle(cfg)
    src = np.array([17, 901])
    q = workloads.synthetic_queues(29, S, n_live, src, 40_000, 60, 50_000, 4 * 300_000)
    # second source: keep its first 20,000 records only
    lens = np.diff(q.qoff)
    keep = np.ones(len(q.rec_id), bool)
    keep[q.qoff[901] + 20_000:q.qoff[902]] = False
    lens[901] = 20_000
    qoff = np.zeros(S + 1, np.int64)
    qoff[1:] = np.cumsum(lens)
    q = workloads.Queues(qoff, q.rec_id[keep], q.unc_here[keep], q.alt[keep], q.unc_alt[keep],
                         q.base_work)
    _say("rebalance long queues: records", len(q.rec_id))
    r = compare_rebalance(eng, o, q)
    per_src = np.bincount(r["src"], minlength=S)
    assert 0 < per_src[17] < 40_000 and 0 < per_src[901] < 20_000, per_src[[17, 901]]
    assert len(np.unique(r["dst"])) > 512


def test_rebalance_many_sources_parity():
    """80 overloaded sources of 200 live instances: more sources than the
    pass spreads one source at a time over the GPU (64), so one workgroup
    commits them all; with 40 sources, the spread form.  Both against the
    oracle."""
    gh = _h()
    S, n_live = 256, 200
    cfg = dict(block=16, key_blocks=4, seeds=(1, 2), vnodes=4, max_slots=S, index_log2_slots=8,
               slo_us=200_000)
    eng = gh.DualMap(cfg, device="cuda:0")
    o = oracle.Oracle(cfg)
    rng = np.random.default_rng(90)
    for n_src in (80, 40):
        src = np.sort(rng.choice(n_live, size=n_src, replace=False))
        q = workloads.synthetic_queues(91 + n_src, S, n_live, src, 600, 300, 100_000,
                                       4 * (cfg["slo_us"] - 5_000))
        _say("rebalance sources", n_src, "records", len(q.rec_id))
        r = compare_rebalance(eng, o, q)
        assert len(np.unique(r["src"])) > n_src // 2


def test_rebalance_candidates_past_lds_parity():
    """One source with 300,000 queued records, nearly all eligible: more
    candidates than the commit kernel keeps acceptance bits for in LDS
    (262,144), so the bits and their prefix counts live in device memory,
    and a queue longer than the register form holds (chunked probes).  The
    queue starts just over the SLO, so the stop rule ends the pass after
    about 1,300 migrations."""
    gh = _h()
    S, n_live = 64, 60
    cfg = dict(block=16, key_blocks=4, seeds=(1, 2), vnodes=4, max_slots=S, index_log2_slots=8,
               slo_us=400_000)
    eng = gh.DualMap(cfg, device="cuda:0")
    o = oracle.Oracle(cfg)
    q = workloads.synthetic_queues(41, S, n_live, np.array([17]), 300_000, 4, 50_000, 1_232_000)
    # the case: eligible candidates (benefit > 0, every target below the SLO)
    u = q.unc_here.astype(np.int64)
    before = np.concatenate([[0], np.cumsum(u)[:-1]])
    t_here = 2_000 + 3 * u + ((q.base_work[17] + before) >> 2)
    t_alt = 2_000 + 3 * q.unc_alt.astype(np.int64) + (q.base_work[q.alt] >> 2)
    assert int((t_here > t_alt).sum()) > 262_144
    _say("rebalance past LDS: records", len(q.rec_id))
    r = compare_rebalance(eng, o, q)
    assert 1_000 < r["count"] < 2_000


@pytest.mark.parametrize("seed", range(4))
def test_rebalance_decode_correction_parity(seed):
    """Decode-bottleneck correction (Sec. A.7): stalled sources, stalled
    targets and instances stalled only by the correction, against the
    oracle; intervals at or under the threshold give the plain pass."""
    gh = _h()
    S, n_live = 16, 12
    cfg = dict(block=16, key_blocks=4, seeds=(1, 2), vnodes=4, max_slots=S, index_log2_slots=8,
               slo_us=80_000)
    eng = gh.DualMap(cfg, device="cuda:0")
    o = oracle.Oracle(cfg)
    rng = np.random.default_rng(50 + seed)
    src = np.sort(rng.choice(n_live, size=2, replace=False))
    q = workloads.synthetic_queues(60 + seed, S, n_live, src, 800, 400, 150_000, 4 * 70_000)
    thresh = 20_000
    interval = rng.integers(0, 60_000, size=S).astype(np.int64)
    _say("rebalance decode correction", seed, "records", len(q.rec_id))
    plain = compare_rebalance(eng, o, q)
    r = compare_rebalance(eng, o, q, interval=interval, thresh=thresh)
    assert r["count"] > 0
    assert (r["rec"].tolist() != plain["rec"].tolist()
            or r["ttft_to"].tolist() != plain["ttft_to"].tolist())
    calm = np.minimum(interval, thresh)
    r2 = compare_rebalance(eng, o, q, interval=calm, thresh=thresh)
    for k in ("rec", "src", "dst", "benefit", "ttft_to", "loads"):
        assert np.array_equal(r2[k], plain[k]), k


def test_rebalance_decode_correction_long_queues_parity():
    """The correction on the commit's long-queue paths: a 40,000-record
    source (chunked queue probes) stalled by a small delay, a 2,000-record
    source (queue in registers), and stalled targets among 1,500 live
    instances."""
    gh = _h()
    S, n_live = 2048, 1500
    cfg = dict(block=16, key_blocks=4, seeds=(1, 2), vnodes=4, max_slots=S, index_log2_slots=8,
               slo_us=400_000)
    eng = gh.DualMap(cfg, device="cuda:0")
    o = oracle.Oracle(cfg)
    q = workloads.synthetic_queues(31, S, n_live, np.array([17, 901]), 40_000, 60, 50_000,
                                   4 * 300_000)
    lens = np.diff(q.qoff)
    keep = np.ones(len(q.rec_id), bool)
    keep[q.qoff[901] + 2_000:q.qoff[902]] = False
    lens[901] = 2_000
    qoff = np.zeros(S + 1, np.int64)
    qoff[1:] = np.cumsum(lens)
    q = workloads.Queues(qoff, q.rec_id[keep], q.unc_here[keep], q.alt[keep], q.unc_alt[keep],
                         q.base_work)
    rng = np.random.default_rng(7)
    interval = np.zeros(S, np.int64)
    interval[17] = 25_000
    interval[901] = 120_000
    stalled_targets = rng.choice(n_live, size=200, replace=False)
    interval[stalled_targets] = rng.integers(30_000, 500_000, size=200)
    _say("rebalance decode correction long queues: records", len(q.rec_id))
    r = compare_rebalance(eng, o, q, interval=interval, thresh=20_000)
    per_src = np.bincount(r["src"], minlength=S)
    assert per_src[17] > 0 and per_src[901] > 0, per_src[[17, 901]]


def test_rebalance_decode_telemetry_errors():
    gh = _h()
    import paper_2602_06502_amd as pk
    S = 8
    cfg = dict(block=16, key_blocks=4, seeds=(1, 2), vnodes=4, max_slots=S, index_log2_slots=8,
               slo_us=50_000)
    eng = gh.DualMap(cfg, device="cuda:0")
    o = oracle.Oracle(cfg)
    q = workloads.synthetic_queues(3, S, S, np.array([1, 5]), 400, 300, 100_000, 4 * 40_000)
    dev = eng.device
    args = [gh.to_dev(a, dev) for a in (q.qoff, q.rec_id, q.unc_here, q.alt, q.unc_alt, q.base_work)]
    good = np.full(S, 1_000, np.int64)
    with pytest.raises(pk.DMError) as ei:
        eng.rebalance(*args, prefill_interval=gh.to_dev(good, dev), decode_threshold_us=-1)
    assert ei.value.status == pk.DM_EINVAL
    bad = good.copy()
    bad[3] = -1
    eng.rebalance(*args, prefill_interval=gh.to_dev(bad, dev), decode_threshold_us=10)
    with pytest.raises(pk.DMError) as ei:
        eng.sync()
    assert ei.value.status == pk.DM_EINVAL
    assert o.rebalance(q.qoff, q.rec_id, q.unc_here, q.alt, q.unc_alt, q.base_work,
                       prefill_interval=bad, decode_threshold_us=10)["status"] == oracle.EINVAL
    # the context stays usable
    compare_rebalance(eng, o, q, interval=good, thresh=10)


def _queues_from_route(chosen, cand, match, off, B, S, base_work):
    """Queues built from a routed batch: each request queued on its chosen
    instance in arrival order; alternative = the other candidate."""
    n = len(chosen)
    c1, c2 = cand[:n], cand[n:]
    lens = np.diff(off)
    unc1, unc2 = lens - B * match[:n].astype(np.int64), lens - B * match[n:].astype(np.int64)
    here_is1 = chosen == c1
    alt = np.where(here_is1, c2, c1).astype(np.uint32)
    uh = np.where(here_is1, unc1, unc2).astype(np.uint32)
    ua = np.where(here_is1, unc2, unc1).astype(np.uint32)
    order = np.argsort(chosen, kind="stable")
    qoff = np.zeros(S + 1, np.int64)
    qoff[1:] = np.cumsum(np.bincount(chosen, minlength=S))
    return workloads.Queues(qoff, order.astype(np.uint64) + 1000, uh[order], alt[order], ua[order],
                            base_work.astype(np.int64))


def test_tiny_rebalance_parity():
    """Tiny-rebalance: queues formed by a Tiny-tight batch (each side from
    its own routing), then one migration pass."""
    wl = workloads.tiny(slo_us=20_000)
    eng, o, g, r, tok, off = run_pair(wl, block_keys=False)

    def base_work(chosen):
        # the two instances holding the most queued tokens start 8 ms under the SLO
        work = np.bincount(chosen, weights=np.diff(off), minlength=8)
        bw = np.zeros(8, np.int64)
        bw[np.argsort(-work, kind="stable")[:2]] = 4 * (20_000 - 8_000)
        return bw

    gch = cpu(g["chosen"])
    qg = _queues_from_route(gch, cpu(g["cand"]), cpu(g["match"]), off, 16, 8, base_work(gch))
    qo = _queues_from_route(r["chosen"], r["cand"], r["match"], off, 16, 8, base_work(r["chosen"]))
    gh = _h()
    dev = eng.device
    gg = eng.rebalance(gh.to_dev(qg.qoff, dev), gh.to_dev(qg.rec_id, dev),
                       gh.to_dev(qg.unc_here, dev), gh.to_dev(qg.alt, dev),
                       gh.to_dev(qg.unc_alt, dev), gh.to_dev(qg.base_work, dev))
    eng.sync()
    rr = o.rebalance(qo.qoff, qo.rec_id, qo.unc_here, qo.alt, qo.unc_alt, qo.base_work)
    n = int(cpu(gg["count"])[0])
    assert n == rr["count"] and n > 0
    for k in ("rec", "src", "dst", "benefit", "ttft_to"):
        assert np.array_equal(cpu(gg[k])[:n], rr[k]), k
    assert np.array_equal(cpu(gg["loads"]), rr["loads"])


# ---------------------------------------------------------------------------
# Scaling
# ---------------------------------------------------------------------------

def test_scale_parity_then_reroute():
    wl = workloads.tiny()
    eng, o, g, r, tok, off = run_pair(wl, block_keys=False)
    gh = _h()
    keys = r["key"]
    add, rm = [9, 10], [2, 6]
    cfg = dict(wl.route.as_dict(), max_slots=12)
    # fresh engines with room for the added ids
    eng = gh.DualMap(cfg, device="cuda:0")
    o = oracle.Oracle(cfg)
    eng.build_rings(range(8))
    o.build_rings(range(8))
    gs = eng.scale(add, rm, gh.to_dev(keys, eng.device))
    eng.sync()
    rs = o.scale(add, rm, keys)
    assert rs["status"] == 0 and rs["violations"] == 0
    for k in ("old", "new", "moved"):
        assert np.array_equal(cpu(gs[k]), rs[k]), k
    assert int(cpu(gs["violations"])[0]) == 0
    for s in (0, 1):
        gp, gi = eng.ring(s)
        op, oi = o.ring(s)
        assert np.array_equal(gp, op) and np.array_equal(gi, oi)
    # bad scale requests change nothing
    import paper_2602_06502_amd as pk
    for a_, r_ in (([1], []), ([], [2]), ([20], []), ([11, 11], [])):
        with pytest.raises(pk.DMError):
            eng.scale(a_, r_, gh.to_dev(keys, eng.device))
    L0 = workloads.initial_loads(wl, 12)
    Ld = gh.to_dev(L0, eng.device)
    g2 = eng.route(gh.to_dev(tok, eng.device), gh.to_dev(off, eng.device), Ld)
    eng.sync()
    r2 = o.route(tok, off, L0)
    compare_route(g2, r2, wl.n_req)
    assert not set(np.unique(r2["cand"]).tolist()) & set(rm)


def test_determinism_repeat():
    wl = workloads.small_random(21, 6, 8, 16, 500, slo_us=5_000)
    gh = _h()
    eng = gh.engine_for(wl)
    gh.prefill_from_prior(eng, wl)
    tok, off = workloads.prompts(wl, wl.n_req)
    L0 = workloads.initial_loads(wl, wl.route.max_slots)
    outs = []
    for _ in range(2):
        Ld = gh.to_dev(L0, eng.device)
        outs.append({k: cpu(v) for k, v in eng.route(gh.to_dev(tok, eng.device),
                                                     gh.to_dev(off, eng.device), Ld).items()})
    for k in outs[0]:
        assert np.array_equal(outs[0][k], outs[1][k])


# ---------------------------------------------------------------------------
# Pipelined batches
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("slo_us", [400_000, 20_000])
def test_pipelined_batches_parity(slo_us):
    """Three consecutive batches routed with pipelining (each batch's
    selection overlapping the next batch's hashing and probing), one loads
    array carried through; the oracle routes the same batches one after the
    other.  Then an index change after the batches must be ordered after
    their selections."""
    wl = workloads.tiny(slo_us=slo_us)
    gh = _h()
    eng = gh.engine_for(wl)
    o = oh.oracle_for(wl)
    gh.prefill_from_prior(eng, wl)
    oh.prefill_from_prior(o, wl)
    tok, off = workloads.prompts(wl, wl.n_req)
    cuts = [0, 300, 301, 1024]  # ragged batches, one of a single request
    L0 = workloads.initial_loads(wl, wl.route.max_slots)
    dev = eng.device
    Ld = gh.to_dev(L0, dev)
    eng.set_pipelining(True)
    eng.set_timing(True)
    outs, refs = [], []
    Lo = L0
    for lo, hi in zip(cuts[:-1], cuts[1:]):
        t = tok[off[lo]:off[hi]]
        f = off[lo:hi + 1] - off[lo]
        outs.append(eng.route(gh.to_dev(t, dev), gh.to_dev(f, dev), Ld, block_keys=True))
        r = o.route(t, f, Lo, block_keys=True)
        refs.append(r)
        Lo = r["loads"]
    eng.sync()
    ms = eng.stage_ms()
    assert all(x >= 0 for x in ms)
    for g, r, (lo, hi) in zip(outs, refs, zip(cuts[:-1], cuts[1:])):
        compare_route(g, r, hi - lo, with_bk=True)
    assert np.array_equal(cpu(Ld), Lo)
    # a later call is ordered after the last selection
    eng.index_clear(0)
    assert eng.index_size(0) == 0
    eng.set_pipelining(False)
    t = tok[off[0]:off[300]]
    f = off[0:301] - off[0]
    g = eng.route(gh.to_dev(t, dev), gh.to_dev(f, dev), Ld)
    eng.sync()
    o.index_clear(0)
    r = o.route(t, f, Lo)
    compare_route(g, r, 300)
    assert np.array_equal(cpu(Ld), r["loads"])


def test_pipelined_shrinking_batches_parity():
    """Pipelined batches of 16,384, then 8,192, then 16,384 requests: each
    batch's selection work arrays must stay clear of those of the batch
    before it, which may still be walking when a smaller batch packs its
    records.  Every output and the final loads against the oracle."""
    import dataclasses
    wl = workloads.small_random(77, 24, 16, 16, 40_960, slo_us=60_000)
    wl = dataclasses.replace(wl, n_prior=2_000,
                             route=dataclasses.replace(wl.route, index_log2_slots=14))
    gh = _h()
    eng, o = gh.engine_for(wl), oh.oracle_for(wl)
    gh.prefill_from_prior(eng, wl)
    oh.prefill_from_prior(o, wl)
    tok, off = workloads.prompts(wl, wl.n_req)
    L0 = workloads.initial_loads(wl, wl.route.max_slots)
    dev = eng.device
    Ld = gh.to_dev(L0, dev)
    cuts = [0, 16_384, 24_576, 40_960]
    eng.set_pipelining(True)
    outs, refs, Lo = [], [], L0
    try:
        for lo, hi in zip(cuts[:-1], cuts[1:]):
            _say("pipelined batch", hi - lo)
            t = tok[off[lo]:off[hi]]
            f = off[lo:hi + 1] - off[lo]
            outs.append(eng.route(gh.to_dev(t, dev), gh.to_dev(f, dev), Ld))
            r = o.route(t, f, Lo)
            refs.append(r)
            Lo = r["loads"]
        eng.sync()
    finally:
        eng.set_pipelining(False)
    for g, r, (lo, hi) in zip(outs, refs, zip(cuts[:-1], cuts[1:])):
        compare_route(g, r, hi - lo)
    assert np.array_equal(cpu(Ld), Lo)


def test_group_resolution_paths_parity():
    """Requests that share a cached prefix P (300 blocks, cached on every
    instance) and so one ring-key group, built to reach every way a group
    member is resolved: the leader's match (its first disagreement with
    the leader comes after the leader's first miss), its own length
    (a prefix of the leader), probes of its kept keys past the first
    disagreement, and the resume walk (more than the kept keys present).
    Every output against the oracle, with and without block keys."""
    gh = _h()
    B = 16
    cfg = dict(block=B, key_blocks=4, seeds=(3, 9), vnodes=16, max_slots=8, index_log2_slots=14)
    rng = np.random.default_rng(23)
    P = rng.integers(0, 50_000, size=300 * B, dtype=np.int32)
    rnd = lambda nb: rng.integers(0, 50_000, size=nb * B, dtype=np.int32)
    prompts = [np.concatenate([P[:30 * B], rnd(20)]) for _ in range(64)]  # leader: the first
    prompts += [
        P[:300 * B],                                    # pending past the kept keys: resume
        np.concatenate([P[:33 * B], rnd(5)]),           # pending: first miss among kept keys
        P[:25 * B],                                     # own length (prefix of the leader)
        np.concatenate([P[:30 * B], rnd(3)]),           # pending at the leader's first miss
        np.concatenate([P[:20 * B], rnd(40)]),          # disagrees before the leader's miss
        prompts[0].copy(),                              # the leader's own prompt: its match
        np.concatenate([P[:300 * B], rnd(1)[:7]]),      # partial tail block
        np.concatenate([P[:37 * B], rnd(2)]),           # first miss on the last kept key
        np.concatenate([P[:38 * B], rnd(2)]),           # first miss just past the kept keys
    ]
    prompts += [rnd(int(k)) for k in rng.integers(0, 40, size=40)]  # groups of their own
    off = np.zeros(len(prompts) + 1, np.int64)
    off[1:] = np.cumsum([len(p) for p in prompts])
    tok = np.concatenate(prompts).astype(np.int32)
    o = oracle.Oracle(cfg)
    o.build_rings(range(8))
    eng = gh.DualMap(cfg, device="cuda:0")
    eng.build_rings(list(range(8)))
    pk = o.chain(0, P)
    assert len(pk) == 300
    for inst in range(8):
        o.index_insert(inst, pk)
        eng.index_insert(inst, gh.to_dev(pk, eng.device))
    eng.sync()
    L0 = np.arange(8, dtype=np.int64) * 1000
    for bk in (False, True):
        _say("group resolution paths, block keys", bk)
        Ld = gh.to_dev(L0, eng.device)
        g = eng.route(gh.to_dev(tok, eng.device), gh.to_dev(off, eng.device), Ld, block_keys=bk)
        eng.sync()
        r = o.route(tok, off, L0, block_keys=bk)
        compare_route(g, r, len(prompts), with_bk=bk)
        assert np.array_equal(cpu(Ld), r["loads"])
    n = len(prompts)
    m1 = r["match"][:n]
    assert m1[64] == 300 and m1[65] == 33 and m1[66] == 25 and m1[67] == 30
    assert m1[68] == 20 and m1[69] == 30 and m1[71] == 37 and m1[72] == 38
