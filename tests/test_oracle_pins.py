"""Pins of the CPU oracle against facts fixed outside the oracle itself:
inverses derived from the mathematics, closed forms, brute force on tiny
inputs, the paper's worked examples and its stated guarantees.

Citations name the paper's sections (DualMap, arXiv 2602.06502).
"""
import math
import os
import random

import numpy as np
import pytest

import oracle
import workloads

M64 = (1 << 64) - 1
GOLDEN_DIR = os.path.join(os.path.dirname(__file__), "golden")


def setup_module(_):
    oracle.build(force=False)


# ---------------------------------------------------------------------------
# mix64 / SplitMix64 (reading of the unnamed hash functions, Sec. 3.2)
# ---------------------------------------------------------------------------

def _unxorshift(y, s):
    x = y
    for _ in range(64 // s + 1):
        x = y ^ (x >> s)
    return x & M64


def mix64_inverse(z):
    """Inverse of the SplitMix64 finaliser, derived step by step: invert the
    final xorshift-31, multiply by the modular inverse of the second
    constant, invert xorshift-27, multiply by the inverse of the first
    constant, invert xorshift-30."""
    z = _unxorshift(z, 31)
    z = (z * pow(0x94D049BB133111EB, -1, 1 << 64)) & M64
    z = _unxorshift(z, 27)
    z = (z * pow(0xBF58476D1CE4E5B9, -1, 1 << 64)) & M64
    return _unxorshift(z, 30)


def test_mix64_roundtrips_through_independent_inverse():
    rng = random.Random(7)
    xs = [0, 1, 2, M64, 1 << 63] + [rng.getrandbits(64) for _ in range(2000)]
    for x in xs:
        assert mix64_inverse(oracle.mix64(x)) == x


def test_mix64_avalanche():
    # flipping any single input bit flips about half the output bits
    rng = random.Random(11)
    flips = np.zeros(64)
    n = 300
    for _ in range(n):
        x = rng.getrandbits(64)
        hx = oracle.mix64(x)
        for b in range(64):
            flips[b] += bin(hx ^ oracle.mix64(x ^ (1 << b))).count("1")
    mean = flips / n
    assert np.all(np.abs(mean - 32) < 3.0), mean


def test_golden_increment_is_two_pow_64_over_phi():
    # floor(2^64 / phi) = floor(2^63 (sqrt5 - 1)) from an integer square root
    golden = math.isqrt(5 << 126) - (1 << 63)
    assert golden == 0x9E3779B97F4A7C15


@pytest.mark.parametrize("seed,B", [(1, 16), (2, 16), (1, 32), (5, 2)])
def test_hash_parameters_follow_the_splitmix_stream(seed, B):
    """Key words, multiplier and chain start are consecutive outputs of a
    SplitMix64 stream at `seed`: their pre-images under mix64 step by the
    golden increment."""
    golden = math.isqrt(5 << 126) - (1 << 63)
    kk, mult, h_init = oracle.params(seed, B)
    assert mult & 1 == 1
    pre_h = mix64_inverse(h_init)
    assert pre_h == (seed + (B + 2) * golden) & M64
    pre_m = {mix64_inverse(mult), mix64_inverse(mult ^ 1)}
    assert (seed + (B + 1) * golden) & M64 in pre_m
    for j in range(B):
        assert int(kk[j]) == oracle.mix64((seed + (j + 1) * golden) & M64) & 0xFFFFFFFF


# ---------------------------------------------------------------------------
# NH block digest and the chain (Sec. A.3.2: one hash per KV block)
# ---------------------------------------------------------------------------

def test_nh_with_zero_keys_is_pairwise_dot_product():
    rng = np.random.default_rng(3)
    for B in (2, 4, 16, 32):
        t = rng.integers(-2**31, 2**31, size=B, dtype=np.int64).astype(np.int32)
        want = sum((int(t[2 * j]) & 0xFFFFFFFF) * (int(t[2 * j + 1]) & 0xFFFFFFFF)
                   for j in range(B // 2)) & M64
        assert oracle.nh(t, np.zeros(B, np.uint32)) == want


def test_nh_keys_enter_as_token_translation_mod_2_32():
    rng = np.random.default_rng(4)
    B = 16
    for _ in range(50):
        t = rng.integers(0, 2**31, size=B).astype(np.int32)
        k = rng.integers(0, 2**32, size=B, dtype=np.uint64).astype(np.uint32)
        shifted = ((t.astype(np.uint64) + k.astype(np.uint64)) & 0xFFFFFFFF).astype(np.uint32).view(np.int32)
        assert oracle.nh(t, k) == oracle.nh(shifted, np.zeros(B, np.uint32))


def _cfg(B=16, K=4, seeds=(1, 2), V=8, S=8):
    return dict(block=B, key_blocks=K, seeds=seeds, vnodes=V, max_slots=S)


@pytest.mark.parametrize("B,seed_idx", [(16, 0), (16, 1), (32, 0), (4, 1)])
def test_chain_matches_closed_form(B, seed_idx):
    """H[b] = H[-1] P^(b+1) + sum_k NH(k) P^(b-k) (mod 2^64), recovered from
    each block key through the independent inverse of mix64."""
    o = oracle.Oracle(_cfg(B=B, seeds=(1, 2)))
    seed = (1, 2)[seed_idx]
    kk, P, H0 = oracle.params(seed, B)
    rng = np.random.default_rng(B)
    t = rng.integers(0, 32000, size=B * 9 + B // 2).astype(np.int32)
    keys = o.chain(seed_idx, t)
    assert len(keys) == 9  # partial trailing tokens are not hashed
    nhs = [oracle.nh(t[b * B:(b + 1) * B], kk) for b in range(9)]
    for b in range(9):
        H = (H0 * pow(P, b + 1, 1 << 64) + sum(nhs[k] * pow(P, b - k, 1 << 64) for k in range(b + 1))) & M64
        assert mix64_inverse(int(keys[b])) ^ seed == H


def test_block_keys_equal_iff_token_prefixes_equal():
    """Tiny collision check: across prompts sharing prefixes of various
    lengths, block key b agrees exactly when blocks 0..b agree token for
    token."""
    B = 4
    o = oracle.Oracle(_cfg(B=B))
    rng = np.random.default_rng(9)
    base = rng.integers(0, 5, size=40).astype(np.int32)
    prompts = []
    for cut in range(0, 40, 3):
        p = base.copy()
        p[cut:] = rng.integers(0, 5, size=40 - cut)
        prompts.append(p)
    chains = [o.chain(0, p) for p in prompts]
    for a in range(len(prompts)):
        for c in range(len(prompts)):
            for b in range(10):
                same = np.array_equal(prompts[a][:(b + 1) * B], prompts[c][:(b + 1) * B])
                assert (chains[a][b] == chains[c][b]) == same


def test_ring_key_is_key_of_last_hashed_block():
    B, K = 16, 4
    o = oracle.Oracle(_cfg(B=B, K=K))
    rng = np.random.default_rng(5)
    for length in (0, 1, 15, 16, 17, 47, 48, 64, 65, 200):
        t = rng.integers(0, 1000, size=length).astype(np.int32)
        for s in (0, 1):
            x = o.ring_key(s, t)
            ch = o.chain(s, t)
            kr = min(K, length // B)
            if kr:
                assert x == int(ch[kr - 1])
            else:  # empty-prefix key: mix64(H[-1] xor seed)
                _, _, H0 = oracle.params((1, 2)[s], B)
                assert mix64_inverse(x) ^ (1, 2)[s] == H0


# ---------------------------------------------------------------------------
# Rings (Sec. 3.4; Sec. A.1.3)
# ---------------------------------------------------------------------------

def test_vnode_positions_are_the_bijective_mix_of_id_and_vnode():
    o = oracle.Oracle(_cfg(S=40, V=16))
    seen = set()
    for s in (0, 1):
        seed = (1, 2)[s]
        for i in range(40):
            for v in range(16):
                p = o.vpos(s, i, v)
                assert mix64_inverse(p) == ((i << 32) | v) ^ oracle.mix64(seed)
                seen.add((s, p))
    assert len(seen) == 2 * 40 * 16


def _brute_owner(entries, x):
    """Linear scan: smallest position >= x, else the smallest overall."""
    ge = [(p, i) for p, i in entries if p >= x]
    return min(ge)[1] if ge else min(entries)[1]


def test_ring_build_and_owner_against_linear_scan():
    ids = [0, 3, 4, 7, 9]
    o = oracle.Oracle(_cfg(S=12, V=6))
    assert o.build_rings(ids) == oracle.OK
    rng = random.Random(1)
    for s in (0, 1):
        pos, own = o.ring(s)
        entries = sorted((o.vpos(s, i, v), i) for i in ids for v in range(6))
        assert [p for p, _ in entries] == [int(p) for p in pos]
        assert [i for _, i in entries] == [int(i) for i in own]
        probes = [0, M64, int(pos[0]), int(pos[-1]), int(pos[-1]) + 1, int(pos[3]) - 1]
        probes += [rng.getrandbits(64) for _ in range(500)]
        for x in probes:
            x &= M64
            assert o.owner(s, x) == _brute_owner(entries, x)


def _read_ring_example():
    rows = []
    with open(os.path.join(GOLDEN_DIR, "ring_example.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                rows.append(line.split())
    return rows


def test_ring_worked_example_A_to_E():
    """Sec. A.1.3: (A,B]->B, (B,C]->C, (C,D]->D; adding E between B and C
    moves only (B,E] to E."""
    place = dict(A=1000, B=2000, E=2500, C=3000, D=4000)
    ident = dict(A=0, B=1, C=2, D=3, E=4)
    rows = _read_ring_example()
    for phase, names in (("before", "ABCD"), ("after", "ABECD")):
        pos = np.array([place[n] for n in names], np.uint64)
        ids = np.array([ident[n] for n in names], np.uint32)
        for ph, lo, hi, own in rows:
            if ph != phase:
                continue
            for x in (place[lo] + 1, (place[lo] + place[hi]) // 2, place[hi]):
                assert oracle.owner_sorted(pos, ids, x) == ident[own]
    # only keys in (B, E] change owner
    before = (np.array([1000, 2000, 3000, 4000], np.uint64), np.array([0, 1, 2, 3], np.uint32))
    after = (np.array([1000, 2000, 2500, 3000, 4000], np.uint64), np.array([0, 1, 4, 2, 3], np.uint32))
    for x in range(0, 5000, 7):
        moved = oracle.owner_sorted(*before, x) != oracle.owner_sorted(*after, x)
        assert moved == (2000 < x <= 2500)


def test_second_candidate_adjustment_dense_ids():
    """Sec. 3.2: if both hashes pick one instance, id2 = (id1 + 1) mod n."""
    n = 6
    o = oracle.Oracle(_cfg(S=n, V=4))
    o.build_rings(range(n))
    rng = random.Random(3)
    hits = 0
    for _ in range(4000):
        x1, x2 = rng.getrandbits(64), rng.getrandbits(64)
        c1, c2, fix = o.candidates(x1, x2)
        if o.owner(0, x1) == o.owner(1, x2):
            hits += 1
            assert fix and c2 == (c1 + 1) % n
        else:
            assert not fix and c2 == o.owner(1, x2)
        assert c1 != c2
    assert hits > 100


def test_second_candidate_adjustment_sparse_ids_and_single_instance():
    o = oracle.Oracle(_cfg(S=10, V=4))
    o.build_rings([0, 3, 5])
    nxt = {0: 3, 3: 5, 5: 0}
    rng = random.Random(4)
    for _ in range(3000):
        x1, x2 = rng.getrandbits(64), rng.getrandbits(64)
        c1, c2, fix = o.candidates(x1, x2)
        if fix:
            assert c2 == nxt[c1]
        assert c1 != c2
    o1 = oracle.Oracle(_cfg(S=4, V=4))
    o1.build_rings([2])
    c1, c2, fix = o1.candidates(5, 6)
    assert (c1, c2, fix) == (2, 2, True)


# ---------------------------------------------------------------------------
# Match, TTFT, selection (Sec. 3.2; Sec. A.1.1; Sec. A.3.2)
# ---------------------------------------------------------------------------

def _lcp(a, b):
    n = min(len(a), len(b))
    k = 0
    while k < n and a[k] == b[k]:
        k += 1
    return k


def test_match_equals_floor_lcp_over_block():
    B = 8
    o = oracle.Oracle(_cfg(B=B, K=2, S=3, V=4))
    o.build_rings([0, 1, 2])
    rng = np.random.default_rng(12)
    A = rng.integers(0, 4, size=120).astype(np.int32)
    for inst in range(3):
        o.index_insert(inst, o.chain(0, A))
    prompts = []
    for cut in list(range(0, 120, 5)) + [120]:
        for extra in (0, 3, 17):
            p = np.concatenate([A[:cut], rng.integers(4, 8, size=extra).astype(np.int32)])
            prompts.append(p)
    off = np.zeros(len(prompts) + 1, np.int64)
    off[1:] = np.cumsum([len(p) for p in prompts])
    out = o.route(np.concatenate(prompts), off, np.zeros(3, np.int64))
    n = len(prompts)
    for r, p in enumerate(prompts):
        want = min(_lcp(A, p), len(p)) // B
        assert out["match"][r] == want and out["match"][n + r] == want


def test_ttft_hand_values():
    o = oracle.Oracle(_cfg())
    assert o.ttft(0, 0) == 2000
    assert o.ttft(100, 10) == 2000 + 300 + 2
    assert o.ttft(7, 3) == 2000 + 21 + 0
    assert o.ttft(0, -1) == 2000 - 1  # floor division
    assert o.ttft(0, 4_000_000) == 1_002_000


@pytest.mark.parametrize("case", [
    # (m1, m2, L1, L2, len, expected chosen (1|2), flags without fixup bit)
    (3, 3, 10, 20, 100, 1, 4),      # equal hits -> less loaded
    (3, 3, 20, 20, 100, 1, 4),      # equal hits, equal load -> c1
    (3, 3, 21, 20, 100, 2, 4),
    (5, 1, 10**6, 0, 100, 1, 0),    # affinity kept while TTFT <= SLO
    (5, 1, 2_000_000, 0, 100, 2, 1),    # affinity TTFT over SLO -> less loaded
    (5, 1, 2_000_000, 2_000_000, 100, 1, 2),  # over, other not less loaded: keep; both over
    (1, 5, 0, 2_000_000, 100, 1, 1),    # symmetric: c2 affine, over -> c1
    (1, 5, 2_000_001, 2_000_000, 100, 2, 2),  # both over, c1 not less loaded: c2 kept
])
def test_selection_truth_table(case):
    m1, m2, L1, L2, length, want, want_flags = case
    o = oracle.Oracle(dict(_cfg(B=16), slo_us=400_000))
    loads = np.array([L1, L2], np.int64)
    ch, t, f = o.select(0, 1, m1, m2, length, loads)
    assert ch == want - 1
    assert f == want_flags
    unc = length - 16 * (m1 if ch == 0 else m2)
    assert t == 2000 + 3 * unc + loads[ch] // 4
    # the SLO threshold is inclusive: TTFT == SLO keeps affinity
    L_eq = 4 * (400_000 - 2000 - 3 * (length - 16 * 5))
    ch, t, f = o.select(0, 1, 5, 1, length, np.array([L_eq, 0], np.int64))
    assert t == 400_000 and ch == 0


@pytest.mark.parametrize("case", [
    # (policy, m1, m2, L1, L2, len, expected chosen (1|2), flags)
    # TTFT = 2000 + 3 unc + L/4 with B = 16, SLO 400,000
    ("cache_affinity", 5, 1, 2_000_000, 0, 100, 1, 0),   # affine even far over the SLO
    ("cache_affinity", 1, 5, 0, 2_000_000, 100, 2, 0),
    ("cache_affinity", 3, 3, 21, 20, 100, 2, 4),          # equal hits: less loaded
    ("cache_affinity", 3, 3, 20, 20, 100, 1, 4),
    ("least_loaded", 5, 1, 11, 10, 100, 2, 1),            # less loaded, fewer cached blocks
    ("least_loaded", 5, 1, 10, 10, 100, 1, 0),            # ties: c1
    ("least_loaded", 1, 5, 10, 10, 100, 1, 1),            # ties: c1 even with fewer blocks
    ("least_loaded", 3, 3, 21, 20, 100, 2, 4),
    # min TTFT: t1 = 2000 + 3 (100 - 16 m1) + L1/4, t2 likewise
    ("min_ttft", 5, 1, 400, 0, 100, 1, 0),   # t1 = 2060 + 100 = 2160 < t2 = 2252
    ("min_ttft", 5, 1, 772, 0, 100, 2, 1),   # t1 = 2060 + 193 = 2253 > 2252
    ("min_ttft", 5, 1, 768, 0, 100, 1, 0),   # t1 = 2060 + 192 = 2252 = t2: ties c1
    ("min_ttft", 3, 3, 8, 4, 100, 2, 4),     # equal hits: t by load, 2000+156+2 vs +1
    ("min_ttft", 3, 3, 7, 4, 100, 1, 4),     # 7/4 = 1 = 4/4: tie, c1
    ("slo_aware", 5, 1, 2_000_000, 0, 100, 2, 1),
])
def test_policy_truth_table(case):
    """The ablation variants of Sec. 4.3 by hand.  bit0 marks a chosen
    candidate with fewer cached blocks, bit1 both over the SLO, bit2 equal
    hits."""
    policy, m1, m2, L1, L2, length, want, want_flags = case
    o = oracle.Oracle(dict(_cfg(B=16), slo_us=400_000))
    assert o.set_policy(policy) == oracle.OK
    loads = np.array([L1, L2], np.int64)
    ch, t, f = o.select(0, 1, m1, m2, length, loads)
    assert ch == want - 1, (ch, want)
    assert f == want_flags
    unc = length - 16 * (m1 if ch == 0 else m2)
    assert t == 2000 + 3 * unc + loads[ch] // 4


def test_policy_rejects_unknown():
    o = oracle.Oracle(_cfg())
    assert o.set_policy(4) == oracle.EINVAL and o.set_policy(-1) == oracle.EINVAL
    assert o.set_policy("slo_aware") == oracle.OK


def _in_order(policy, cand, match, lens, L0, B, slo):
    """Literal in-order replay of one rule over a routed batch (Sec. 3.2 and
    the single-criterion rules of Sec. 4.3) from its candidates and hits."""
    n = len(lens)
    L = L0.astype(np.int64).copy()
    out = []
    for r in range(n):
        c = (int(cand[r]), int(cand[n + r]))
        m = (int(match[r]), int(match[n + r]))
        u = [int(lens[r]) - B * m[0], int(lens[r]) - B * m[1]]
        t = [2000 + 3 * u[k] + int(L[c[k]]) // 4 for k in (0, 1)]
        if policy == "least_loaded" or m[0] == m[1]:
            k = 0 if L[c[0]] <= L[c[1]] else 1
            if policy == "min_ttft":
                k = 0 if t[0] <= t[1] else 1
        elif policy == "min_ttft":
            k = 0 if t[0] <= t[1] else 1
        elif policy == "cache_affinity":
            k = 0 if m[0] > m[1] else 1
        else:
            a = 0 if m[0] > m[1] else 1
            k = a if t[a] <= slo or not L[c[1 - a]] < L[c[a]] else 1 - a
        out.append(c[k])
        L[c[k]] += u[k]
    return np.array(out), L


@pytest.mark.parametrize("policy", ["slo_aware", "cache_affinity", "least_loaded", "min_ttft"])
def test_policy_routes_match_in_order_replay(policy):
    """Whole batches under each rule equal the literal request-by-request
    replay, and the per-rule invariants hold: cache affinity takes the
    larger hit of every request (so its hit rate bounds every rule's from
    above, the index being a snapshot), least loaded the candidate with the
    smaller pre-update load."""
    import oracle.harness as oh
    wl = workloads.tiny(slo_us=20_000)
    st = oh.setup(wl)
    o = st["oracle"]
    assert o.set_policy(policy) == oracle.OK
    tok, off, L0 = st["tokens"], st["offsets"], st["loads0"]
    out = o.route(tok, off, L0.copy())
    lens = np.diff(off)
    want, Lw = _in_order(policy, out["cand"], out["match"], lens, L0, wl.route.block, 20_000)
    assert np.array_equal(out["chosen"], want)
    assert np.array_equal(out["loads"], Lw)
    n = len(lens)
    m_ch = np.where(out["chosen"] == out["cand"][:n], out["match"][:n], out["match"][n:])
    best = np.maximum(out["match"][:n], out["match"][n:])
    if policy == "cache_affinity":
        assert np.array_equal(m_ch, best)
    assert np.all(m_ch <= best)
    o.set_policy("slo_aware")


def _read_narrative():
    rows = []
    with open(os.path.join(GOLDEN_DIR, "slo_narrative.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                r, inst, why = line.split()
                rows.append((int(r), int(inst), why))
    return rows


def test_slo_narrative_scenario():
    """Fig. 'SLO-aware request routing': instance 1 (id 0 here) caches all
    prefixes, instance 2 (id 1) none; requests 1-4 stay, 5 switches, 6-7
    (equal hits) go to the less-loaded instance."""
    B, slo = 16, 10_000
    o = oracle.Oracle(dict(block=B, key_blocks=4, seeds=(1, 2), vnodes=8, max_slots=2, slo_us=slo))
    o.build_rings([0, 1])
    rng = np.random.default_rng(21)
    tpl = rng.integers(0, 1000, size=160).astype(np.int32)       # 10 blocks, cached on id 0
    shared = rng.integers(0, 1000, size=160).astype(np.int32)    # cached on both
    o.index_insert(0, o.chain(0, tpl))
    o.index_insert(0, o.chain(0, shared))
    o.index_insert(1, o.chain(0, shared))
    reqs = []
    for r in range(7):
        base = tpl if r < 5 else shared
        reqs.append(np.concatenate([base, rng.integers(2000, 3000, size=32).astype(np.int32)]))
    off = np.zeros(8, np.int64)
    off[1:] = np.cumsum([len(p) for p in reqs])
    # id 0 starts just below the SLO knee: TTFT = 2000 + 3*32 + L/4 <= 10000
    L0 = np.array([31_616 - 3 * 32, 0], np.int64)
    out = o.route(np.concatenate(reqs), off, L0)
    for (r, inst, why) in _read_narrative():
        assert out["chosen"][r - 1] == inst - 1, (r, why)
        if why == "slo_switch":
            assert out["flags"][r - 1] & 1
        if why.startswith("equal"):
            assert out["flags"][r - 1] & 4


def test_cache_affinity_guarantee():
    """Sec. 2.3: m requests sharing a prefix get hit rate >= max(0, 1 - 2/m)
    (routing one at a time, each routed chain then cached on its instance)."""
    B = 16
    for seed in range(5):
        o = oracle.Oracle(dict(block=B, key_blocks=4, seeds=(1, 2), vnodes=16, max_slots=8, slo_us=20_000))
        o.build_rings(range(8))
        rng = np.random.default_rng(100 + seed)
        prefix = rng.integers(0, 5000, size=8 * B).astype(np.int32)
        loads = rng.integers(0, 80_000, size=8).astype(np.int64)
        m = 25
        hits = 0
        for _ in range(m):
            p = np.concatenate([prefix, rng.integers(5000, 9000, size=40).astype(np.int32)])
            out = o.route(p, np.array([0, len(p)], np.int64), loads, block_keys=True)
            ch = int(out["chosen"][0])
            got = out["match"][0] if ch == out["cand"][0] else out["match"][1]
            hits += int(got >= 8)
            o.index_insert(ch, out["block_keys"])
            loads = out["loads"]
        assert hits / m >= max(0.0, 1 - 2 / m)


def test_two_choices_spread_less_than_one_choice():
    """Sec. 2.3 (power of two choices): with equal cache hits everywhere the
    rule joins the less-loaded candidate; the max-minus-mean load gap is far
    below placing every request on its first candidate."""
    gaps1, gaps2 = [], []
    for seed in range(10):
        wl = workloads.small_random(seed, 16, 64, 16, 4000)
        o = oracle.Oracle(dict(wl.route.as_dict(), max_slots=16))
        o.build_rings(range(16))
        rng = np.random.default_rng(seed)
        tok = rng.integers(0, 1 << 30, size=4000 * 64).astype(np.int32)
        off = np.arange(0, 4000 * 64 + 1, 64, dtype=np.int64)
        out = o.route(tok, off, np.zeros(16, np.int64))
        two = np.bincount(out["chosen"], minlength=16)
        one = np.bincount(out["cand"][:4000], minlength=16)
        gaps2.append(two.max() - two.mean())
        gaps1.append(one.max() - one.mean())
    assert np.mean(gaps2) * 4 < np.mean(gaps1)
    # max load stays within m/n + log log n / log 2 + O(1) (Eq. potc_2_choices)
    assert np.max(gaps2) <= math.log(math.log(16)) / math.log(2) + 4


# ---------------------------------------------------------------------------
# Rebalance (Sec. 3.3; Sec. A.1.2)
# ---------------------------------------------------------------------------

def brute_rebalance(cfg, qoff, rec, here, alt, other, W0, interval=None, thresh=0):
    """Literal pass recomputing every queue TTFT from scratch at each step.
    With `interval`, an instance with queued requests whose prefill interval
    exceeds `thresh` is stalled in decode and every TTFT estimated on it gets
    the interval added (Sec. A.7)."""
    base, per, div, slo = cfg["ttft_base_us"], cfg["ttft_per_token_us"], cfg["queue_div"], cfg["slo_us"]
    S = len(W0)
    queues = {i: list(range(qoff[i], qoff[i + 1])) for i in range(S)}
    stalled = [interval is not None and bool(queues[i]) and interval[i] > thresh for i in range(S)]

    def T(unc, load, inst):
        return (int(interval[inst]) if stalled[inst] else 0) + base + per * unc + load // div

    def qts(i, q):
        ahead, out = W0[i], []
        for r in q:
            out.append(T(int(here[r]), ahead, i))
            ahead += int(here[r])
        return out

    L = [W0[i] + sum(int(here[r]) for r in queues[i]) for i in range(S)]
    over = [bool(queues[i]) and max(qts(i, queues[i])) > slo for i in range(S)]
    L0 = list(L)
    migs = []
    for i in sorted([i for i in range(S) if over[i]], key=lambda i: (-L0[i], i)):
        ts = qts(i, queues[i])
        cands = []
        for p, r in enumerate(queues[i]):
            j = int(alt[r])
            b = ts[p] - T(int(other[r]), L0[j], j)
            if b > 0 and not over[j]:
                cands.append((-b, p, r))
        cands.sort()
        cur = list(queues[i])
        for negb, p, r in cands:
            now = qts(i, cur)
            if not now or max(now) <= slo:
                break
            j = int(alt[r])
            tj = T(int(other[r]), L[j], j)
            if tj < slo:
                cur.remove(r)
                L[i] -= int(here[r])
                L[j] += int(other[r])
                migs.append((int(rec[r]), i, j, -negb, tj))
    return migs, L


def _random_queues(seed, S=5, maxq=12):
    rng = np.random.default_rng(seed)
    lens = rng.integers(0, maxq + 1, size=S)
    qoff = np.zeros(S + 1, np.int64)
    qoff[1:] = np.cumsum(lens)
    Q = int(qoff[-1])
    owner = np.repeat(np.arange(S), lens)
    alt = (owner + rng.integers(1, S, size=Q)) % S
    here = rng.integers(0, 30, size=Q).astype(np.uint32)
    other = rng.integers(0, 30, size=Q).astype(np.uint32)
    rec = np.arange(Q, dtype=np.uint64) + 100
    W0 = rng.integers(0, 120, size=S).astype(np.int64)
    return qoff, rec, here, alt.astype(np.uint32), other, W0


@pytest.mark.parametrize("seed", range(60))
def test_rebalance_matches_brute_force(seed):
    cfg = dict(block=16, key_blocks=4, seeds=(1, 2), vnodes=4, max_slots=5,
               ttft_base_us=2, ttft_per_token_us=1, queue_div=4, slo_us=40 + seed % 20)
    o = oracle.Oracle(cfg)
    qoff, rec, here, alt, other, W0 = _random_queues(seed)
    got = o.rebalance(qoff, rec, here, alt, other, W0)
    want, L = brute_rebalance(cfg, qoff, rec, here, alt, other, W0)
    assert got["status"] == oracle.OK
    assert got["count"] == len(want)
    g = list(zip(got["rec"].tolist(), got["src"].tolist(), got["dst"].tolist(),
                 got["benefit"].tolist(), got["ttft_to"].tolist()))
    assert g == want
    assert got["loads"].tolist() == L


@pytest.mark.parametrize("seed", range(40))
def test_rebalance_decode_correction_matches_brute_force(seed):
    """Decode-bottleneck correction (Sec. A.7) against the literal pass."""
    cfg = dict(block=16, key_blocks=4, seeds=(1, 2), vnodes=4, max_slots=5,
               ttft_base_us=2, ttft_per_token_us=1, queue_div=4, slo_us=50 + seed % 20)
    o = oracle.Oracle(cfg)
    qoff, rec, here, alt, other, W0 = _random_queues(1000 + seed)
    rng = np.random.default_rng(seed)
    interval = rng.integers(0, 40, size=5).astype(np.int64)
    thresh = int(rng.integers(0, 30))
    got = o.rebalance(qoff, rec, here, alt, other, W0, prefill_interval=interval,
                      decode_threshold_us=thresh)
    want, L = brute_rebalance(cfg, qoff, rec, here, alt, other, W0, interval, thresh)
    assert got["status"] == oracle.OK
    g = list(zip(got["rec"].tolist(), got["src"].tolist(), got["dst"].tolist(),
                 got["benefit"].tolist(), got["ttft_to"].tolist()))
    assert g == want
    assert got["loads"].tolist() == L


def _decode_case(interval1, queue1):
    """Instance 0 holds two records of 10 uncached tokens (alternative 1, 5
    tokens there); instance 1 holds one record of 1 token if queue1."""
    cfg = dict(block=16, key_blocks=4, seeds=(1, 2), vnodes=4, max_slots=3,
               ttft_base_us=2, ttft_per_token_us=1, queue_div=4, slo_us=40)
    o = oracle.Oracle(cfg)
    n1 = 1 if queue1 else 0
    qoff = np.array([0, 2, 2 + n1, 2 + n1], np.int64)
    here = np.array([10, 10] + [1] * n1, np.uint32)
    alt = np.array([1, 1] + [2] * n1, np.uint32)
    other = np.array([5, 5] + [1] * n1, np.uint32)
    rec = np.array([7, 8] + [9] * n1, np.uint64)
    W0 = np.zeros(3, np.int64)
    return o, (qoff, rec, here, alt, other, W0), np.array([30, interval1, 0], np.int64)


def test_rebalance_decode_correction_hand_values():
    """Sec. A.7 by hand.  TTFT = 2 + unc + load/4, SLO 40.  Instance 0's
    queue estimates 12 and 14 us: no overload.  With a prefill interval of
    30 us over a 20 us threshold it is stalled in decode: 42 and 44 us,
    overloaded.  Instance 1 (empty queue, so never stalled) estimates 7 us
    for either record: benefits 35 and 37; the 37 record moves first
    (target TTFT 7), the queue still estimates 42, the other moves (target
    TTFT 2 + 5 + 5/4 = 8)."""
    o, q, interval = _decode_case(100, queue1=False)
    plain = o.rebalance(*q)
    assert plain["count"] == 0
    got = o.rebalance(*q, prefill_interval=interval, decode_threshold_us=20)
    assert got["status"] == oracle.OK and got["count"] == 2
    assert got["rec"].tolist() == [8, 7] and got["src"].tolist() == [0, 0]
    assert got["dst"].tolist() == [1, 1]
    assert got["benefit"].tolist() == [37, 35] and got["ttft_to"].tolist() == [7, 8]
    assert got["loads"].tolist() == [0, 10, 0]
    # at the threshold exactly the instance is not stalled (strictly above)
    at = o.rebalance(*q, prefill_interval=interval, decode_threshold_us=30)
    assert at["count"] == 0
    # instance 1 with queued work and a 100 us interval is stalled too: its
    # record estimates 100 + 2 + 1 = 103 us, so instance 1 is overloaded and
    # no target for instance 0; its own record moves to instance 2 (benefit
    # 103 - 3 = 100, target TTFT 3), instance 0 keeps its queue
    o, q, interval = _decode_case(100, queue1=True)
    got = o.rebalance(*q, prefill_interval=interval, decode_threshold_us=20)
    assert got["status"] == oracle.OK and got["count"] == 1
    assert got["rec"].tolist() == [9] and got["src"].tolist() == [1] and got["dst"].tolist() == [2]
    assert got["benefit"].tolist() == [100] and got["ttft_to"].tolist() == [3]
    assert got["loads"].tolist() == [20, 0, 1]
    # every interval at or under the threshold: the plain pass
    o2 = oracle.Oracle(dict(block=16, key_blocks=4, seeds=(1, 2), vnodes=4, max_slots=5,
                            ttft_base_us=2, ttft_per_token_us=1, queue_div=4, slo_us=45))
    for seed in range(5):
        qq = _random_queues(2000 + seed)
        a = o2.rebalance(*qq)
        b = o2.rebalance(*qq, prefill_interval=np.full(5, 20, np.int64), decode_threshold_us=20)
        for k in ("rec", "src", "dst", "benefit", "ttft_to", "loads"):
            assert a[k].tolist() == b[k].tolist()


def test_rebalance_decode_correction_rejects_bad_telemetry():
    o, q, interval = _decode_case(100, queue1=False)
    assert o.rebalance(*q, prefill_interval=interval, decode_threshold_us=-1)["status"] == oracle.EINVAL
    bad = interval.copy()
    bad[2] = -5
    assert o.rebalance(*q, prefill_interval=bad, decode_threshold_us=20)["status"] == oracle.EINVAL
    bad[2] = (1 << 40) + 1
    assert o.rebalance(*q, prefill_interval=bad, decode_threshold_us=20)["status"] == oracle.EINVAL


def test_rebalance_invariants_and_cap():
    cfg = dict(block=16, key_blocks=4, seeds=(1, 2), vnodes=4, max_slots=5,
               ttft_base_us=2, ttft_per_token_us=1, queue_div=4, slo_us=45)
    o = oracle.Oracle(cfg)
    total_moves = 0
    for seed in range(100, 140):
        qoff, rec, here, alt, other, W0 = _random_queues(seed)
        got = o.rebalance(qoff, rec, here, alt, other, W0)
        total_moves += got["count"]
        recidx = {int(r): k for k, r in enumerate(rec)}
        L_start = np.array([W0[i] + here[qoff[i]:qoff[i + 1]].astype(np.int64).sum() for i in range(5)])
        delta = 0
        for r, i, j, b, tj in zip(got["rec"], got["src"], got["dst"], got["benefit"], got["ttft_to"]):
            k = recidx[int(r)]
            assert b > 0 and tj < cfg["slo_us"] and int(alt[k]) == j and qoff[i] <= k < qoff[i + 1]
            delta += int(other[k]) - int(here[k])
        assert got["loads"].sum() == L_start.sum() + delta
        if got["count"] > 1:
            capped = o.rebalance(qoff, rec, here, alt, other, W0, cap=1)
            assert capped["status"] == oracle.EFULL and capped["count"] == got["count"]
    assert total_moves > 20


# ---------------------------------------------------------------------------
# Scaling (Sec. 3.4; Sec. A.1.3)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(4))
def test_scale_moves_only_affected_keys(seed):
    N, V, S = 16, 64, 24
    o = oracle.Oracle(_cfg(S=S, V=V))
    o.build_rings(range(N))
    rng = np.random.default_rng(seed)
    keys = rng.integers(0, 2**64, size=2 * 20000, dtype=np.uint64)
    rm = np.sort(rng.choice(N, size=2, replace=False)).astype(np.uint32)
    add = np.array([16, 17, 18], np.uint32)
    out = o.scale(add, rm, keys)
    assert out["status"] == oracle.OK
    assert out["violations"] == 0
    n = 20000
    live = sorted(set(range(N)) - set(rm.tolist()) | set(add.tolist()))
    for s in (0, 1):
        entries = sorted((o.vpos(s, i, v), i) for i in live for v in range(V))
        for k in range(0, n, 97):
            assert out["new"][s * n + k] == _brute_owner(entries, int(keys[s * n + k]))
        frac = out["moved"][s] / n
        expect = 2 / N + 3 / (N + 1) - (2 / N) * (3 / (N + 1))
        assert abs(frac - expect) < 0.06, (frac, expect)
    assert o.n_live() == N + 1


def test_scale_rejects_bad_sets_and_keeps_state():
    o = oracle.Oracle(_cfg(S=8, V=4))
    o.build_rings([0, 1, 2])
    keys = np.arange(10, dtype=np.uint64)
    assert o.scale([1], [], keys)["status"] == oracle.EINVAL      # add existing
    assert o.scale([], [5], keys)["status"] == oracle.EINVAL      # remove unknown
    assert o.scale([9], [], keys)["status"] == oracle.EINVAL      # out of range
    assert o.scale([], [0, 1, 2], keys)["status"] == oracle.EINVAL  # empty result
    assert o.n_live() == 3


# ---------------------------------------------------------------------------
# Index set semantics and the sort primitive
# ---------------------------------------------------------------------------

def test_index_set_semantics_and_reserved_keys():
    o = oracle.Oracle(_cfg(S=2))
    keys = np.array([5, 5, 0, 1, 1 << 63, 7], np.uint64)
    o.index_insert(0, keys)
    # 0 and 1 map to 2^63 and 2^63+1; 2^63 itself collides with canon(0)
    assert o.index_size(0) == 4
    for k in (5, 0, 1, 7, 1 << 63):
        assert o.index_contains(0, k)
    assert not o.index_contains(1, 5)
    o.index_erase(0, np.array([5, 99], np.uint64))
    assert not o.index_contains(0, 5) and o.index_size(0) == 3
    o.index_clear(0)
    assert o.index_size(0) == 0


def test_radix_sort_matches_numpy():
    rng = np.random.default_rng(0)
    for n in (0, 1, 2, 100, 100_000):
        a = rng.integers(0, 2**64, size=n, dtype=np.uint64)
        assert np.array_equal(oracle.sort_u64(a), np.sort(a))


def test_metadata_footprint_fixture():
    """Sec. A.3.2: 16 B per block (8 B hash + 8 B id).  The device table
    spends 8 B per slot at load factor <= 1/2, i.e. at least 16 B per cached
    block -- the same footprint."""
    vals = {}
    with open(os.path.join(GOLDEN_DIR, "metadata_footprint.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                k, v = line.split()
                vals[k] = int(v)
    assert vals["bytes_per_block"] == 8 + 8
    assert 8 / 0.5 == vals["bytes_per_block"]


# ---------------------------------------------------------------------------
# Adaptive hash-key length (Sec. 3.2; Sec. A.1.1, Fig. prefix-len)
# ---------------------------------------------------------------------------

def _tree_model(batches, K, B, n_live):
    """The prefix hotness tree over token tuples (no hashing): for each batch,
    every request's key length K_r (walk from depth K while the prefix is
    extended, at most its full blocks) and, after the window closes, the
    extended prefixes.  The close applies the one-level rule (hot leaf:
    extend; extended and cold: shrink) repeatedly until nothing changes,
    with counts taken directly from the token prefixes."""
    ext = set()
    for batch in batches:
        counts = {}
        klens = []
        for p in batch:
            nfull = len(p) // B
            if nfull <= K:
                kr = nfull
            else:
                kr = K
                while kr < nfull and tuple(p[:kr * B]) in ext:
                    kr += 1
            for d in range(K, nfull + 1):
                node = tuple(p[:d * B])
                counts[node] = counts.get(node, 0) + 1
            klens.append(kr)
        W = len(batch)
        if W:
            old = set(ext)
            hot = lambda v: counts.get(v, 0) * n_live > 2 * W
            cold = lambda v: counts.get(v, 0) * n_live < W
            tree = {v for v in old if not cold(v)}
            # a child of an extended node (or a root) that is a hot leaf
            # extends; repeat until no leaf is hot
            while True:
                grow = {v for v in counts if v not in tree and hot(v) and
                        (len(v) == K * B or v[:len(v) - B] in tree)}
                # extended nodes are kept only under a kept parent
                tree = {v for v in tree | grow if len(v) == K * B or v[:len(v) - B] in tree | grow}
                if not grow:
                    break
            ext = tree
        yield klens, set(ext)


def _node_key(o, node):
    return oracle.canon(int(o.chain(0, np.array(node, np.int32))[-1]))


def _route_windows(o, batches, n_live):
    for batch in batches:
        tok = np.concatenate([np.asarray(p, np.int32) for p in batch]) if batch else \
            np.zeros(0, np.int32)
        off = np.zeros(len(batch) + 1, np.int64)
        off[1:] = np.cumsum([len(p) for p in batch])
        out = o.route(tok, off, np.zeros(n_live, np.int64))
        assert o.keylen_window() == oracle.OK
        yield out, tok, off


def _check_tree_against_model(o, batches, K, B, n_live):
    depths = []
    for (out, tok, off), (klens, ext) in zip(_route_windows(o, batches, n_live),
                                             _tree_model(batches, K, B, n_live)):
        assert out["key_len"].tolist() == klens
        n = len(klens)
        for r, kr in enumerate(klens):
            p = tok[off[r]:off[r + 1]]
            assert int(out["key"][r]) == o.ring_key_at(0, p, kr)
            assert int(out["key"][n + r]) == o.ring_key_at(1, p, kr)
        want = sorted(_node_key(o, v) for v in ext)
        assert o.keylen_tree().tolist() == want
        # the tree stays connected: a node below the roots has its parent
        for v in ext:
            if len(v) > K * B:
                assert tuple(v[:len(v) - B]) in ext
        depths.append(klens)
    return depths


def _blk(rng, B):
    return list(rng.integers(0, 1 << 20, size=B))


def test_keylen_hand_windows():
    """K = 1, B = 4, 4 live instances.  Window 1: six of eight requests start
    with block A (counts: A 6; 6*4 = 24 > 2*8): A extends.  Window 2: the A
    requests now hash two blocks, so their ring keys change; A still sees 6
    requests (24 >= 8) and stays.  Window 3: one A request of eight
    (4 < 8): A is cold and shrinks back.  Window 4: A requests hash one
    block again."""
    B, K, n_live = 4, 1, 4
    rng = np.random.default_rng(5)
    A = _blk(rng, B)
    a_reqs = [A + _blk(rng, B) + [7, 7] for _ in range(6)]
    others = [_blk(rng, B) + _blk(rng, B) for _ in range(2)]
    w1 = a_reqs + others
    w3 = [a_reqs[0]] + [_blk(rng, B) + _blk(rng, B) for _ in range(7)]
    w4 = a_reqs[:2] + others
    o = oracle.Oracle(dict(block=B, key_blocks=K, seeds=(1, 2), vnodes=16, max_slots=n_live))
    o.build_rings(range(n_live))
    assert o.keylen_enable(64) == oracle.OK
    outs = list(_route_windows(o, [w1], n_live))
    assert outs[0][0]["key_len"].tolist() == [1] * 8
    assert o.keylen_tree().tolist() == [_node_key(o, A)]
    k1 = outs[0][0]["key"][:6].copy()
    out2 = list(_route_windows(o, [w1], n_live))[0][0]
    assert out2["key_len"].tolist() == [2] * 6 + [1, 1]
    assert len(set(out2["key"][:6].tolist())) == 6 and not set(out2["key"][:6]) & set(k1)
    assert o.keylen_tree().tolist() == [_node_key(o, A)]
    out3 = list(_route_windows(o, [w3], n_live))[0][0]
    assert out3["key_len"][0] == 2
    assert o.keylen_tree().tolist() == []
    out4 = list(_route_windows(o, [w4], n_live))[0][0]
    assert out4["key_len"].tolist() == [1, 1, 1, 1]
    assert out4["key"][:2].tolist() == k1[:2].tolist()
    # and the same windows through the token-tuple model
    o2 = oracle.Oracle(dict(block=B, key_blocks=K, seeds=(1, 2), vnodes=16, max_slots=n_live))
    o2.build_rings(range(n_live))
    o2.keylen_enable(64)
    _check_tree_against_model(o2, [w1, w1, w3, w4], K, B, n_live)


def test_keylen_thresholds_are_strict_and_inclusive():
    """Hot needs rho > 2/n (4 of 8 with n = 4 is exactly 2/n: no); cold needs
    rho < 1/n (2 of 8 is exactly 1/n: stays)."""
    B, K, n_live = 4, 1, 4
    rng = np.random.default_rng(6)
    A = _blk(rng, B)
    mk = lambda k: [A + _blk(rng, B) for _ in range(k)] + [_blk(rng, B) + _blk(rng, B)
                                                           for _ in range(8 - k)]
    o = oracle.Oracle(dict(block=B, key_blocks=K, seeds=(1, 2), vnodes=16, max_slots=n_live))
    o.build_rings(range(n_live))
    o.keylen_enable(8)
    list(_route_windows(o, [mk(4)], n_live))
    assert o.keylen_tree().tolist() == []
    list(_route_windows(o, [mk(5)], n_live))
    assert o.keylen_tree().tolist() == [_node_key(o, A)]
    list(_route_windows(o, [mk(2)], n_live))
    assert o.keylen_tree().tolist() == [_node_key(o, A)]
    list(_route_windows(o, [mk(1)], n_live))
    assert o.keylen_tree().tolist() == []
    # an empty window changes nothing
    list(_route_windows(o, [mk(5)], n_live))
    list(_route_windows(o, [[]], n_live))
    assert o.keylen_tree().tolist() == [_node_key(o, A)]


def test_keylen_extends_to_where_requests_part():
    """A template of three blocks shared by every request: the first close
    extends the path through the whole template (each level is hot in turn:
    16 of 16 requests, 16 * 8 > 2 * 16), and the requests' own fourth
    blocks (one request each) stay leaves.  From the second window on every
    request hashes four blocks: its own fourth block decides its pair.  When
    the template drops to 3 of 16 requests (3 * 8 = 24: not above 2 * 16,
    not below 16) the tree stays; at 1 of 16 (8 < 16) all three levels are
    cold and go."""
    B, K, n_live = 4, 1, 8
    rng = np.random.default_rng(7)
    T = _blk(rng, B) + _blk(rng, B) + _blk(rng, B)
    batch = [T + _blk(rng, B) + _blk(rng, B) for _ in range(16)]
    mix3 = batch[:3] + [_blk(rng, B) * 2 for _ in range(13)]
    mix1 = batch[:1] + [_blk(rng, B) * 2 for _ in range(15)]
    o = oracle.Oracle(dict(block=B, key_blocks=K, seeds=(1, 2), vnodes=16, max_slots=n_live))
    o.build_rings(range(n_live))
    o.keylen_enable(16)
    depths = _check_tree_against_model(o, [batch, batch, mix3, mix1, mix1], K, B, n_live)
    assert [d[0] for d in depths] == [1, 4, 4, 4, 1]
    assert len(o.keylen_tree()) == 0
    assert len(set(o.ring_key_at(0, np.array(p, np.int32), 4) for p in batch)) == 16


def test_keylen_disabled_or_empty_tree_is_fixed_K():
    wl = workloads.tiny(slo_us=20_000)
    import oracle.harness as oh
    st = oh.setup(wl)
    o = st["oracle"]
    a = o.route(st["tokens"], st["offsets"], st["loads0"])
    o.keylen_enable(1024)
    b = o.route(st["tokens"], st["offsets"], st["loads0"])
    for k in ("key", "cand", "match", "chosen", "ttft", "flags", "key_len"):
        assert np.array_equal(a[k], b[k]), k
    nfull = np.diff(st["offsets"]) // wl.route.block
    assert np.array_equal(a["key_len"], np.minimum(nfull, wl.route.key_blocks))
    o.keylen_enable(0)


@pytest.mark.parametrize("seed", range(6))
def test_keylen_random_windows_match_token_model(seed):
    """Zipf-popular templates with random tails over several windows: key
    lengths, ring keys and the tree after every window against the
    token-tuple model (brute-force counts of every path prefix)."""
    rng = np.random.default_rng(100 + seed)
    B, K, n_live = 4, 2, 8
    templates = [[int(x) for x in rng.integers(0, 50, size=B * int(rng.integers(K + 1, 9)))]
                 for _ in range(6)]
    w = 1.0 / np.arange(1, 7) ** 1.4
    w /= w.sum()
    batches = []
    for _ in range(7):
        batch = []
        for _ in range(int(rng.integers(40, 120))):
            t = templates[int(rng.choice(6, p=w))]
            cut = int(rng.integers(0, len(t) + 1)) if rng.random() < 0.2 else \
                int(rng.integers(K * B, len(t) + 1))
            batch.append(t[:cut] + [int(x) for x in rng.integers(0, 50, size=int(rng.integers(0, 5 * B)))])
        batches.append(batch)
    o = oracle.Oracle(dict(block=B, key_blocks=K, seeds=(1, 2), vnodes=16, max_slots=n_live))
    o.build_rings(range(n_live))
    o.keylen_enable(4096)
    depths = _check_tree_against_model(o, batches, K, B, n_live)
    assert max(max(d) for d in depths) > K  # the tree did extend


def test_keylen_capacity_and_state_errors():
    B, K, n_live = 4, 1, 8
    rng = np.random.default_rng(8)
    A, C = _blk(rng, B), _blk(rng, B)
    batch = [A + _blk(rng, B) for _ in range(4)] + [C + _blk(rng, B) for _ in range(4)]
    o = oracle.Oracle(dict(block=B, key_blocks=K, seeds=(1, 2), vnodes=16, max_slots=n_live))
    assert o.keylen_window() == oracle.EINVAL  # tree off
    o.build_rings(range(n_live))
    o.keylen_enable(1)
    tok = np.concatenate([np.asarray(p, np.int32) for p in batch])
    off = np.arange(0, len(tok) + 1, 2 * B, dtype=np.int64)
    o.route(tok, off, np.zeros(n_live, np.int64))
    # A and C both hot (4 * 8 > 2 * 8), room for one: the tree is unchanged
    assert o.keylen_window() == oracle.EFULL
    assert o.keylen_tree().tolist() == []
    o.keylen_enable(2)
    o.route(tok, off, np.zeros(n_live, np.int64))
    assert o.keylen_window() == oracle.OK
    assert o.keylen_tree().tolist() == sorted([_node_key(o, A), _node_key(o, C)])


# ---------------------------------------------------------------------------
# KV save with LRU eviction (the serving step after routing, Sec. A.3.2)
# ---------------------------------------------------------------------------

def _kv_case(o, B, chains, inst, clock, cap):
    toks, off = [], [0]
    keys = []
    for ch in chains:
        toks.append(np.asarray(ch, np.int32))
        off.append(off[-1] + len(ch))
        keys.append(o.chain(0, np.asarray(ch, np.int32)))
    bk = np.concatenate(keys) if keys else np.zeros(0, np.uint64)
    return o.kv_save(np.array(off, np.int64), bk, np.array(inst, np.uint32), clock, cap), bk


def test_kv_save_hand_values():
    """cap 3 on instance 0.  Request A = blocks (a0, a1, a2) touches a2, a1,
    a0 at times 0, 1, 2 (deepest first); request B = (a0, b1) touches b1 at
    3 and a0 at 4.  Four distinct keys: the least recent, a2, is dropped in
    the same call, so a0, a1, b1 join the index and nothing leaves; the
    cache stays prefix-closed."""
    import sys
    sys.path.insert(0, os.path.dirname(__file__))
    B = 4
    o = oracle.Oracle(dict(block=B, key_blocks=1, seeds=(1, 2), vnodes=4, max_slots=2))
    rng = np.random.default_rng(11)
    a = [int(x) for x in rng.integers(0, 1000, size=3 * B)]
    b = a[:B] + [int(x) for x in rng.integers(1000, 2000, size=B)]
    (rc, added, removed), bk = _kv_case(o, B, [a, b], [0, 0], 0, 3)
    assert rc == oracle.OK and (added, removed) == (3, 0)
    ka, kb = o.chain(0, np.array(a, np.int32)), o.chain(0, np.array(b, np.int32))
    assert o.index_size(0) == 3 and o.index_size(1) == 0
    for k, present in ((ka[0], True), (ka[1], True), (ka[2], False), (kb[1], True)):
        assert bool(o.index_contains(0, int(k))) == present
    # a later batch touching only a2 (its own chain a0, a1, a2 again) at
    # clock 5: times a2 5, a1 6, a0 7; b1 (time 3) is now the least recent
    (rc, added, removed), _ = _kv_case(o, B, [a], [0], 5, 3)
    assert (added, removed) == (1, 1)
    assert not o.index_contains(0, int(kb[1])) and o.index_contains(0, int(ka[2]))


@pytest.mark.parametrize("seed", range(5))
def test_kv_save_matches_lru_model(seed):
    """Batches of template-sharing prompts over 4 instances against the LRU
    model of the multi-batch driver (tests/sim.py, written independently):
    after every batch each instance's index holds exactly the model's keys,
    and the added and removed counts agree."""
    import sys
    sys.path.insert(0, os.path.dirname(__file__))
    import sim
    B, S = 4, 4
    o = oracle.Oracle(dict(block=B, key_blocks=1, seeds=(1, 2), vnodes=4, max_slots=S))
    lru = sim.LRUIndex(S, cap=40 + 10 * seed)
    rng = np.random.default_rng(200 + seed)
    tpl = [list(rng.integers(0, 100, size=B * int(rng.integers(2, 9)))) for _ in range(5)]
    clock = 0
    for _ in range(6):
        chains, inst = [], []
        for _ in range(int(rng.integers(5, 40))):
            t = tpl[int(rng.integers(0, 5))]
            cut = int(rng.integers(0, len(t) + 1))
            chains.append([int(x) for x in t[:cut]] +
                          [int(x) for x in rng.integers(0, 100, size=int(rng.integers(0, 3 * B)))])
            inst.append(int(rng.integers(0, S)))
        (rc, added, removed), bk = _kv_case(o, B, chains, inst, clock, lru.cap)
        assert rc == oracle.OK
        nfull = np.array([len(c) // B for c in chains])
        upd = lru.touch(np.array(inst), bk, nfull)
        clock += int(nfull.sum())
        assert added == sum(len(a) for a, _ in upd.values())
        assert removed == sum(len(r) for _, r in upd.values())
        for c in range(S):
            assert o.index_size(c) == len(lru.keys[c])
            assert all(o.index_contains(c, int(k)) for k in lru.keys[c])


def test_kv_save_lower_cap_applies_to_every_instance():
    """Instance 1 holds 3 saved keys; a save with cap 2 that sends it nothing
    still leaves it its 2 most recent (the least recent is erased), and
    instance 0, sent one chain of 2 blocks, keeps both."""
    B = 4
    o = oracle.Oracle(dict(block=B, key_blocks=1, seeds=(1, 2), vnodes=4, max_slots=2))
    rng = np.random.default_rng(13)
    c1 = [int(x) for x in rng.integers(0, 50, size=B * 3)]
    (rc, added, removed), bk1 = _kv_case(o, B, [c1], [1], 0, 0)
    assert rc == oracle.OK and (added, removed) == (3, 0)
    c0 = [int(x) for x in rng.integers(50, 100, size=B * 2)]
    (rc, added, removed), bk0 = _kv_case(o, B, [c0], [0], 3, 2)
    assert rc == oracle.OK and (added, removed) == (2, 1)
    assert o.index_size(0) == 2 and o.index_size(1) == 2
    # times of instance 1's blocks: block 2 at 0, block 1 at 1, block 0 at 2
    assert not o.index_contains(1, int(bk1[2])) and o.index_contains(1, int(bk1[0]))


def test_kv_save_unbounded_and_errors():
    B = 4
    o = oracle.Oracle(dict(block=B, key_blocks=1, seeds=(1, 2), vnodes=4, max_slots=2))
    rng = np.random.default_rng(12)
    chains = [[int(x) for x in rng.integers(0, 50, size=B * 3)] for _ in range(4)]
    (rc, added, removed), bk = _kv_case(o, B, chains, [1, 1, 1, 1], 0, 0)
    assert rc == oracle.OK and removed == 0 and added == len(np.unique(bk))
    assert o.index_size(1) == len(np.unique(bk))
    (rc, _, _), _ = _kv_case(o, B, chains[:1], [2], 0, 0)
    assert rc == oracle.EINVAL


# ---------------------------------------------------------------------------
# Queued requests: append, migrate, drain (the state the rebalancing pass
# reads, Sec. 3.3)
# ---------------------------------------------------------------------------

def _qs_csr(qs):
    qoff, rec, here, alt, there, base = qs.csr()
    return [qoff, rec, here, alt, there, base]


@pytest.mark.parametrize("seed", range(6))
def test_queue_operations_match_queue_model(seed):
    """Append routed batches, apply migration lists, drain: the oracle's CSR
    operations against the multi-batch driver's queue model (tests/sim.py,
    written independently), after every step."""
    import sys
    sys.path.insert(0, os.path.dirname(__file__))
    import sim
    S, B = 6, 4
    o = oracle.Oracle(dict(block=B, key_blocks=1, seeds=(1, 2), vnodes=4, max_slots=S))
    rng = np.random.default_rng(300 + seed)
    base = rng.integers(0, 50, size=S).astype(np.int64)
    qs = sim.QueueState(S, base)
    q = _qs_csr(qs)
    rec_base = 0
    for step in range(5):
        nb = int(rng.integers(1, 30))
        lens = rng.integers(0, 40, size=nb)
        off = np.zeros(nb + 1, np.int64)
        off[1:] = np.cumsum(lens)
        c1 = rng.integers(0, S, size=nb)
        c2 = (c1 + rng.integers(1, S, size=nb)) % S
        cand = np.concatenate([c1, c2]).astype(np.uint32)
        match = np.concatenate([rng.integers(0, 1 + lens // B), rng.integers(0, 1 + lens // B)])
        match = np.minimum(match, np.concatenate([lens // B, lens // B])).astype(np.uint32)
        chosen = np.where(rng.random(nb) < 0.5, c1, c2).astype(np.uint32)
        q = list(o.queue_append(q, off, cand, match, chosen, rec_base))
        u1 = lens - B * match[:nb].astype(np.int64)
        u2 = lens - B * match[nb:].astype(np.int64)
        first = chosen == c1
        qs.append(np.arange(rec_base, rec_base + nb, dtype=np.uint64), chosen,
                  np.where(first, c2, c1), np.where(first, u1, u2), np.where(first, u2, u1))
        rec_base += nb
        for a, b in zip(q, _qs_csr(qs)):
            assert np.array_equal(a, b)
        # migrate a few records from their queues to their alternatives
        Q = int(q[0][-1])
        if Q:
            pick = rng.choice(Q, size=min(Q, int(rng.integers(0, 6))), replace=False)
            owner = np.searchsorted(q[0], np.arange(Q), side="right") - 1
            mrec, msrc, mdst = q[1][pick], owner[pick].astype(np.uint32), q[3][pick]
            q = list(o.queue_migrate(q, mrec, msrc, mdst))
            qs.migrate(mrec, msrc, mdst)
            for a, b in zip(q, _qs_csr(qs)):
                assert np.array_equal(a, b)
        units = rng.integers(0, 80, size=S).astype(np.int64)
        q = list(o.queue_drain(q, units))
        qs.drain(units)
        for a, b in zip(q, _qs_csr(qs)):
            assert np.array_equal(a, b)


def test_queue_reprobe_hand_values():
    """Instance 0 caches blocks {10, 11}, instance 1 {10}; B = 16.  Chain
    [10, 11, 12] of 100 tokens: 2 blocks cached on 0 (68 uncached), 1 on 1
    (84).  Chain [11, 10] of 40 tokens queued on 1: none there (40), both on
    0 (8).  An empty chain of 5 tokens: 5 everywhere."""
    o = oracle.Oracle(dict(block=16, key_blocks=1, seeds=(1, 2), vnodes=4, max_slots=2))
    o.index_insert(0, np.array([10, 11], np.uint64))
    o.index_insert(1, np.array([10], np.uint64))
    coff = np.array([0, 3, 3, 5], np.int64)
    keys = np.array([10, 11, 12, 11, 10], np.uint64)
    plen = np.array([100, 5, 40], np.int64)
    q = (np.array([0, 1, 3], np.int64), np.array([0, 1, 2], np.uint64),
         np.array([1, 2, 3], np.uint32), np.array([1, 0, 0], np.uint32),
         np.array([4, 5, 6], np.uint32), np.array([7, 9], np.int64))
    qoff, rec, here, alt, there, base = o.queue_reprobe(q, coff, keys, plen)
    assert here.tolist() == [68, 5, 40] and there.tolist() == [84, 5, 8]
    assert qoff.tolist() == [0, 1, 3] and rec.tolist() == [0, 1, 2]
    assert alt.tolist() == [1, 0, 0] and base.tolist() == [7, 9]
    with pytest.raises(RuntimeError):  # an id without a chain
        o.queue_reprobe(q, coff[:3], keys, plen[:2])
    with pytest.raises(RuntimeError):  # 2 blocks of 16 cannot fit 31 tokens
        o.queue_reprobe(q, coff, keys, np.array([100, 5, 31], np.int64))


def test_queue_reprobe_matches_routing_until_caches_change():
    """Right after routing, the re-probed uncached tokens are the ones the
    routing pass computed (append's), and they stay so after migrations
    (roles swap with the records).  Once a record's whole chain is saved on
    its alternative, its cost there is just the partial tail, len mod B."""
    import oracle.harness as oh
    wl = workloads.small_random(41, 6, 8, 16, 200)
    o = oh.oracle_for(wl)
    oh.prefill_from_prior(o, wl)
    B = wl.route.block
    tok, off = workloads.prompts(wl, wl.n_req, sub=0)
    n = len(off) - 1
    r = o.route(tok, off, workloads.initial_loads(wl, wl.route.max_slots), block_keys=True)
    S = wl.route.max_slots
    empty = (np.zeros(S + 1, np.int64), np.zeros(0, np.uint64), np.zeros(0, np.uint32),
             np.zeros(0, np.uint32), np.zeros(0, np.uint32), np.zeros(S, np.int64))
    q = o.queue_append(empty, off, r["cand"], r["match"], r["chosen"], 0)
    lens = np.diff(off)
    coff = np.zeros(n + 1, np.int64)
    coff[1:] = np.cumsum(lens // B)
    q2 = o.queue_reprobe(q, coff, r["block_keys"], lens)
    for a, b in zip(q, q2):
        assert np.array_equal(a, b)
    Q = int(q[0][-1])
    owner = np.searchsorted(q[0], np.arange(Q), side="right") - 1
    pick = np.arange(0, Q, 3)
    q = o.queue_migrate(q, q[1][pick], owner[pick].astype(np.uint32), q[3][pick])
    q2 = o.queue_reprobe(q, coff, r["block_keys"], lens)
    for a, b in zip(q, q2):
        assert np.array_equal(a, b)
    # save some records' chains on their alternatives
    saved = q[1][::4].astype(np.int64)
    alt_of = dict(zip(q[1].tolist(), q[3].tolist()))
    for rid in saved.tolist():
        o.index_insert(alt_of[rid], r["block_keys"][coff[rid]:coff[rid + 1]])
    q3 = o.queue_reprobe(q, coff, r["block_keys"], lens)
    pos = {rid: i for i, rid in enumerate(q[1].tolist())}
    for rid in saved.tolist():
        assert q3[4][pos[rid]] == lens[rid] % B
    # every record, one cached block at a time through the index
    for i in range(S):
        for p in range(q3[0][i], q3[0][i + 1]):
            rid = int(q3[1][p])
            chain = r["block_keys"][coff[rid]:coff[rid + 1]]
            for inst, got in ((i, q3[2][p]), (int(q3[3][p]), q3[4][p])):
                m = 0
                while m < len(chain) and o.index_contains(inst, int(chain[m])):
                    m += 1
                assert got == lens[rid] - B * m


def test_queue_drain_hand_values():
    """Base 5 and records of 3, 4, 6 tokens: 10 units serve the base (5),
    the first record (3) and 2 of the second, which keeps 2."""
    S = 1
    o = oracle.Oracle(dict(block=4, key_blocks=1, seeds=(1, 2), vnodes=4, max_slots=S))
    q = (np.array([0, 3], np.int64), np.array([7, 8, 9], np.uint64),
         np.array([3, 4, 6], np.uint32), np.zeros(3, np.uint32), np.array([1, 1, 1], np.uint32),
         np.array([5], np.int64))
    qoff, rec, here, alt, there, base = o.queue_drain(q, np.array([10], np.int64))
    assert qoff.tolist() == [0, 2] and rec.tolist() == [8, 9] and here.tolist() == [2, 6]
    assert base.tolist() == [0]
