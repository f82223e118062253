"""Pins for the oracle's cache semantics, Belady bound and metrics (CPU only)."""
import os

import numpy as np
import pytest

from oracle import belady, metrics
from oracle.cache import (F_HIT, F_ISSUED, F_RES_AFTER, F_RES_START, KIND_ACCESS,
                          KIND_PREFETCH, LayerCache, Rec)
from tests._bruteforce import ListCache

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _read_golden(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(line.split())
    return rows


def _random_trace(rng, E, k, T, skew=True):
    p = None
    if skew:
        p = rng.dirichlet(np.full(E, 0.5))
    return [list(rng.choice(E, size=k, replace=False, p=p)) for _ in range(T)]


# ---- the oracle against the list-scan formulation -----------------------------
POLICIES = ["lru", "lfu", "lfu-aged:1", "lfu-aged:4", "lfu-aged:32"]


@pytest.mark.parametrize("policy", POLICIES)
def test_cache_matches_list_scan_on_random_traces(policy):
    rng = np.random.default_rng(11 + POLICIES.index(policy))
    for _ in range(300):
        E = int(rng.integers(2, 9))
        k = int(rng.integers(1, min(E, 4) + 1))
        S = int(rng.integers(k, E + 1))
        T = int(rng.integers(1, 200))
        trace = _random_trace(rng, E, k, T, skew=rng.random() < 0.7)
        a, b = LayerCache(E, S, policy), ListCache(E, S, policy)
        for ids in trace:
            assert [r.astuple() for r in a.access(ids)] == b.access(ids)


@pytest.mark.parametrize("policy", POLICIES)
def test_prefetch_matches_list_scan(policy):
    rng = np.random.default_rng(13)
    for _ in range(200):
        E = int(rng.integers(2, 9))
        k = int(rng.integers(1, min(E, 3) + 1))
        S = int(rng.integers(k, E + 1))
        m = int(rng.integers(0, k + 1))
        a, b = LayerCache(E, S, policy), ListCache(E, S, policy)
        for ids in _random_trace(rng, E, k, int(rng.integers(1, 80))):
            if rng.random() < 0.7:
                guesses = list(rng.choice(E, size=k, replace=False))
                assert [r.astuple() for r in a.prefetch(guesses, m)] == b.prefetch(guesses, m)
            assert [r.astuple() for r in a.access(ids)] == b.access(ids)


def test_cold_start_textbook_reference_string():
    # The classic page-replacement exercise: reference string
    # 7 0 1 2 0 3 0 4 2 3 0 3 2 1 2 0 1 7 0 1 with 3 empty frames gives
    # 12 faults under LRU and 9 under the optimal (MIN) policy.
    seq = [7, 0, 1, 2, 0, 3, 0, 4, 2, 3, 0, 3, 2, 1, 2, 0, 1, 7, 0, 1]
    c = LayerCache(8, 3, "lru", initial=[-1, -1, -1])
    misses = sum(1 for x in seq for r in c.access([x]) if not r.flags & F_HIT)
    assert misses == 12
    assert len(seq) - belady.min_hits(seq, 3, [-1, -1, -1]) == 9


def test_hand_worked_lru_and_lfu():
    # E = 4, S = 2, K = 1, warm start slots [0, 1] (expert 0 least recent),
    # demand 2 0 2 3 0 0 1.  Worked by hand from the definitions:
    # LRU: t0 2 evicts 0 (slot 0); t1 0 evicts 1 (slot 1); t2 hit 2;
    #      t3 3 evicts 0 (last 2 < 3); t4 0 evicts 2 (slot 0); t5 hit; t6 1 evicts 3.
    # LFU: as LRU up to t3; t4 0 evicts 3 (count 1 < count(2) = 2) from slot 1;
    #      t5 hit; t6 1 evicts 2 (count 2 < count(0) = 3) from slot 0.
    seq = [2, 0, 2, 3, 0, 0, 1]
    want = {
        "lru": [(0, 0, 0), (0, 1, 1), (1, 0, -1), (0, 1, 0), (0, 0, 2), (1, 0, -1), (0, 1, 3)],
        "lfu": [(0, 0, 0), (0, 1, 1), (1, 0, -1), (0, 1, 0), (0, 1, 3), (1, 1, -1), (0, 0, 2)],
    }
    for policy, rows in want.items():
        c = LayerCache(4, 2, policy)
        got = [(r.flags & F_HIT, r.slot, r.victim) for x in seq for r in c.access([x])]
        assert got == rows, policy
    # MIN from the same start: 2 evicts 1 (next use furthest), 3 evicts 2 (never
    # used again): hits at 0, 2, 0, 0.
    assert belady.min_hits(seq, 2, [0, 1]) == 4


def test_hand_worked_aged_lfu():
    # E = 4, S = 3, K = 1, warm start slots [0, 1, 2], period A = 2,
    # demand 0 0 0 0 1 1 2 3 0 (one clock tick per lookup, ticks 1..9).
    # Ticks 1-7 hit: count 0/1/2 = 4/2/1, last 0/1/2 = 4/6/7.
    # Tick 8, 3 misses: ages 4/2/1 give aged counts 4>>2 = 1, 2>>1 = 1,
    #   1>>0 = 1; equal, so the least recent goes: 0 leaves slot 0.
    #   (LFU would evict 2, the smallest count.)
    # Tick 9, 0 misses: candidates 3 (count 1, age 1 -> 1), 1 (count 2, age 3
    #   -> 2>>1 = 1), 2 (count 1, age 2 -> 1>>1 = 0): 2 leaves slot 2.
    #   (LRU would evict 1, the least recent.)
    seq = [0, 0, 0, 0, 1, 1, 2, 3, 0]
    want = [(1, 0, -1)] * 4 + [(1, 1, -1)] * 2 + [(1, 2, -1), (0, 0, 0), (0, 2, 2)]
    got = {}
    for policy in ("lfu-aged:2", "lru", "lfu"):
        c = LayerCache(4, 3, policy)
        got[policy] = [(r.flags & F_HIT, r.slot, r.victim) for x in seq for r in c.access([x])]
    assert got["lfu-aged:2"] == want
    assert got["lru"] != want and got["lfu"] != want
    assert LayerCache(4, 3, "lfu-aged:2").key(0)[0] == 0   # count 0 ages to 0


def test_aged_lfu_with_a_long_period_is_lfu():
    rng = np.random.default_rng(23)
    for _ in range(100):
        E = int(rng.integers(2, 12))
        k = int(rng.integers(1, min(E, 4) + 1))
        S = int(rng.integers(k, E + 1))
        a, b = LayerCache(E, S, "lfu-aged:1000000"), LayerCache(E, S, "lfu")
        for ids in _random_trace(rng, E, k, int(rng.integers(1, 100))):
            if rng.random() < 0.3:
                g = list(rng.choice(E, size=k, replace=False))
                assert [r.astuple() for r in a.prefetch(g, 1)] == [r.astuple() for r in b.prefetch(g, 1)]
            assert [r.astuple() for r in a.access(ids)] == [r.astuple() for r in b.access(ids)]
        batch = _random_trace(rng, E, k, int(rng.integers(1, 30)))
        assert [r.astuple() for r in a.prefill(batch)] == [r.astuple() for r in b.prefill(batch)]


def test_aged_lfu_policy_spec():
    from oracle.cache import parse_policy
    assert parse_policy("lfu-aged:32") == ("lfu-aged", 32)
    assert parse_policy("lru") == ("lru", None)
    for bad in ("lfu-aged", "lfu-aged:0", "lfu-aged:-3", "lru:2", "mru"):
        with pytest.raises(ValueError):
            LayerCache(4, 2, bad)


def test_all_slots_means_all_hits_and_persistent_routing_means_no_later_misses():
    rng = np.random.default_rng(14)
    for policy in ("lru", "lfu"):
        c = LayerCache(6, 6, policy)
        assert all(r.flags & F_HIT for ids in _random_trace(rng, 6, 2, 50)
                   for r in c.access(ids))
        c = LayerCache(8, 3, policy)
        fixed = [5, 7]
        recs = [c.access(fixed) for _ in range(20)]
        assert all(r.flags & F_HIT for rr in recs[1:] for r in rr)


def test_counts_persist_across_eviction():
    c = LayerCache(4, 2, "lfu")
    for _ in range(3):
        c.access([3])      # 3 gets count 3, resident
    c.access([2])          # 2 evicts the other expert
    c.access([1])          # 1 evicts 2 (count 1 < 3)
    assert c.count[3] == 3 and c.expert_slot[2] == -1 and c.count[2] == 1
    c.access([2])          # 2 returns: its count continues from 1
    assert c.count[2] == 2


def test_whole_token_is_pinned():
    # With S = K the token's own experts must never evict one another.
    rng = np.random.default_rng(15)
    for policy in ("lru", "lfu"):
        c = LayerCache(6, 3, policy)
        for ids in _random_trace(rng, 6, 3, 100):
            c.access(ids)
            assert set(c.resident()) == set(ids)


# ---- Belady ------------------------------------------------------------------
def test_min_equals_exhaustive_on_tiny_traces():
    rng = np.random.default_rng(16)
    for _ in range(300):
        E = int(rng.integers(2, 6))
        S = int(rng.integers(1, min(3, E) + 1))
        seq = list(rng.integers(0, E, size=int(rng.integers(1, 11))))
        init = list(range(S)) if rng.random() < 0.5 else [-1] * S
        assert belady.min_hits(seq, S, init) == belady.exhaustive_max_hits(seq, S, init)


@pytest.mark.parametrize("policy", POLICIES)
def test_policies_never_beat_min(policy):
    rng = np.random.default_rng(17)
    for _ in range(200):
        E = int(rng.integers(2, 9))
        k = int(rng.integers(1, min(E, 3) + 1))
        S = int(rng.integers(k, E + 1))
        trace = _random_trace(rng, E, k, int(rng.integers(1, 120)))
        c = LayerCache(E, S, policy)
        hits = sum(bool(r.flags & F_HIT) for ids in trace for r in c.access(ids))
        assert hits <= belady.min_hits(belady.flatten(trace), S, list(range(S)))


# ---- prefetch semantics ---------------------------------------------------------
def test_prefetch_max_zero_leaves_access_trace_unchanged():
    rng = np.random.default_rng(18)
    for policy in ("lru", "lfu"):
        a, b = LayerCache(8, 4, policy), LayerCache(8, 4, policy)
        for ids in _random_trace(rng, 8, 2, 100):
            recs = a.prefetch(list(rng.choice(8, 2, replace=False)), 0)
            assert all(not (r.flags & F_ISSUED) for r in recs)
            assert [r.astuple() for r in a.access(ids)] == [r.astuple() for r in b.access(ids)]


def test_perfect_guesses_remove_all_demand_misses():
    rng = np.random.default_rng(19)
    for policy in ("lru", "lfu"):
        c = LayerCache(8, 4, policy, layer=1)
        for ids in _random_trace(rng, 8, 2, 100):
            pf = c.prefetch(ids, 2)
            acc = c.access(ids)
            assert all(r.flags & F_HIT for r in acc)
            issued = sum(bool(r.flags & F_ISSUED) for r in pf)
            assert sum(bool(r.flags & 2) for r in acc) == issued   # every issued one used
        assert c.stats.pf_wasted == 0


def test_prefetch_does_not_count_as_use():
    c = LayerCache(4, 2, "lfu")
    c.prefetch([3, 0], 2)
    assert c.count[3] == 0 and c.expert_slot[3] >= 0
    assert c.clock == 1


# ---- metrics: the paper's identities ---------------------------------------------
def test_recall_is_twice_precision_for_four_slots_top2_and_table2_agrees():
    rng = np.random.default_rng(20)
    for policy in ("lru", "lfu"):
        c = LayerCache(8, 4, policy)
        recs = [r for ids in _random_trace(rng, 8, 2, 300) for r in c.access(ids)]
        p, r = metrics.cache_pr(recs, 4)
        assert r == pytest.approx(2 * p, rel=1e-12)
        assert r == pytest.approx(metrics.hit_rate(recs), rel=1e-12)
    for _, prec, rec in _read_golden("table2_cache_precision_recall.txt"):
        assert float(rec) == pytest.approx(2 * float(prec), abs=1e-9)


def test_guess_precision_equals_recall_and_sec54_value():
    rng = np.random.default_rng(21)
    recs = []
    for t in range(200):
        for l in range(1, 4):
            ids = rng.choice(8, 2, replace=False)
            guesses = rng.choice(8, 2, replace=False)
            recs += [Rec(KIND_PREFETCH, t, l, i, int(g), 0, -1, -1) for i, g in enumerate(guesses)]
            recs += [Rec(KIND_ACCESS, t, l, i, int(e), 0, -1, -1) for i, e in enumerate(ids)]
        # layer 0 has activations but never a guess: it must not enter the statistic
        recs += [Rec(KIND_ACCESS, t, 0, i, i, 0, -1, -1) for i in range(2)]
    p, r, tp, ng, na = metrics.guess_pr(recs)
    assert p == r and ng == na == 200 * 3 * 2
    (prec, rec), = _read_golden("sec54_guess_precision_recall.txt")
    assert float(prec) == float(rec)


def test_random_repeat_probability_sec31():
    (E, pct), = _read_golden("sec31_random_repeat.txt")
    assert 100.0 / int(E) == pytest.approx(float(pct))


def test_table2_lfu_speedup_on_a6000_is_846_percent():
    rows = {g: (float(a), float(b)) for g, a, b in _read_golden("table2_tokens_per_second.txt")}
    lru, lfu = rows["A6000"]
    assert round(100 * (lfu / lru - 1), 1) == 84.6


# ---- prefill residency rule ------------------------------------------------------
def test_prefill_counts_and_residency_rule():
    rng = np.random.default_rng(22)
    for policy in ("lfu", "lru", "lfu-aged:3"):
        for _ in range(100):
            E = int(rng.integers(4, 17))
            k = int(rng.integers(1, min(4, E) + 1))
            S = int(rng.integers(k, E + 1))
            c = LayerCache(E, S, policy)
            for ids in _random_trace(rng, E, k, int(rng.integers(0, 20))):
                c.access(ids)
            before = dict(enumerate(c.slot_expert))
            start = set(c.resident())
            cnt0 = list(c.count)
            batch = _random_trace(rng, E, k, int(rng.integers(1, 60)))
            recs = c.prefill(batch)
            n = np.bincount(np.array(batch).reshape(-1), minlength=E)
            assert sum(c.count) - sum(cnt0) == len(batch) * k
            assert [r.rank for r in recs] == list(n)
            # brute force R*: sort every expert by the stated key
            if policy == "lfu":
                order = sorted(range(E), key=lambda e: (-(cnt0[e] + n[e]), e not in start, e))
            elif policy == "lfu-aged:3":
                aged = [(cnt0[e] + n[e]) >> ((c.clock - c.last[e]) // 3) for e in range(E)]
                order = sorted(range(E), key=lambda e: (-aged[e], e not in start, e))
            else:
                order = sorted(range(E), key=lambda e: (-c.last[e], e not in start, e))
            rstar = set(order[:S])
            assert set(c.resident()) == rstar
            for s, e in before.items():
                if e in rstar:
                    assert c.slot_expert[s] == e          # kept experts keep slots
            for r in recs:
                assert bool(r.flags & F_RES_START) == (r.expert in start)
                assert bool(r.flags & F_RES_AFTER) == (r.expert in rstar)


def test_hand_worked_aged_lfu_prefill():
    # E = 4, S = 2, K = 1, warm start slots [0, 1], period A = 2.  Lookups
    # 0 0 0 (ticks 1-3: count(0) = 3, last(0) = 3), then one batch of rows
    # 2 2 1 3 (ticks 4-7).  At tick 7: counts 3/1/2/1, last 3/6/5/7, so the
    # aged counts are 3>>2 = 0, 1>>0 = 1, 2>>1 = 1, 1>>0 = 1.  The three
    # tied at 1 order resident-first (1), then by id (2): R* = {1, 2}.
    # (LFU would keep {0, 2}, LRU {3, 1}.)  Expert 1 keeps slot 1; 2 takes
    # slot 0 from 0; 3 streams through without a slot.
    c = LayerCache(4, 2, "lfu-aged:2")
    for _ in range(3):
        c.access([0])
    recs = [r.astuple() for r in c.prefill([[2], [2], [1], [3]])]
    assert recs == [(2, 3, 0, 0, 0, 1, -1, -1), (2, 3, 0, 1, 1, 3, 1, -1),
                    (2, 3, 0, 2, 2, 6, 0, 0), (2, 3, 0, 1, 3, 4, -1, -1)]
    for policy, keep in (("lfu", {0, 2}), ("lru", {1, 3})):
        c = LayerCache(4, 2, policy)
        for _ in range(3):
            c.access([0])
        c.prefill([[2], [2], [1], [3]])
        assert set(c.resident()) == keep
