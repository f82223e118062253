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


# Hand-worked guesses for three layers and three tokens (E = 4, K = 2).  Layer
# 0 has activations only (nothing guesses it).  Per (layer, token):
#   activations  L0: {0,1} {0,2} {1,3}   L1: {2,3} {2,0} {1,0}   L2: {0,3} {1,2} {3,2}
#   guesses                              L1: {2,3} {2,1} {0,1}   L2: {0,1} {1,2} {3,0}
#   true pos.                            L1:   2     1     2     L2:   1     2     1
# so TP = 9 of 12 guesses and 12 activations: P = R = 3/4 (Sec. 5.4).
_HAND_ACT = {0: [[0, 1], [0, 2], [1, 3]], 1: [[2, 3], [2, 0], [1, 0]], 2: [[0, 3], [1, 2], [3, 2]]}
_HAND_GUESS = {1: [[2, 3], [2, 1], [0, 1]], 2: [[0, 1], [1, 2], [3, 0]]}


def _hand_records(guess_layer_shift=0, guess_token_shift=0):
    recs = []
    for l, rows in _HAND_ACT.items():
        for t, ids in enumerate(rows):
            recs += [Rec(KIND_ACCESS, t, l, r, e, 0, -1, -1) for r, e in enumerate(ids)]
    for l, rows in _HAND_GUESS.items():
        for t, ids in enumerate(rows):
            recs += [Rec(KIND_PREFETCH, t + guess_token_shift, l + guess_layer_shift, r, e, 0, -1, -1)
                     for r, e in enumerate(ids)]
    return recs


def test_guess_pr_hand_worked_three_layers_three_tokens():
    assert metrics.guess_pr(_hand_records()) == (0.75, 0.75, 9, 12, 12)
    # a guess belongs to the guessed layer and the same token: keyed one token
    # late, L1 t0 {2,3} meets t1 {2,0} (1), L1 t1 meets t2 (1), L2 t0 {0,1}
    # meets {1,2} (1), L2 t1 {1,2} meets {3,2} (1); the t2 guesses find no
    # activations: 4 of 8
    assert metrics.guess_pr(_hand_records(guess_token_shift=1)) == (0.5, 0.5, 4, 8, 8)
    # keyed to the layer that made the guess (l - 1): L1's guesses against
    # L0's activations give 0 + 1 + 1, L2's against L1's 0 + 1 + 1: 4 of 12
    p, r, tp, ng, na = metrics.guess_pr(_hand_records(guess_layer_shift=-1))
    assert (tp, ng, na) == (4, 12, 12) and p == r == pytest.approx(1 / 3)
    # perfect guesses (guess = the same token's activations at that layer)
    perfect = [Rec(KIND_PREFETCH, t, l, r, e, 0, -1, -1)
               for l in (1, 2) for t, ids in enumerate(_HAND_ACT[l]) for r, e in enumerate(ids)]
    acts = [x for x in _hand_records() if x.kind == KIND_ACCESS]
    assert metrics.guess_pr(acts + perfect) == (1.0, 1.0, 12, 12, 12)
    # the product's analytics give the same numbers on the same records
    from paper_2511_05814_amd import analysis
    for shift, want in (({}, 0.75), ({"guess_token_shift": 1}, 0.5)):
        tup = [x.astuple() for x in _hand_records(**shift)]
        assert analysis.guess_precision_recall(tup) == (want, want)


def test_transfer_precision_hand_worked_lfu():
    # One layer's cache (layer 1), E = 5, S = 3, K = 2, LFU, warm start
    # slots [0, 1, 2], last = -3, -2, -1 (experts 3 and 4: -4).  Keys
    # (count, last, slot); prefetches tick the clock but leave counts alone.
    c = LayerCache(5, 3, "lfu", layer=1)
    recs = []
    # token 0: guesses [3, 0] (max 2).  3 is fetched at tick 1 into slot 1,
    # evicting 1 (key (0,-2,1) < (0,-1,2); 0 is pinned as a guess); 0 is resident.
    recs += c.prefetch([3, 0], 2)
    # access [3, 4]: 3 hits and is the prefetch's first use (useful); 4 misses
    # at tick 3 and evicts 0 (slot 0, key (0,-3,0)).
    recs += c.access([3, 4])
    # token 1: guesses [1, 0] (max 2).  1 at tick 4 evicts 2 (count 0) from slot
    # 2; 0 at tick 5 evicts 3 (key (1,2,1) < 4's (1,3,0)) from slot 1.
    recs += c.prefetch([1, 0], 2)
    # access [0, 2]: 0 hits (useful); 2 misses at tick 7 and evicts the
    # prefetched, never used 1 (count 0): wasted before its use.
    recs += c.access([0, 2])
    # token 2: guesses [3, 1] (max 1).  3 at tick 8 evicts 4 (key (1,3,0));
    # 1 is not fetched (cap reached).
    recs += c.prefetch([3, 1], 1)
    # access [1, 0]: 1 misses at tick 9 and evicts 2 (key (1,7,2) before 3's
    # (1,8,0)); 0 hits; the prefetched 3 was never used: wasted.
    recs += c.access([1, 0])
    assert [r.astuple() for r in recs] == [
        (1, 0, 1, 0, 3, 2, 1, 1), (1, 0, 1, 1, 0, 1, 0, -1),
        (0, 0, 1, 0, 3, 3, 1, -1), (0, 0, 1, 1, 4, 0, 0, 0),
        (1, 1, 1, 0, 1, 2, 2, 2), (1, 1, 1, 1, 0, 2, 1, 3),
        (0, 1, 1, 0, 0, 3, 1, -1), (0, 1, 1, 1, 2, 0, 2, 1),
        (1, 2, 1, 0, 3, 2, 0, 4), (1, 2, 1, 1, 1, 0, -1, -1),
        (0, 2, 1, 0, 1, 0, 2, 2), (0, 2, 1, 1, 0, 1, 1, -1),
    ]
    s = c.stats
    assert (s.pf_guesses, s.pf_issued, s.pf_useful, s.pf_wasted) == (6, 4, 2, 2)
    assert metrics.transfer_precision(recs) == 0.5          # 2 useful of 4 issued
    # guesses {3,0} {1,0} {3,1} against activations {3,4} {0,2} {1,0}: 1 + 1 + 1
    assert metrics.guess_pr(recs) == (0.5, 0.5, 3, 6, 6)
    from paper_2511_05814_amd import analysis
    tup = [r.astuple() for r in recs]
    assert analysis.transfer_precision(tup) == 0.5
    assert analysis.guess_precision_recall(tup) == (0.5, 0.5)
    # with perfect guesses every fetched guess is used: transfer precision 1
    c = LayerCache(5, 3, "lfu", layer=1)
    recs = []
    for ids in ([3, 4], [0, 2], [1, 0]):
        recs += c.prefetch(ids, 2) + c.access(ids)
    assert c.stats.pf_issued == 4 and c.stats.pf_wasted == 0
    assert metrics.transfer_precision(recs) == 1.0
    assert metrics.guess_pr(recs)[:2] == (1.0, 1.0)


def test_cache_pr_reproduces_table2_pairs():
    # a run of 1000 lookups of K = 2 with 1164 (LRU) or 1196 (LFU) hits and 4
    # slots gives exactly Table 2's printed cache precision / recall
    for _, prec, rec in _read_golden("table2_cache_precision_recall.txt"):
        hits = round(float(rec) * 20)
        recs = [Rec(KIND_ACCESS, t, 0, r, r, F_HIT if 2 * t + r < hits else 0, r, -1)
                for t in range(1000) for r in range(2)]
        p, r = metrics.cache_pr(recs, 4)
        assert (round(100 * p, 1), round(100 * r, 1)) == (float(prec), float(rec))


def test_histogram_and_repeat_rates_hand_worked():
    # layer 0, four lookups: [1, 2] [2, 3] [2, 3] [5, 6]; layer 1 is noise
    rows = [[1, 2], [2, 3], [2, 3], [5, 6]]
    recs = [Rec(KIND_ACCESS, t, 0, r, e, 0, -1, -1) for t, ids in enumerate(rows) for r, e in enumerate(ids)]
    recs += [Rec(KIND_ACCESS, t, 1, r, (e + 3) % 8, 0, -1, -1) for t, ids in enumerate(rows)
             for r, e in enumerate(ids)]
    assert metrics.activation_histogram(recs, 0, 8) == [0, 1, 3, 2, 0, 1, 1, 0]
    # token 1 repeats 2 (1 of 2), token 2 repeats 2 and 3 (2 of 2), token 3 none
    assert metrics.repeat_rate(recs, 0) == 3 / 6
    # first-ranked experts 1, 2, 2, 5: one repeat in three consecutive pairs
    assert metrics.top1_repeat_rate(recs, 0) == 1 / 3
    # a gap in the lookup indices breaks the pair
    gap = [x for x in recs if not (x.layer == 0 and x.token == 1)]
    assert metrics.top1_repeat_rate(gap, 0) == 0.0 and metrics.repeat_rate(gap, 0) == 0.0
    from paper_2511_05814_amd import analysis
    tup = [x.astuple() for x in recs]
    assert analysis.activation_histogram(tup, 0, 8) == metrics.activation_histogram(recs, 0, 8)
    assert analysis.repeat_rate(tup, 0) == metrics.repeat_rate(recs, 0)
    assert analysis.top1_repeat_rate(tup, 0) == metrics.top1_repeat_rate(recs, 0)


def test_repeat_rates_of_random_routing_are_k_over_e_and_one_over_e():
    # Sec. 3.1: with random choices the same expert comes back with
    # probability 1/E (12.5 % for 8 experts); a top-K set shares K/E of its
    # experts with the previous one on average
    rng = np.random.default_rng(24)
    E, K, T = 8, 2, 40000
    recs = [Rec(KIND_ACCESS, t, 0, r, int(e), 0, -1, -1)
            for t in range(T) for r, e in enumerate(rng.choice(E, K, replace=False))]
    assert metrics.top1_repeat_rate(recs, 0) == pytest.approx(1 / E, abs=0.01)
    assert metrics.repeat_rate(recs, 0) == pytest.approx(K / E, abs=0.01)
    (e8, pct), = _read_golden("sec31_random_repeat.txt")
    assert 100 / int(e8) == pytest.approx(float(pct))


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
