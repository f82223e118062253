"""The package's trace analytics agree with the oracle's metrics on traces the
oracle's caches produce (CPU only)."""
import numpy as np
import pytest

from oracle import belady, metrics
from oracle.cache import LayerCache
from paper_2511_05814_amd import analysis


def _trace(seed, policy, prefetch):
    rng = np.random.default_rng(seed)
    L, E, K, S = 3, 8, 2, 4
    caches = [LayerCache(E, S, policy, layer=l) for l in range(L)]
    p = rng.dirichlet(np.full(E, 0.5))
    recs = []
    for t in range(150):
        for l in range(L):
            ids = rng.choice(E, K, replace=False, p=p)
            recs += caches[l].access(ids)
            if prefetch and l + 1 < L:
                recs += caches[l + 1].prefetch(rng.choice(E, K, replace=False, p=p), 2)
    return recs


@pytest.mark.parametrize("policy,prefetch", [("lru", False), ("lfu", False), ("lfu", True)])
def test_analysis_matches_oracle_metrics(policy, prefetch):
    recs = _trace(3, policy, prefetch)
    tup = [r.astuple() for r in recs]
    assert analysis.hit_rate(tup) == pytest.approx(metrics.hit_rate(recs))
    assert analysis.cache_precision_recall(tup, 4) == pytest.approx(metrics.cache_pr(recs, 4))
    assert analysis.per_layer_hit_rate(tup) == pytest.approx(metrics.per_layer_hit_rate(recs))
    if prefetch:
        p, r = analysis.guess_precision_recall(tup)
        op, orr, *_ = metrics.guess_pr(recs)
        assert (p, r) == pytest.approx((op, orr)) and p == r
        assert analysis.transfer_precision(tup) == pytest.approx(metrics.transfer_precision(recs))


def test_histogram_and_repeat_rate():
    recs = [(0, t, 0, r, e, 0, 0, -1) for t, ids in enumerate([[1, 2], [2, 3], [2, 3], [5, 6]])
            for r, e in enumerate(ids)]
    assert analysis.activation_histogram(recs, 0, 8) == [0, 1, 3, 2, 0, 1, 1, 0]
    # token 1 repeats 1 of 2 (expert 2), token 2 repeats 2 of 2, token 3 none
    assert analysis.repeat_rate(recs, 0) == pytest.approx(3 / 6)


@pytest.mark.parametrize("policy", ["lru", "lfu"])
def test_belady_matches_oracle_min_and_bounds_the_policy(policy):
    recs = _trace(5, policy, False)
    tup = [r.astuple() for r in recs]
    seqs = analysis.demand_sequences(tup)
    for l, seq in seqs.items():
        assert analysis.belady_hits(seq, 4) == belady.min_hits(seq, 4, list(range(4)))
        hits = sum(1 for r in tup if r[0] == 0 and r[2] == l and r[5] & 1)
        assert hits <= analysis.belady_hits(seq, 4)
    assert analysis.belady_hit_rate(tup, 4) >= analysis.hit_rate(tup)


def test_belady_textbook_and_exhaustive():
    # the 20-reference string with 3 frames from an empty cache: OPT has 9
    # faults, i.e. 11 hits; a warm start of experts 0..2 is a different start,
    # so check against the exhaustive optimum from that start instead
    seq = [7, 0, 1, 2, 0, 3, 0, 4, 2, 3, 0, 3, 2, 1, 2, 0, 1, 7, 0, 1]
    assert analysis.belady_hits(seq, 3) == belady.exhaustive_max_hits(seq, 3, [0, 1, 2])
    rng = np.random.default_rng(9)
    for _ in range(30):
        seq = list(rng.integers(0, 5, size=10))
        for s in (1, 2, 3):
            assert analysis.belady_hits(seq, s) == belady.exhaustive_max_hits(seq, s, list(range(s)))
