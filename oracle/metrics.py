"""Cache and speculation metrics (test infrastructure only).

* Cache precision and recall compare the resident set with the activated set
  at each lookup (Sec. 4.2, Sec. 5.3, Table 2): recall = activated experts
  found resident / activated experts (= the hit rate), precision = activated
  experts found resident / resident experts.  With a cache that is always full
  (S resident) and K activated experts per lookup, recall = (S/K) precision;
  Table 2's pairs (29.1, 58.2) and (29.9, 59.8) satisfy it for S = 4, K = 2.
* Speculative guess precision and recall (Sec. 5.4): a guess is a true
  positive if the expert is activated at that layer for the same token.  With
  K guesses and K activations every wrong guess is one false positive and one
  false negative, so precision = recall.  Layer 0 has no guess and is left out.
* Transfer precision (this implementation's reading; the paper only logged
  guesses, Sec. 4.3): prefetched experts whose next lookup at that layer uses
  them / prefetched experts fetched.
* Per-layer activation histograms (Sec. 5.2) and the rate at which a token
  reuses the previous token's experts at a layer, compared in Sec. 3.1 with
  the 1/E of random routing.

Pins: guess_pr and transfer_precision against hand-worked three-token traces
(including records keyed one token or one layer off, which must change the
result); cache_pr against Table 2's printed pairs; the histogram and repeat
rates against hand-worked traces and against their closed forms (K/E and 1/E)
under uniform random routing.
"""
from __future__ import annotations

from collections import defaultdict
from typing import Iterable

from .cache import F_HIT, F_ISSUED, F_USEFUL, KIND_ACCESS, KIND_PREFETCH, Rec


def cache_pr(records: Iterable[Rec], slots: int):
    """(precision, recall) of the cache over the access records."""
    hits = lookups_x_k = 0
    tokens = set()
    for r in records:
        if r.kind != KIND_ACCESS:
            continue
        lookups_x_k += 1
        hits += bool(r.flags & F_HIT)
        tokens.add((r.layer, r.token))
    if not tokens:
        return 0.0, 0.0
    return hits / (slots * len(tokens)), hits / lookups_x_k


def hit_rate(records: Iterable[Rec]) -> float:
    acc = [r for r in records if r.kind == KIND_ACCESS]
    return sum(bool(r.flags & F_HIT) for r in acc) / max(1, len(acc))


def guess_pr(records: Iterable[Rec]):
    """(precision, recall, true positives, guesses, activations) of the
    next-layer guesses against the same token's activations."""
    records = list(records)
    act = defaultdict(set)
    for r in records:
        if r.kind == KIND_ACCESS:
            act[(r.layer, r.token)].add(r.expert)
    guess = defaultdict(set)
    for r in records:
        if r.kind == KIND_PREFETCH:
            guess[(r.layer, r.token)].add(r.expert)
    tp = n_guess = n_act = 0
    for key, g in guess.items():
        if key not in act:
            continue
        tp += len(g & act[key])
        n_guess += len(g)
        n_act += len(act[key])
    if n_guess == 0:
        return 0.0, 0.0, 0, 0, 0
    return tp / n_guess, tp / n_act, tp, n_guess, n_act


def transfer_precision(records: Iterable[Rec]) -> float:
    """Useful prefetches / issued prefetches, from access and prefetch records."""
    records = list(records)
    issued = sum(1 for r in records if r.kind == KIND_PREFETCH and r.flags & F_ISSUED)
    useful = sum(1 for r in records if r.kind == KIND_ACCESS and r.flags & F_USEFUL)
    return useful / issued if issued else 0.0


def per_layer_hit_rate(records: Iterable[Rec]):
    h = defaultdict(int)
    n = defaultdict(int)
    for r in records:
        if r.kind == KIND_ACCESS:
            n[r.layer] += 1
            h[r.layer] += bool(r.flags & F_HIT)
    return {l: h[l] / n[l] for l in sorted(n)}


def activation_histogram(records: Iterable[Rec], layer: int, experts: int):
    """Activations of each expert at one layer (Sec. 5.2)."""
    h = [0] * experts
    for r in records:
        if r.kind == KIND_ACCESS and r.layer == layer:
            h[r.expert] += 1
    return h


def _by_lookup(records, layer):
    ids = defaultdict(dict)
    for r in records:
        if r.kind == KIND_ACCESS and r.layer == layer:
            ids[r.token][r.rank] = r.expert
    return ids


def repeat_rate(records: Iterable[Rec], layer: int) -> float:
    """Over consecutive lookups (t-1, t) at one layer: experts of token t that
    token t-1 also selected / experts of token t."""
    ids = _by_lookup(records, layer)
    same = total = 0
    for t in sorted(ids):
        if t - 1 in ids:
            prev = set(ids[t - 1].values())
            same += sum(1 for e in ids[t].values() if e in prev)
            total += len(ids[t])
    return same / total if total else 0.0


def top1_repeat_rate(records: Iterable[Rec], layer: int) -> float:
    """Over consecutive lookups (t-1, t) at one layer: the share whose
    first-ranked experts are the same (1/E under uniform random routing)."""
    ids = _by_lookup(records, layer)
    pairs = [(ids[t - 1][0], ids[t][0]) for t in sorted(ids) if t - 1 in ids]
    return sum(1 for a, b in pairs if a == b) / len(pairs) if pairs else 0.0
