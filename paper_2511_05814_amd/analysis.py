"""Trace analytics over the device trace (host side, integer bookkeeping only).

The paper's tracing system records, per layer and token, which experts were
activated and which were cached (Sec. 3.1), and derives cache precision and
recall (Sec. 4.2, Table 2) and the speculative guesses' precision and recall
(Sec. 5.4).  These functions compute the same quantities from the records
the library writes (`moe_trace_rec` tuples: kind, token, layer, rank, expert,
flags, slot, victim).
"""
from __future__ import annotations

from collections import defaultdict
from typing import Iterable, Sequence

ACCESS, PREFETCH, PREFILL = 0, 1, 2


def split(records: Iterable[Sequence[int]]):
    acc, pf, pre = [], [], []
    for r in records:
        (acc if r[0] == ACCESS else pf if r[0] == PREFETCH else pre).append(r)
    return acc, pf, pre


def hit_rate(records) -> float:
    acc, _, _ = split(records)
    return sum(1 for r in acc if r[5] & 1) / max(1, len(acc))


def per_layer_hit_rate(records):
    n, h = defaultdict(int), defaultdict(int)
    for r in records:
        if r[0] == ACCESS:
            n[r[2]] += 1
            h[r[2]] += r[5] & 1
    return {l: h[l] / n[l] for l in sorted(n)}


def cache_precision_recall(records, slots: int):
    """recall = activated experts found resident / activated experts;
    precision = the same hits / resident experts at each lookup (S per lookup)."""
    acc, _, _ = split(records)
    lookups = {(r[2], r[1]) for r in acc}
    hits = sum(1 for r in acc if r[5] & 1)
    if not acc:
        return 0.0, 0.0
    return hits / (slots * len(lookups)), hits / len(acc)


def guess_precision_recall(records):
    """Guesses for (layer, token) against that token's activations at that layer.
    Every wrong guess is one false positive and one false negative, so the two
    agree when each side has K experts (Sec. 5.4)."""
    act, guess = defaultdict(set), defaultdict(set)
    for r in records:
        if r[0] == ACCESS:
            act[(r[2], r[1])].add(r[4])
        elif r[0] == PREFETCH:
            guess[(r[2], r[1])].add(r[4])
    tp = ng = na = 0
    for key, g in guess.items():
        if key in act:
            tp += len(g & act[key])
            ng += len(g)
            na += len(act[key])
    return (tp / ng if ng else 0.0), (tp / na if na else 0.0)


def transfer_precision(records) -> float:
    """Prefetched experts used by the next lookup / prefetched experts fetched."""
    issued = sum(1 for r in records if r[0] == PREFETCH and r[5] & 2)
    useful = sum(1 for r in records if r[0] == ACCESS and r[5] & 2)
    return useful / issued if issued else 0.0


def activation_histogram(records, layer: int, experts: int):
    """Activations per expert at one layer (Sec. 5.2's histograms)."""
    h = [0] * experts
    for r in records:
        if r[0] == ACCESS and r[2] == layer:
            h[r[4]] += 1
    return h


def repeat_rate(records, layer: int) -> float:
    """Fraction of a token's experts that the previous token also selected at
    this layer (Sec. 3.1 compares this with 1/E for random choice)."""
    by_tok = defaultdict(set)
    for r in records:
        if r[0] == ACCESS and r[2] == layer:
            by_tok[r[1]].add(r[4])
    toks = sorted(by_tok)
    same = total = 0
    for a, b in zip(toks[:-1], toks[1:]):
        if b == a + 1:
            same += len(by_tok[a] & by_tok[b])
            total += len(by_tok[b])
    return same / total if total else 0.0


def top1_repeat_rate(records, layer: int) -> float:
    """Fraction of tokens whose first-ranked expert at this layer is the
    previous token's first-ranked expert (consecutive lookups only).  With
    uniform random routing this is 1/E, the baseline Sec. 3.1 quotes."""
    first = {}
    for r in records:
        if r[0] == ACCESS and r[2] == layer and r[3] == 0:
            first[r[1]] = r[4]
    toks = sorted(first)
    pairs = [(a, b) for a, b in zip(toks[:-1], toks[1:]) if b == a + 1]
    return sum(1 for a, b in pairs if first[a] == first[b]) / len(pairs) if pairs else 0.0


# Layers whose activation histograms Sec. 5.2 shows (1-based, as the paper
# numbers them): the first two layers and pairs around each quarter.
PAPER_HISTOGRAM_LAYERS = (1, 2, 7, 8, 15, 16, 23, 24, 31, 32)


def report(records, layers: int, experts: int, top_k: int):
    """The analyses of Sec. 3.1 and Sec. 5.2 over one run's trace: hit rate
    per layer, activation histograms of the paper's layer set (those that
    exist; 0-based layer = paper layer - 1), and per layer the share of a
    token's experts the previous token also selected (random routing: K/E)
    and the first-ranked expert's repeat rate (random routing: 1/E)."""
    acc, _, _ = split(records)
    hist_layers = [p - 1 for p in PAPER_HISTOGRAM_LAYERS if p <= layers] or list(range(min(layers, 2)))
    rep = [repeat_rate(acc, l) for l in range(layers)]
    top1 = [top1_repeat_rate(acc, l) for l in range(layers)]
    return {
        "per_layer_hit_rate": [round(v, 4) for v in per_layer_hit_rate(acc).values()],
        "activation_histograms": {str(l + 1): activation_histogram(acc, l, experts) for l in hist_layers},
        "histogram_layers_are": "1-based layer numbers as in Sec. 5.2",
        "repeat_rate": {"mean": round(sum(rep) / max(1, len(rep)), 4),
                        "per_layer": [round(v, 4) for v in rep],
                        "random_routing": round(top_k / experts, 4)},
        "top1_repeat_rate": {"mean": round(sum(top1) / max(1, len(top1)), 4),
                             "per_layer": [round(v, 4) for v in top1],
                             "random_routing": round(1 / experts, 4)},
    }


def demand_sequences(records):
    """Per layer, the experts of its access records in (token, rank) order."""
    acc, _, _ = split(records)
    by_layer = defaultdict(list)
    for r in sorted(acc, key=lambda r: (r[2], r[1], r[3])):
        by_layer[r[2]].append(r[4])
    return dict(by_layer)


def belady_hits(seq, slots: int) -> int:
    """Hits of Belady's MIN (evict the resident expert whose next use lies
    furthest ahead; never-again experts first, lower id first among those) on
    one layer's demand sequence from the warm start (experts 0..slots-1
    resident).  An upper bound for any demand-fetching policy on the same
    sequence; next uses come from one backward pass, so the cost is
    O(len(seq) * slots)."""
    n = len(seq)
    never = n  # beyond every position
    nxt = [never] * n
    seen = {}
    for i in range(n - 1, -1, -1):
        nxt[i] = seen.get(seq[i], never)
        seen[seq[i]] = i
    # next use of each warm-start expert from position 0
    first = {}
    for i, e in enumerate(seq):
        first.setdefault(e, i)
    resident = {e: first.get(e, never) for e in range(slots)}
    hits = 0
    for i, x in enumerate(seq):
        if x in resident:
            hits += 1
        else:
            victim = max(resident, key=lambda e: (resident[e], -e))
            del resident[victim]
        resident[x] = nxt[i]
    return hits


def belady_hit_rate(records, slots: int) -> float:
    """Belady MIN hit rate over every layer's demand sequence in the trace."""
    seqs = demand_sequences(records)
    total = sum(len(s) for s in seqs.values())
    return sum(belady_hits(s, slots) for s in seqs.values()) / max(1, total)
