"""Per-layer expert cache semantics, step by step (test infrastructure only).

What the paper fixes:
* experts live in main memory and are loaded on demand; a fixed number of
  them per layer stays on the GPU ("cache size = 4") and a selected expert
  that is already there is reused (Sec. 2.2, Sec. 3.1, Sec. 5.1 figure captions);
* the baseline evicts the least recently used expert (Sec. 3.1);
* the proposed policy keeps one usage count per expert and evicts the least
  frequently used one (Sec. 4.2);
* a better policy would weigh popularity together with how long an expert has
  gone unused (Sec. 6.1); the third policy here is one such key;
* speculative loading applies layer l+1's gate to layer l's hidden state and
  takes its top-K as the guess for layer l+1 (Sec. 3.2, Sec. 4.3).

Readings where the paper is silent (each is listed in the design notes):
* warm start: slot s holds expert s for s < S, all counts 0, last[s] = s - S;
* a token's K experts are looked up in rank order; the clock ticks once per
  lookup; hit <=> resident when the token arrives at the layer;
* the victim of a miss is the resident expert outside the token's selected
  set that minimises (last, slot) for LRU or (count, last, slot) for LFU;
* aged LFU ("lfu-aged:A", A >= 1 ticks): the victim minimises
  (floor(count / 2^floor(age / A)), last, slot) with age = clock - last at the
  moment of the choice: the usage count halves once per A ticks without use
  (the stored count itself is never changed); with A beyond any age it is LFU;
* counts persist across eviction;
* a prefetch inserts up to `max_n` non-resident guesses in rank order, each
  taking one clock tick, victim chosen by the same key with all K guesses
  pinned; it sets last but not count; resident guesses are left untouched;
* a prefetched expert is useful iff the next demand lookup of that layer uses
  it; otherwise it is wasted (also when evicted before that lookup);
* batched prefill: counts += per-expert routing counts, the clock ticks once
  per (token, rank) in token-major order, then the S experts with the largest
  key (LFU: count, aged LFU: the aged count at the batch's last tick, LRU:
  last; ties: resident first, then lower id) become the resident set; kept experts keep their slots, newcomers take the freed slots
  (both ascending).

A cold start (`initial` with -1 entries) is supported for textbook checks:
an empty slot is always taken before any eviction, lowest slot first.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence

LRU, LFU, LFU_AGED = "lru", "lfu", "lfu-aged"


def parse_policy(spec: str):
    """'lru', 'lfu' or 'lfu-aged:A' -> (name, A or None)."""
    name, _, arg = spec.partition(":")
    if name == LFU_AGED:
        if not arg.isdigit() or int(arg) < 1:
            raise ValueError(f"aged LFU needs a period of at least one tick: {spec!r}")
        return name, int(arg)
    if name not in (LRU, LFU) or arg:
        raise ValueError(spec)
    return name, None

# record kinds and flag bits (shared vocabulary with the trace format)
KIND_ACCESS, KIND_PREFETCH, KIND_PREFILL = 0, 1, 2
F_HIT, F_USEFUL = 1, 2                       # access records
F_RESIDENT, F_ISSUED = 1, 2                  # prefetch records
F_RES_START, F_RES_AFTER, F_FETCHED = 1, 2, 4  # prefill records


@dataclass(frozen=True)
class Rec:
    kind: int
    token: int
    layer: int
    rank: int
    expert: int
    flags: int
    slot: int
    victim: int

    def astuple(self):
        return (self.kind, self.token, self.layer, self.rank, self.expert,
                self.flags, self.slot, self.victim)


@dataclass
class Stats:
    hits: int = 0
    misses: int = 0
    evictions: int = 0
    pf_guesses: int = 0
    pf_issued: int = 0
    pf_useful: int = 0
    pf_wasted: int = 0
    lookups: int = 0


class LayerCache:
    """The cache of one layer: S slots over E experts."""

    def __init__(self, experts: int, slots: int, policy: str, layer: int = 0,
                 initial: Optional[Sequence[int]] = None):
        policy, self.aging = parse_policy(policy)
        if not (1 <= slots <= experts):
            raise ValueError("need 1 <= slots <= experts")
        self.E, self.S, self.policy, self.layer = experts, slots, policy, layer
        self.slot_expert: List[int] = list(initial) if initial is not None else list(range(slots))
        if len(self.slot_expert) != slots:
            raise ValueError("initial residency must have one entry per slot")
        self.expert_slot = [-1] * experts
        self.count = [0] * experts
        self.last = [-(slots + 1)] * experts
        for s, e in enumerate(self.slot_expert):
            if e >= 0:
                self.expert_slot[e] = s
                self.last[e] = s - slots
        self.clock = 0
        self.prefetched = [False] * experts
        self.lookups = 0
        self.stats = Stats()

    # -- policy ------------------------------------------------------------
    def aged_count(self, e: int) -> int:
        """Usage count halved (rounding down) once per `aging` ticks since the
        expert's last use, at the current clock."""
        halvings = (self.clock - self.last[e]) // self.aging
        return self.count[e] // (2 ** halvings)

    def key(self, e: int):
        s = self.expert_slot[e]
        if self.policy == LRU:
            return (self.last[e], s)
        if self.policy == LFU_AGED:
            return (self.aged_count(e), self.last[e], s)
        return (self.count[e], self.last[e], s)

    def choose_victim(self, pinned) -> tuple:
        """(slot, evicted expert or -1) for an insertion with `pinned` protected."""
        for s, e in enumerate(self.slot_expert):
            if e < 0:
                return s, -1
        cands = [e for e in self.slot_expert if e not in pinned]
        if not cands:
            raise RuntimeError("no evictable slot (slots < top_k?)")
        v = min(cands, key=self.key)
        return self.expert_slot[v], v

    def _place(self, e: int, pinned) -> tuple:
        s, v = self.choose_victim(pinned)
        if v >= 0:
            self.expert_slot[v] = -1
            if self.prefetched[v]:
                self.prefetched[v] = False
                self.stats.pf_wasted += 1
        self.slot_expert[s] = e
        self.expert_slot[e] = s
        return s, v

    def resident(self) -> List[int]:
        return [e for e in self.slot_expert if e >= 0]

    # -- demand lookup of one token ------------------------------------------
    def access(self, ids: Sequence[int]) -> List[Rec]:
        ids = [int(e) for e in ids]
        if len(set(ids)) != len(ids):
            raise ValueError("duplicate expert in one token's selection")
        t = self.lookups
        self.lookups += 1
        self.stats.lookups += 1
        pinned = set(ids)
        out = []
        for r, j in enumerate(ids):
            self.clock += 1
            self.count[j] += 1
            self.last[j] = self.clock
            if self.expert_slot[j] >= 0:
                useful = self.prefetched[j]
                if useful:
                    self.prefetched[j] = False
                    self.stats.pf_useful += 1
                self.stats.hits += 1
                out.append(Rec(KIND_ACCESS, t, self.layer, r, j,
                               F_HIT | (F_USEFUL if useful else 0), self.expert_slot[j], -1))
            else:
                s, v = self._place(j, pinned)
                self.stats.misses += 1
                self.stats.evictions += int(v >= 0)
                out.append(Rec(KIND_ACCESS, t, self.layer, r, j, 0, s, v))
        for e in range(self.E):
            if self.prefetched[e]:
                self.prefetched[e] = False
                self.stats.pf_wasted += 1
        return out

    # -- speculative prefetch before the next lookup ---------------------------
    def prefetch(self, guesses: Sequence[int], max_n: int) -> List[Rec]:
        guesses = [int(e) for e in guesses]
        t = self.lookups
        pinned = set(guesses)
        out = []
        issued = 0
        for r, j in enumerate(guesses):
            self.stats.pf_guesses += 1
            if self.expert_slot[j] >= 0:
                out.append(Rec(KIND_PREFETCH, t, self.layer, r, j, F_RESIDENT,
                               self.expert_slot[j], -1))
            elif issued < max_n:
                self.clock += 1
                s, v = self._place(j, pinned)
                self.last[j] = self.clock
                self.prefetched[j] = True
                issued += 1
                self.stats.pf_issued += 1
                out.append(Rec(KIND_PREFETCH, t, self.layer, r, j, F_ISSUED, s, v))
            else:
                out.append(Rec(KIND_PREFETCH, t, self.layer, r, j, 0, -1, -1))
        return out

    # -- batched prefill of T tokens -------------------------------------------
    def prefill(self, ids_tk) -> List[Rec]:
        rows = [[int(e) for e in row] for row in ids_tk]
        T = len(rows)
        t0 = self.lookups
        self.lookups += T
        self.stats.lookups += T
        start = set(self.resident())
        n = [0] * self.E
        for row in rows:                      # token-major, rank order
            for j in row:
                self.clock += 1
                self.last[j] = self.clock
                n[j] += 1
        for e in range(self.E):
            self.count[e] += n[e]
        routed = sum(n)
        hits = sum(n[e] for e in start)
        self.stats.hits += hits
        self.stats.misses += routed - hits

        # a prefetched expert the batch routes to was used (even if the new
        # residency then drops it); one it does not route to was wasted
        for e in range(self.E):
            if self.prefetched[e]:
                self.prefetched[e] = False
                if n[e] > 0:
                    self.stats.pf_useful += 1
                else:
                    self.stats.pf_wasted += 1

        if self.policy == LFU:
            prio = lambda e: (-self.count[e], 0 if e in start else 1, e)
        elif self.policy == LFU_AGED:
            prio = lambda e: (-self.aged_count(e), 0 if e in start else 1, e)
        else:
            prio = lambda e: (-self.last[e], 0 if e in start else 1, e)
        rstar = set(sorted(range(self.E), key=prio)[:self.S])
        freed = sorted([s for s, e in enumerate(self.slot_expert) if e < 0]
                       + [self.expert_slot[e] for e in start if e not in rstar])
        newcomers = sorted(rstar - start)
        victim_of = {}
        for s, e in zip(freed, newcomers):
            v = self.slot_expert[s]
            if v >= 0:
                self.expert_slot[v] = -1
                if self.prefetched[v]:
                    self.prefetched[v] = False
                    self.stats.pf_wasted += 1
                self.stats.evictions += 1
            self.slot_expert[s] = e
            self.expert_slot[e] = s
            victim_of[e] = v
        out = []
        for e in range(self.E):
            fl = (F_RES_START if e in start else 0) | (F_RES_AFTER if e in rstar else 0)
            if (n[e] > 0 and e not in start) or e in victim_of:
                fl |= F_FETCHED
            out.append(Rec(KIND_PREFILL, t0, self.layer, n[e], e, fl,
                           self.expert_slot[e], victim_of.get(e, -1)))
        return out

    def state(self):
        """(slot_expert, expert_slot, count, last, clock) as plain lists."""
        return (list(self.slot_expert), list(self.expert_slot), list(self.count),
                list(self.last), self.clock)


def make_caches(layers: int, experts: int, slots: int, policy: str) -> List[LayerCache]:
    return [LayerCache(experts, slots, policy, layer=l) for l in range(layers)]
