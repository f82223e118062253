"""A second, deliberately different formulation of the cache policies, used
only to pin the oracle's cache.

The oracle keeps per-expert clocks and counters and takes a keyed minimum.
This checker keeps a recency list (least recent first) and scans it: LRU
evicts the first unpinned entry, LFU the unpinned entry with the smallest
count, earliest in the list on equal counts.  Aged LFU ("lfu-aged:A") keeps
an idle counter per expert that every tick raises and a use clears, and
halves a copy of the count step by step, once per A idle ticks, before the
same smallest-count scan.  Record tuples use the same
layout as the oracle's: (kind, token, layer, rank, expert, flags, slot, victim).
"""


class ListCache:
    def __init__(self, E, S, policy, layer=0, initial=None):
        self.policy, _, period = policy.partition(":")
        self.period = int(period) if period else None
        self.E, self.S, self.layer = E, S, layer
        init = list(initial) if initial is not None else list(range(S))
        self.slot = {e: s for s, e in enumerate(init) if e >= 0}
        self.free = [s for s, e in enumerate(init) if e < 0]
        self.order = [e for _, e in sorted((s, e) for e, s in self.slot.items())]  # slot 0 oldest
        self.count = {e: 0 for e in range(E)}
        self.pf = set()
        self.t = 0
        # warm start: the expert in slot s was last used S - s ticks ago
        self.idle = {e: 0 for e in range(E)}
        for e, s in self.slot.items():
            self.idle[e] = S - s

    def _tick(self, used):
        for e in self.idle:
            self.idle[e] += 1
        self.idle[used] = 0

    def _weight(self, e):
        c = self.count[e]
        if self.policy == "lfu-aged":
            for _ in range(self.idle[e] // self.period):
                c //= 2
        return c

    def _evict_for(self, pinned):
        if self.free:
            s = min(self.free)
            self.free.remove(s)
            return s, -1
        cands = [e for e in self.order if e not in pinned]
        if self.policy == "lru":
            v = cands[0]
        else:
            low = min(self._weight(e) for e in cands)
            v = [e for e in cands if self._weight(e) == low][0]
        s = self.slot.pop(v)
        self.order.remove(v)
        self.pf.discard(v)
        return s, v

    def access(self, ids):
        out = []
        pinned = set(ids)
        t = self.t
        self.t += 1
        for r, j in enumerate(ids):
            self.count[j] += 1
            self._tick(j)
            if j in self.slot:
                useful = j in self.pf
                self.pf.discard(j)
                self.order.remove(j)
                self.order.append(j)
                out.append((0, t, self.layer, r, j, 1 | (2 if useful else 0), self.slot[j], -1))
            else:
                s, v = self._evict_for(pinned)
                self.slot[j] = s
                self.order.append(j)
                out.append((0, t, self.layer, r, j, 0, s, v))
        self.pf.clear()
        return out

    def prefetch(self, guesses, max_n):
        out = []
        pinned = set(guesses)
        n = 0
        for r, j in enumerate(guesses):
            if j in self.slot:
                out.append((1, self.t, self.layer, r, j, 1, self.slot[j], -1))
            elif n < max_n:
                self._tick(j)
                s, v = self._evict_for(pinned)
                self.slot[j] = s
                self.order.append(j)
                self.pf.add(j)
                n += 1
                out.append((1, self.t, self.layer, r, j, 2, s, v))
            else:
                out.append((1, self.t, self.layer, r, j, 0, -1, -1))
        return out
