"""Reference model of the HBM weight arena: placement and LRU eviction (oracle).

Test infrastructure only. Rules it follows:

* All device memory for models is reserved once and managed internally, so no native
  allocation happens per swap (paper Sec. 4.4, "Memory block allocation").
* Eviction only invalidates a model's device region; the host copy is always kept and
  nothing is copied back (Sec. 4.3, "Model eviction").
* Victims are chosen least-recently-used (Sec. 5.4; the paper's LRU baseline in Sec. 7.3).

* Heaviness-aware variant (Sec. 5.4, "Model eviction policy"): models are heavy or light
  by how much swapping them slows their inference; light models are evicted first, and
  only when no light model is resident does LRU pick among the heavy ones.

Readings where the paper is silent: a logical clock ticks once per request, so there are
no ties; a model is placed in the lowest-addressed free gap that fits (first fit); while
no gap fits, one victim at a time is invalidated: the least recently used resident model
(policy "lru"), or the least recently used resident light model if there is one, else the
least recently used heavy model (policy "heaviness"; a model's class is given, and may be
changed between requests). An eviction is counted as a fragmentation eviction when the
total free space already sufficed before it. A model larger than the whole arena is refused
with no state change.

* Contiguous-window variant (policy "lru_window", beyond the paper): when no gap fits, the
  victims are chosen together as the set of extents one contiguous range of the needed size
  overlaps, taking the range whose most recently used victim is the oldest (then fewer victim
  bytes, then the lower address), instead of invalidating the globally least recently used
  model one at a time, which frees space scattered over the arena.
"""
from __future__ import annotations


def round_up(n: int, a: int) -> int:
    return (n + a - 1) // a * a


class NoSpace(Exception):
    pass


class ArenaSim:
    def __init__(self, capacity: int, align: int = 256, policy: str = "lru"):
        assert policy in ("lru", "heaviness", "lru_window")
        self.capacity = capacity
        self.align = align
        self.policy = policy
        self.heavy = {}         # model id -> True if heavy (heaviness policy)
        self.size = {}          # model id -> extent bytes
        self.where = {}         # resident model id -> offset
        self.last = {}          # model id -> clock of last request
        self.clock = 0
        self.hits = self.misses = self.evictions = self.frag_evictions = 0
        self.bytes_swapped = 0

    def register(self, mid: int, nbytes: int, heavy: bool = False) -> None:
        self.size[mid] = round_up(nbytes, self.align)
        self.last[mid] = 0
        self.heavy[mid] = heavy

    def set_heavy(self, mid: int, heavy: bool) -> None:
        self.heavy[mid] = heavy

    def unregister(self, mid: int) -> None:
        self.where.pop(mid, None)
        del self.size[mid], self.last[mid], self.heavy[mid]

    def victim(self) -> int:
        candidates = list(self.where)
        if self.policy == "heaviness":
            light = [m for m in candidates if not self.heavy[m]]
            candidates = light or candidates
        return min(candidates, key=lambda m: self.last[m])

    def used(self) -> int:
        return sum(self.size[m] for m in self.where)

    def window_victims(self, need: int) -> list:
        """Policy "lru_window": the resident models to invalidate so that one contiguous range of
        `need` bytes becomes free. Every range starting at address 0 or where a resident extent
        ends is a candidate; its victims are the extents it overlaps. The candidate whose most
        recently used victim is the oldest wins, then the one with fewer victim bytes, then the
        lower address. Victims are returned least recently used first."""
        ext = sorted((o, m) for m, o in self.where.items())
        best = None
        for start in [0] + [o + self.size[m] for o, m in ext]:
            if start + need > self.capacity:
                continue
            hit = [m for o, m in ext if o < start + need and o + self.size[m] > start]
            key = (max(self.last[m] for m in hit), sum(self.size[m] for m in hit), start)
            if best is None or key < best[0]:
                best = (key, hit)
        return sorted(best[1], key=lambda m: self.last[m])

    def gaps(self):
        """Free gaps (offset, length) in address order."""
        out, cur = [], 0
        for off, m in sorted((o, m) for m, o in self.where.items()):
            if off > cur:
                out.append((cur, off - cur))
            cur = off + self.size[m]
        if cur < self.capacity:
            out.append((cur, self.capacity - cur))
        return out

    def first_fit(self, need: int):
        for off, ln in self.gaps():
            if ln >= need:
                return off
        return None

    def request(self, mid: int) -> dict:
        need = self.size[mid]
        if need > self.capacity:
            raise NoSpace(mid)
        self.clock += 1
        self.last[mid] = self.clock
        if mid in self.where:
            self.hits += 1
            return {"hit": True, "offset": self.where[mid], "evicted": []}
        self.misses += 1
        evicted = []
        off = self.first_fit(need)
        if off is None and self.policy == "lru_window":
            for victim in self.window_victims(need):
                if self.capacity - self.used() >= need:
                    self.frag_evictions += 1
                del self.where[victim]
                self.evictions += 1
                evicted.append(victim)
            off = self.first_fit(need)
        while off is None:
            victim = self.victim()
            if self.capacity - self.used() >= need:
                self.frag_evictions += 1
            del self.where[victim]
            self.evictions += 1
            evicted.append(victim)
            off = self.first_fit(need)
        self.where[mid] = off
        self.bytes_swapped += self.size[mid]
        return {"hit": False, "offset": off, "evicted": evicted}

    def evict(self, mid: int) -> None:
        self.where.pop(mid, None)

    def largest_free(self) -> int:
        return max((ln for _, ln in self.gaps()), default=0)

    def stats(self) -> dict:
        return {"capacity": self.capacity, "used": self.used(), "largest_free": self.largest_free(),
                "resident": len(self.where), "hits": self.hits, "misses": self.misses,
                "evictions": self.evictions, "frag_evictions": self.frag_evictions,
                "bytes_swapped": self.bytes_swapped}
