"""Two-tier partitioned placement for the HBM weight arena (oracle).

Test infrastructure only. It follows the paper's appendix "Memory Block Allocation" (with
Sec. 4.4, "Memory block allocation"): device memory is divided into partitions; a partition
either holds blocks of one common size, shared by different models, or serves irregular
sizes with the buddy scheme (Knowlton's allocator, the paper's citation); the blocks of one
model are kept together, so evicting the model can free whole partitions.

Readings (the paper gives neither sizes nor tie rules):

* A model's weights form one block (one contiguous extent): a model's blocks are
  co-located by construction.
* Partitions: floor(C / P) partitions of P bytes, then, if at least `align` bytes remain,
  one short partition of the rest (C capacity, P the partition size, a multiple of the
  alignment).
* A model's size class is its size rounded up to the alignment. A class is common while at
  least two registered models have it; other classes are irregular.
* A model of size s is placed as follows.
  - s > P: a run of consecutive free partitions whose sizes add up to at least s; the run
    with the lowest first index; the model sits at the run's start.
  - common class, s <= P: a slot of a partition dedicated to the class. Slots sit at
    offsets k * s from the partition's start, k < floor(partition size / s). The
    dedicated partition with the most occupied slots that has a free slot is used (ties:
    lowest index), its lowest free slot; if none has one, the free partition with the
    highest index among those that hold at least one slot is dedicated to the class.
  - irregular class, s <= P: a buddy block. Block sizes of a partition of size S are
    S / 2^j, halving only while the half stays a multiple of the alignment; the model takes
    the smallest block size that holds it. Among buddy partitions that have a free block at
    least that large, the one with the most bytes in allocated blocks is used (ties:
    lowest index); in it, the smallest free block that is large enough (ties: lowest
    offset), split in halves down to the needed size, the lower half kept each time. If no
    buddy partition can serve, the free partition with the highest index that is large
    enough becomes a buddy partition. A freed block merges with its buddy while the buddy
    is free and of the same size.
  - Runs are taken from the low end and new dedicated or buddy partitions from the high
    end, so that small models do not split the runs large ones need.
* A partition whose last block or slot is freed becomes free again; its class or buddy
  tree is forgotten.
* Eviction: the victim order is the first-fit arena's (least recently used, or light
  before heavy under the heaviness policy), one victim at a time until a placement exists.
  An eviction counts as a fragmentation eviction when the free bytes (capacity minus the
  sizes of the resident models) already sufficed for the request.
* Consolidation (the appendix's consolidation of blocks across partitions; optional): when a
  request cannot be placed, before each eviction one partition is evacuated if possible:
  the slot or buddy partition with the fewest bytes in use (ties: lowest index) whose
  occupants can all be placed, in increasing offset order and by the rules above, in other
  partitions of the same kind (slots of the same class, buddy blocks) without dedicating a
  free partition. It becomes free, and placement is tried again; only when no partition
  can be evacuated is a victim evicted. The request reports its evictions and moves
  (model, old offset, new offset) interleaved in the order made; the device replays them
  in that order before the requester's weights land.
"""
from __future__ import annotations

import copy

from .arena_sim import ArenaSim, NoSpace, round_up


class _Part:
    """One partition: its byte range and what it currently holds."""

    def __init__(self, start: int, size: int):
        self.start = start
        self.size = size
        self.kind = "free"           # "free" | "slab" | "buddy" | "run"
        self.cls = None              # slab: the size class
        self.slots = {}              # slab: slot index -> model id
        self.free_blocks = set()     # buddy: free (offset, size), offsets from the start
        self.used_blocks = {}        # buddy: offset -> (size, model id)
        self.run_owner = None        # run: the model id

    def reset(self):
        self.__init__(self.start, self.size)

    def n_slots(self, cls: int) -> int:
        return self.size // cls

    def buddy_bytes(self) -> int:
        return sum(sz for sz, _ in self.used_blocks.values())


class PartitionArenaSim(ArenaSim):
    def __init__(self, capacity: int, partition: int, align: int = 256, policy: str = "lru",
                 consolidate: bool = False):
        super().__init__(capacity, align, policy)
        self.consolidate = consolidate
        self.evacuations = 0
        self.bytes_moved = 0
        assert partition > 0 and partition % align == 0
        self.partition = partition
        self.parts = []
        n_full = capacity // partition
        for i in range(n_full):
            self.parts.append(_Part(i * partition, partition))
        rest = capacity - n_full * partition
        if rest >= align:
            self.parts.append(_Part(n_full * partition, rest))
        self.placed = {}             # resident model id -> ("slab", part, slot) | ("buddy", part, off) | ("run", first, last)

    # ---- classes
    def common(self, mid: int) -> bool:
        s = self.size[mid]
        return sum(1 for m in self.size if self.size[m] == s) >= 2

    # ---- buddy helpers
    def block_size(self, part_size: int, need: int):
        """Smallest reachable block size of a partition of part_size bytes that holds need."""
        b = part_size
        if b < need:
            return None
        while b % (2 * self.align) == 0 and b // 2 >= need:
            b //= 2
        return b

    # ---- placement
    def _free_parts_high_first(self, need: int):
        return [i for i in range(len(self.parts) - 1, -1, -1)
                if self.parts[i].kind == "free" and self.parts[i].size >= need]

    def try_place(self, mid: int, avoid=None):
        """Places mid (no eviction); None if impossible. avoid: a partition index that must
        not be used; then no free partition is dedicated either (evacuation)."""
        s = self.size[mid]
        if s > self.partition:
            for i in range(len(self.parts)):
                total, j = 0, i
                while j < len(self.parts) and self.parts[j].kind == "free" and total < s:
                    total += self.parts[j].size
                    j += 1
                if total >= s:
                    for k in range(i, j):
                        self.parts[k].kind = "run"
                        self.parts[k].run_owner = mid
                    self.placed[mid] = ("run", i, j - 1)
                    return self.parts[i].start
            return None
        if self.common(mid):
            best = None
            for i, p in enumerate(self.parts):
                if i == avoid:
                    continue
                if p.kind == "slab" and p.cls == s and len(p.slots) < p.n_slots(s):
                    if best is None or len(p.slots) > len(self.parts[best].slots):
                        best = i
            if best is None:
                cand = [] if avoid is not None else self._free_parts_high_first(s)
                if not cand:
                    return None
                best = cand[0]
                self.parts[best].kind = "slab"
                self.parts[best].cls = s
            p = self.parts[best]
            k = min(set(range(p.n_slots(s))) - set(p.slots))
            p.slots[k] = mid
            self.placed[mid] = ("slab", best, k)
            return p.start + k * s
        # irregular: buddy
        best, best_used = None, -1
        for i, p in enumerate(self.parts):
            if p.kind != "buddy" or i == avoid:
                continue
            t = self.block_size(p.size, s)
            if t is None or not any(sz >= t for _, sz in p.free_blocks):
                continue
            u = p.buddy_bytes()
            if u > best_used:
                best, best_used = i, u
        if best is None:
            cand = [] if avoid is not None else self._free_parts_high_first(s)
            if not cand:
                return None
            best = cand[0]
            p = self.parts[best]
            p.kind = "buddy"
            p.free_blocks = {(0, p.size)}
        p = self.parts[best]
        t = self.block_size(p.size, s)
        off, sz = min((b for b in p.free_blocks if b[1] >= t), key=lambda b: (b[1], b[0]))
        p.free_blocks.remove((off, sz))
        while sz > t:
            sz //= 2
            p.free_blocks.add((off + sz, sz))
        p.used_blocks[off] = (sz, mid)
        self.placed[mid] = ("buddy", best, off)
        return p.start + off

    def release(self, mid: int):
        where = self.placed.pop(mid)
        if where[0] == "run":
            for k in range(where[1], where[2] + 1):
                self.parts[k].reset()
            return
        p = self.parts[where[1]]
        if where[0] == "slab":
            del p.slots[where[2]]
            if not p.slots:
                p.reset()
            return
        off = where[2]
        sz, _ = p.used_blocks.pop(off)
        while sz < p.size:
            buddy = off + sz if (off // sz) % 2 == 0 else off - sz
            if (buddy, sz) not in p.free_blocks:
                break
            p.free_blocks.remove((buddy, sz))
            off = min(off, buddy)
            sz *= 2
        p.free_blocks.add((off, sz))
        if not p.used_blocks:
            p.reset()

    # ---- consolidation
    def occupants(self, i: int):
        """(offset, model) of partition i's occupants in increasing offset order."""
        p = self.parts[i]
        if p.kind == "slab":
            return sorted((p.start + k * p.cls, m) for k, m in p.slots.items())
        return sorted((p.start + o, m) for o, (_, m) in p.used_blocks.items())

    def in_use(self, i: int) -> int:
        p = self.parts[i]
        return len(p.slots) * p.cls if p.kind == "slab" else p.buddy_bytes()

    def evacuate(self):
        """Frees one slot or buddy partition by moving its occupants; the moves, or None."""
        order = sorted((self.in_use(i), i) for i, p in enumerate(self.parts) if p.kind in ("slab", "buddy"))
        for _, i in order:
            saved = (copy.deepcopy(self.parts), dict(self.placed))
            moves = []
            for old, m in self.occupants(i):
                self.release(m)
                new = self.try_place(m, avoid=i)
                if new is None:
                    break
                moves.append((m, old, new))
            else:
                for m, _, new in moves:
                    self.where[m] = new
                    self.bytes_moved += self.size[m]
                self.evacuations += 1
                return moves
            self.parts, self.placed = saved
        return None

    # ---- the request path (same counters and victim order as the first-fit arena)
    def request(self, mid: int) -> dict:
        need = self.size[mid]
        if need > self.capacity:
            raise NoSpace(mid)
        self.clock += 1
        self.last[mid] = self.clock
        if mid in self.where:
            self.hits += 1
            out = {"hit": True, "offset": self.where[mid], "evicted": []}
            if self.consolidate:
                out["steps"] = []
            return out
        self.misses += 1
        evicted, steps = [], []
        off = self.try_place(mid)
        while off is None:
            if self.consolidate:
                mv = self.evacuate()
                if mv is not None:
                    steps += [("move",) + m for m in mv]
                    off = self.try_place(mid)
                    continue
            victim = self.victim()
            if self.capacity - self.used() >= need:
                self.frag_evictions += 1
            self.evict(victim)
            self.evictions += 1
            evicted.append(victim)
            steps.append(("evict", victim))
            off = self.try_place(mid)
        self.where[mid] = off
        self.bytes_swapped += need
        out = {"hit": False, "offset": off, "evicted": evicted}
        if self.consolidate:
            out["steps"] = steps
        return out

    def evict(self, mid: int) -> None:
        if mid in self.where:
            del self.where[mid]
            self.release(mid)

    def unregister(self, mid: int) -> None:
        self.evict(mid)
        del self.size[mid], self.last[mid], self.heavy[mid]

    def free_partitions(self) -> int:
        return sum(1 for p in self.parts if p.kind == "free")

    def stats(self) -> dict:
        d = super().stats()
        d["partitions"] = len(self.parts)
        d["partitions_free"] = self.free_partitions()
        if self.consolidate:
            d["evacuations"] = self.evacuations
            d["bytes_moved"] = self.bytes_moved
        return d


__all__ = ["PartitionArenaSim", "round_up"]
