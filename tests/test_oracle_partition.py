"""Pins of the oracle's two-tier partitioned placement (oracle/partition_sim.py).

Each pin checks the oracle against something other than itself: the first-fit simulator it
must reduce to when partitions are one alignment unit, a textbook LRU cache it must equal
when all models share one size, worked examples of the buddy scheme (Knowlton's
allocator, cited by the paper's appendix "Memory Block Allocation") and of slots and runs
derived by hand, and structural invariants over random traces.
"""
from collections import OrderedDict

import pytest
from hypothesis import given, settings, strategies as st

from oracle.arena_sim import ArenaSim
from oracle.partition_sim import PartitionArenaSim

A = 256


@settings(max_examples=80, deadline=None)
@given(sizes=st.lists(st.integers(2, 40), min_size=2, max_size=9),
       ops=st.lists(st.tuples(st.sampled_from(["req", "req", "req", "evict"]), st.integers(0, 8)), max_size=70),
       units=st.integers(8, 120), policy=st.sampled_from(["lru", "heaviness"]), bits=st.integers(0, 511))
def test_unit_partitions_reduce_to_first_fit(sizes, ops, units, policy, bits):
    """Partitions of one alignment unit and models larger than one unit: every model is a
    run of free units taken from the lowest address that fits, which is first fit."""
    sizes = [s * A - A // 3 for s in sizes]          # rounds up to s units, each > 1 unit
    cap = units * A
    ff = ArenaSim(cap, A, policy)
    pa = PartitionArenaSim(cap, A, A, policy)
    for i, nb in enumerate(sizes):
        h = bool(bits >> i & 1)
        ff.register(i, nb, h)
        pa.register(i, nb, h)
    for op, k in ops:
        k %= len(sizes)
        if op == "evict":
            ff.evict(k)
            pa.evict(k)
            continue
        if ff.size[k] > cap:
            continue
        assert pa.request(k) == ff.request(k)
    s_pa = pa.stats()
    assert {k: s_pa[k] for k in ff.stats()} == ff.stats()


@settings(max_examples=80, deadline=None)
@given(n_models=st.integers(2, 30), per_part=st.integers(1, 5), n_parts=st.integers(1, 4),
       slack=st.integers(0, 3), seq=st.lists(st.integers(0, 29), min_size=1, max_size=120))
def test_single_size_is_an_lru_cache(n_models, per_part, n_parts, slack, seq):
    """All models of one size s <= P: slots of dedicated partitions, n_parts * floor(P / s)
    of them; every eviction frees a slot the next model can use, so hits, misses and
    victims are those of an LRU cache with that many entries."""
    s = 3 * A
    part = per_part * s + slack * A
    slots = n_parts * (part // s)
    pa = PartitionArenaSim(n_parts * part, part, A)
    for i in range(n_models):
        pa.register(i, s)
    cache = OrderedDict()
    hits = 0
    for k in seq:
        k %= n_models
        r = pa.request(k)
        if k in cache:
            cache.move_to_end(k)
            hits += 1
            assert r["hit"] and r["evicted"] == []
            continue
        want = []
        if len(cache) == slots:
            want.append(cache.popitem(last=False)[0])
        cache[k] = True
        assert not r["hit"] and r["evicted"] == want
    assert pa.hits == hits and pa.evictions == max(0, pa.misses - slots)
    assert sorted(pa.where) == sorted(cache)


def test_buddy_worked_example():
    """One buddy partition of 16 units (4096 bytes), irregular sizes only. Block sizes
    4096, 2048, 1024, 512, 256; every step derived by hand from the buddy rules: the
    smallest free block that holds the request (lowest offset on ties), halved with the
    lower half kept; a freed block merges with its free buddy of equal size."""
    pa = PartitionArenaSim(4096, 4096, A)
    # distinct rounded sizes, so every class is irregular (F, of A's rounded size 768, is
    # registered only once A is gone)
    names = {"A": 700, "B": 1800, "C": 300, "D": 200, "E": 900, "G": 4000, "F": 600}
    ids = {nm: i for i, nm in enumerate(names)}
    for nm, nb in names.items():
        if nm != "F":
            pa.register(ids[nm], nb)

    def req(nm):
        r = pa.request(ids[nm])
        assert r["evicted"] == []
        return r["offset"]

    def free_blocks():
        return sorted(pa.parts[0].free_blocks)

    assert req("A") == 0                   # 768 -> block 1024: 4096 split to 2048+2048, 2048 to 1024+1024
    assert free_blocks() == [(1024, 1024), (2048, 2048)]
    assert req("B") == 2048                # 2048 -> the free 2048 block
    assert req("C") == 1024                # 512: the free 1024 split, lower half
    assert free_blocks() == [(1536, 512)]
    assert req("D") == 1536                # 256: the free 512 split
    assert free_blocks() == [(1792, 256)]
    pa.unregister(ids["A"])                # its buddy (1024 at 1024) is split: no merge
    pa.register(ids["F"], names["F"])
    assert free_blocks() == [(0, 1024), (1792, 256)]
    assert req("E") == 0                   # 1024 fits the freed block exactly
    pa.evict(ids["C"])                     # buddy 512 at 1536 is split: no merge
    assert free_blocks() == [(1024, 512), (1792, 256)]
    pa.evict(ids["D"])                     # 256 at 1536 + 1792 -> 512 at 1536; + 1024 -> 1024 at 1024
    assert free_blocks() == [(1024, 1024)]
    assert req("F") == 1024                # 768 -> block 1024
    for nm in ("E", "F", "B"):
        pa.evict(ids[nm])
    assert pa.parts[0].kind == "free"      # all merged: the partition is free again
    assert req("G") == 0 and pa.parts[0].kind == "buddy"
    assert pa.evictions == 0 and pa.frag_evictions == 0


def test_slots_buddy_and_runs_worked_example():
    """Three partitions of 2048 bytes and a short one of 512: a common class (two models of
    768 bytes), an irregular model and runs; every offset derived by hand."""
    pa = PartitionArenaSim(3 * 2048 + 512, 2048, A)
    assert [(p.start, p.size) for p in pa.parts] == [(0, 2048), (2048, 2048), (4096, 2048), (6144, 512)]
    pa.register(0, 700)       # class 768, common (models 0, 1 and later 2)
    pa.register(1, 768)
    pa.register(3, 300)       # 512, irregular
    pa.register(4, 3000)      # 3072 > 2048: a run of two partitions
    # a slot class: the short partition cannot hold a slot, so the highest free full one (2)
    assert pa.request(0)["offset"] == 4096
    assert pa.request(1)["offset"] == 4096 + 768          # same partition, next slot (2 per partition)
    assert pa.request(3)["offset"] == 6144                 # buddy: highest free partition that holds 512
    assert pa.request(4)["offset"] == 0                    # run: partitions 0 and 1, from the low end
    assert pa.free_partitions() == 0
    pa.register(2, 768)
    # class 768 needs a slot: partition 2 is full, nothing is free; LRU victims in order
    # 0 (frees slot 0 of partition 2, enough). The free bytes before it, 6656 - 5120 = 1536,
    # are slack inside partitions but would hold 768: a fragmentation eviction
    r = pa.request(2)
    assert r == {"hit": False, "offset": 4096, "evicted": [0]}
    assert pa.frag_evictions == 1
    # model 0 again: LRU order 1, 3, 4, 2. Evicting 1 frees slot 1 of partition 2
    r = pa.request(0)
    assert r == {"hit": False, "offset": 4096 + 768, "evicted": [1]}
    assert pa.frag_evictions == 2
    # model 1 again: LRU order 3, 4, 2, 0; evicting 3 (the short buddy partition) frees
    # 512 bytes, too small for a slot; evicting 4 frees partitions 0 and 1 -> a fresh slot
    # partition, the highest free one that holds 768: partition 1
    r = pa.request(1)
    assert r == {"hit": False, "offset": 2048, "evicted": [3, 4]}
    # free bytes before evicting 3: 1536, before evicting 4: 6656 - 2*768 - 3072 = 2048;
    # both suffice for 768: two more fragmentation evictions
    assert pa.frag_evictions == 4


def _consolidation_setup(consolidate):
    # three partitions of 2048 bytes; four models of 768 bytes (a common class, two slots per
    # partition) and one of 3072 (a run of two partitions)
    pa = PartitionArenaSim(3 * 2048, 2048, A, consolidate=consolidate)
    for i in range(4):
        pa.register(i, 768)
    pa.register(9, 3072)
    assert [pa.request(i)["offset"] for i in range(4)] == [4096, 4096 + 768, 2048, 2048 + 768]
    pa.evict(0)
    pa.evict(2)       # partition 1 holds model 3 (slot 1), partition 2 model 1 (slot 1)
    return pa


def test_consolidation_worked_example():
    """Derived by hand. The run needs partitions 0 and 1; partition 1's only model fits in
    partition 2's free slot, so partition 1 is evacuated (fewest bytes in use, lowest index
    first) instead of evicting anything."""
    pa = _consolidation_setup(True)
    r = pa.request(9)
    assert r == {"hit": False, "offset": 0, "evicted": [], "steps": [("move", 3, 2048 + 768, 4096)]}
    assert pa.where[3] == 4096 and pa.evacuations == 1 and pa.bytes_moved == 768
    assert pa.evictions == 0 and pa.frag_evictions == 0
    # now partition 2 is full (models 3, 1) and nothing is free: evacuating it fails (no
    # other partition of the class), the state is restored, and the LRU model (1) goes
    r = pa.request(0)
    assert r == {"hit": False, "offset": 4096 + 768, "evicted": [1], "steps": [("evict", 1)]}
    assert pa.where[3] == 4096 and pa.parts[2].kind == "slab" and pa.parts[2].slots == {0: 3, 1: 0}
    assert pa.frag_evictions == 1             # 6144 - (768 + 768 + 3072) = 1536 free before
    # the same start without consolidation: LRU evicts model 1 (partition 2 frees, but 0 and
    # 2 are not adjacent), then model 3; both evictions had enough free bytes
    pb = _consolidation_setup(False)
    r = pb.request(9)
    assert r == {"hit": False, "offset": 0, "evicted": [1, 3]} and pb.frag_evictions == 2


def test_consolidation_move_into_a_victims_slot():
    """Derived by hand: the order of evictions and moves matters to the device (a move may
    fill the slot a victim just left, whose readers must finish first), so the request
    reports them interleaved. Three partitions of 2048, 768-byte models (two slots per
    partition): partition 2 holds models 0 and 1, partition 1 model 2, partition 0 is free.
    A 3072-byte model needs a run of two free partitions. Partition 1 cannot be evacuated
    (partition 2 is full) nor partition 2 (one free slot for two models), so LRU evicts
    model 0; now partition 1's model moves into the slot model 0 left, partition 1 is free,
    and the run takes partitions 0 and 1."""
    pa = PartitionArenaSim(3 * 2048, 2048, A, consolidate=True)
    for i in range(3):
        pa.register(i, 768)
    pa.register(9, 3072)
    assert [pa.request(i)["offset"] for i in range(3)] == [4096, 4096 + 768, 2048]
    r = pa.request(9)
    assert r == {"hit": False, "offset": 0, "evicted": [0], "steps": [("evict", 0), ("move", 2, 2048, 4096)]}
    assert pa.where == {1: 4096 + 768, 2: 4096, 9: 0}


@settings(max_examples=60, deadline=None)
@given(sizes=st.lists(st.integers(1, 60).map(lambda x: x * 97), min_size=2, max_size=10),
       dup=st.lists(st.integers(0, 9), max_size=6),
       ops=st.lists(st.tuples(st.sampled_from(["req", "req", "req", "evict"]), st.integers(0, 15)), max_size=90),
       part_units=st.integers(1, 24), n_parts=st.integers(1, 5), tail=st.integers(0, 3))
def test_partition_invariants(sizes, dup, ops, part_units, n_parts, tail):
    """Resident extents never overlap and stay in the arena; a model no larger than a
    partition lies inside one partition (a buddy block also on a multiple of its block size
    there); a larger one starts on a partition boundary; emptying the arena frees every
    partition."""
    sizes = sizes + [sizes[d % len(sizes)] for d in dup]
    part = part_units * A
    cap = n_parts * part + tail * A
    pa = PartitionArenaSim(cap, part, A)
    for i, nb in enumerate(sizes):
        pa.register(i, nb)
    for op, k in ops:
        k %= len(sizes)
        if op == "evict":
            pa.evict(k)
        elif pa.size[k] <= cap:
            pa.request(k)
        ext = sorted((o, o + pa.size[m]) for m, o in pa.where.items())
        for (a0, a1), (b0, _) in zip(ext, ext[1:]):
            assert a1 <= b0
        assert all(0 <= a0 and a1 <= cap for a0, a1 in ext)
        starts = [p.start for p in pa.parts]
        for m, o in pa.where.items():
            kind = pa.placed[m][0]
            if pa.size[m] > part:
                assert kind == "run" and o in starts
                continue
            p = pa.parts[pa.placed[m][1]]
            assert p.start <= o and o + pa.size[m] <= p.start + p.size
            if kind == "buddy":
                sz = p.used_blocks[o - p.start][0]
                assert (o - p.start) % sz == 0 and sz >= pa.size[m]
                assert sz % (2 * A) != 0 or sz // 2 < pa.size[m]      # the smallest block that holds it
    for m in list(pa.where):
        pa.evict(m)
    assert pa.free_partitions() == len(pa.parts)


def test_short_tail_and_oversize():
    pa = PartitionArenaSim(2 * 1024 + 100, 1024, A)        # tail of 100 bytes < one unit: dropped
    assert len(pa.parts) == 2
    pa.register(0, 2048)
    assert pa.request(0)["offset"] == 0                    # a run of both partitions
    pa.register(1, 4096)
    from oracle.arena_sim import NoSpace
    with pytest.raises(NoSpace):
        pa.request(1)
