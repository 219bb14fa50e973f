"""Hand-worked pins of the arena placement/LRU model and of the chunk grouping rule."""
import pytest

import synth
from oracle.arena_sim import ArenaSim, NoSpace
from oracle import chunks


def test_lru_evicts_least_recent_first_fit_lowest_address():
    a = ArenaSim(1000, align=100)
    for mid, nb in enumerate([300, 300, 300, 500]):
        a.register(mid, nb)
    assert a.request(0) == {"hit": False, "offset": 0, "evicted": []}
    assert a.request(1) == {"hit": False, "offset": 300, "evicted": []}
    assert a.request(2) == {"hit": False, "offset": 600, "evicted": []}
    assert a.request(0)["hit"]                       # order now 1 < 2 < 0
    r = a.request(3)                                  # 500 B: evict 1 (gap 300..600 too small), then 2
    assert r["evicted"] == [1, 2] and r["offset"] == 300
    # 100 B were free before the first eviction and 400 B before the second: neither sufficed alone
    assert a.frag_evictions == 0 and a.evictions == 2
    assert a.stats()["used"] == 800 and a.stats()["largest_free"] == 200
    assert (a.hits, a.misses, a.bytes_swapped) == (1, 4, 1400)


def test_fragmentation_eviction_counted():
    a = ArenaSim(1000, align=100)
    for mid, nb in enumerate([400, 200, 400, 300]):
        a.register(mid, nb)
    a.request(0); a.request(1); a.request(2)         # [0:400) [400:600) [600:1000)
    a.request(2); a.request(0)                       # LRU order 1 < 2 < 0
    a.evict(1)                                       # 200 free at 400..600 (explicit: not counted)
    a.register(4, 100)
    assert a.request(4)["offset"] == 400             # first fit lowest address
    r = a.request(3)                                 # 300 B: free 100 (at 500..600) -> evict 2 (LRU)
    assert r["evicted"] == [2] and r["offset"] == 500
    assert a.frag_evictions == 0 and a.evictions == 1


def test_frag_eviction_when_total_free_suffices():
    a = ArenaSim(900, align=100)
    for mid, nb in enumerate([300, 300, 300, 400]):
        a.register(mid, nb)
    a.request(0); a.request(1); a.request(2)
    a.evict(0); a.evict(2)                           # free 0..300 and 600..900: 600 free, no 400 gap
    r = a.request(3)
    assert r["evicted"] == [1] and r["offset"] == 0 and a.frag_evictions == 1


def test_too_large_is_refused_without_state_change():
    a = ArenaSim(1000)
    a.register(0, 2000)
    with pytest.raises(NoSpace):
        a.request(0)
    assert a.clock == 0 and a.misses == 0


def test_requester_is_never_its_own_victim_and_hits_do_not_move():
    a = ArenaSim(1000, align=1)
    a.register(0, 600); a.register(1, 600)
    assert a.request(0)["offset"] == 0
    r = a.request(1)
    assert r["evicted"] == [0] and r["offset"] == 0
    assert a.request(1) == {"hit": True, "offset": 0, "evicted": []}


def test_chunk_plan_hand_worked():
    # layers: 0 -> 100 B, 1 -> 50 B, 2 -> 300 B, 3 -> 10 B (offsets with padding gaps)
    t = [(0, 0, 60), (0, 64, 36), (1, 128, 50), (2, 256, 300), (3, 768, 10)]
    assert chunks.plan(t, 1024, 120) == [
        {"begin": 0, "end": 256, "first_layer": 0, "last_layer": 1},
        {"begin": 256, "end": 768, "first_layer": 2, "last_layer": 2},
        {"begin": 768, "end": 1024, "first_layer": 3, "last_layer": 3}]
    one = chunks.plan(t, 1024, 1 << 40)
    assert one == [{"begin": 0, "end": 1024, "first_layer": 0, "last_layer": 3}]
    per_layer = chunks.plan(t, 1024, 0)
    assert [c["first_layer"] for c in per_layer] == [0, 1, 2, 3]
    # tensor granularity: layer 0's two tensors become separate transfers at G = 0, and
    # at G = 120 the first group closes inside layer 1's predecessor boundary rules
    per_tensor = chunks.plan(t, 1024, 0, per_tensor=True)
    assert [(c["begin"], c["end"], c["first_layer"], c["last_layer"]) for c in per_tensor] == [
        (0, 64, 0, 0), (64, 128, 0, 0), (128, 256, 1, 1), (256, 768, 2, 2), (768, 1024, 3, 3)]
    # G = 90: 60 + 36 closes after layer 0's second tensor; 50 B of layer 1 alone stays
    # open until layer 2's 300 B join it
    assert [(c["begin"], c["end"], c["first_layer"], c["last_layer"]) for c in chunks.plan(t, 1024, 90, per_tensor=True)] == [
        (0, 128, 0, 0), (128, 768, 1, 2), (768, 1024, 3, 3)]
    # G = 50: the 60 B tensor closes a group by itself, so layer 0 spans two transfers
    assert [(c["begin"], c["end"], c["first_layer"], c["last_layer"]) for c in chunks.plan(t, 1024, 50, per_tensor=True)] == [
        (0, 64, 0, 0), (64, 256, 0, 1), (256, 768, 2, 2), (768, 1024, 3, 3)]


def test_chunk_plans_of_workloads():
    def plan(cfg, g):
        m = synth.config_model(cfg)
        return chunks.plan([(x.layer, x.offset, x.nbytes) for x in m.tensors], m.total_bytes, g)
    assert len(plan(1, 2 << 20)) == 1
    p2 = plan(2, 2 << 20)
    assert len(p2) == 24 and all(c["end"] - c["begin"] == 33_562_624 for c in p2)
    p4 = plan(4, 2 << 20)
    assert len(p4) == 13 and p4[0]["end"] == 47_674_368
    p3 = plan(3, 2 << 20)
    assert p3[-1]["first_layer"] <= 53 and sum(c["end"] - c["begin"] for c in p3) == synth.config_model(3).total_bytes
    # one transfer per tensor: 53 conv weights + 53 biases + FC weight and bias
    m3 = synth.config_model(3)
    pt = chunks.plan([(x.layer, x.offset, x.nbytes) for x in m3.tensors], m3.total_bytes, 0, per_tensor=True)
    assert len(pt) == len(m3.tensors) == 108
    assert [c["begin"] for c in pt[1:]] == [x.offset for x in m3.tensors[1:]]
