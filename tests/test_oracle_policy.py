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


# ------------------------------------------------------------------ pipelined request model

from oracle import pipeline


def test_pipeline_simulation_closed_forms():
    begin, total = [0, 100, 300, 600], 1000          # units of 100, 200, 300, 400 B
    us = [5.0, 7.0, 11.0, 13.0]
    r, o, h = 10.0, 3.0, 2.0                         # 10 B/us, 3 us per copy, 2 us hand-off
    # one group: everything lands at o + 1000 / r, then all layers run
    assert pipeline.simulate(begin, total, us, [0], r, o, h) == pytest.approx(3 + 100 + 2 + 36)
    # no compute: k groups cost k fixed costs plus the bytes, then the hand-off
    z = [0.0] * 4
    assert pipeline.simulate(begin, total, z, [0, 1, 2, 3], r, o, h) == pytest.approx(4 * 3 + 100 + 2)
    assert pipeline.simulate(begin, total, z, [0, 2], r, o, h) == pytest.approx(2 * 3 + 100 + 2)
    # hand-worked: groups {0,1} (300 B) and {2,3} (700 B)
    # group 0 lands at 3 + 30 = 33, layers 0-1 run 35 .. 47; group 1 lands at 33 + 3 + 70 = 106,
    # layers 2-3 run 108 .. 132
    assert pipeline.simulate(begin, total, us, [0, 2], r, o, h) == pytest.approx(132.0)
    # compute-bound: with a fast link the time is the first hand-off plus all layers, plus
    # the idle gap of any group that lands after its predecessor's layers finish
    fast = pipeline.simulate(begin, total, [100.0] * 4, [0, 1, 2, 3], 1e9, 1.0, 0.5)
    assert fast == pytest.approx(1.0 + 0.5 + 400.0)


def test_best_grouping_hand_worked():
    # two heavy-compute layers up front and a big last layer: the first layer goes alone so
    # it computes while the rest streams, the rest stay together (one fixed cost)
    begin, total = [0, 10, 20], 1010
    us = [50.0, 50.0, 1.0]
    first, t = pipeline.best_grouping(begin, total, us, 10.0, 5.0, 0.0)
    # [0],[1,2]: lands 6 and 6+5+100=111 -> layers run 6..56, 111..162 ; [0],[1],[2]: layer 2's
    # group lands at 6+6+5+99 = 116 -> 117 ; [0,1],[2]: 7..107, lands 7+5+99=111 -> 112
    assert first == [0, 1, 2] or first == [0, 2]
    assert t == pytest.approx(min(pipeline.simulate(begin, total, us, f, 10.0, 5.0, 0.0)
                                  for f in ([0], [0, 1], [0, 2], [0, 1, 2])))
    # with a huge fixed cost per copy a single group wins
    first, _ = pipeline.best_grouping(begin, total, us, 10.0, 1e6, 0.0)
    assert first == [0]


# ------------------------------------------------------------------ heaviness-aware eviction

def test_window_policy_hand_worked():
    # capacity 100: a, b, c of 30 at 0, 30, 60, recency b < c < a, then d (40) with 10 free at 90.
    # LRU one at a time: b, then c (free [30, 100)), d at 30. The window policy's candidate
    # ranges start at 0 (overlaps a: newest victim a), 30 (b and c: newest c, 60 bytes), 60
    # (c: newest c, 30 bytes), 90 (does not fit): c alone, d at 60.
    for policy, want_off, want_ev in (("lru", 30, ["b", "c"]), ("lru_window", 60, ["c"])):
        a = ArenaSim(100, align=1, policy=policy)
        for m, nb in (("a", 30), ("b", 30), ("c", 30), ("d", 40)):
            a.register(m, nb)
        for m in ("a", "b", "c", "a"):
            a.request(m)
        assert a.request("d") == {"hit": False, "offset": want_off, "evicted": want_ev}
        assert a.stats()["evictions"] == len(want_ev)
    # ties on the newest victim go to fewer victim bytes, then to the lower address
    a = ArenaSim(90, align=1, policy="lru_window")
    for m, nb in (("p", 20), ("q", 20), ("r", 20), ("s", 30), ("t", 40)):
        a.register(m, nb)
    for m in ("p", "q", "r", "s"):
        a.request(m)                      # p 0, q 20, r 40, s 60; full
    # t (40): ranges 0 (p, q: newest q), 20 (q, r: newest r), 40 (r, s: newest s), 60 (s,
    # then past the end: does not fit) -> newest q is the oldest -> p and q
    assert a.request("t") == {"hit": False, "offset": 0, "evicted": ["p", "q"]}


def test_heaviness_policy_evicts_light_first_then_lru_among_heavy():
    a = ArenaSim(1000, align=100, policy="heaviness")
    a.register(0, 300, heavy=True)
    a.register(1, 300, heavy=False)
    a.register(2, 300, heavy=True)
    a.register(3, 300, heavy=True)
    for m in (0, 1, 2):
        a.request(m)                                  # [0:300) [300:600) [600:900)
    a.request(0)                                      # LRU order: 1 < 2 < 0
    # LRU would evict 1 too (it is also the least recent): make the light model the most recent
    a.request(1)                                      # LRU order: 2 < 0 < 1
    r = a.request(3)                                  # needs 300 B, 100 free
    assert r["evicted"] == [1] and r["offset"] == 300  # the light model goes although most recent
    a.register(4, 400, heavy=True)
    r = a.request(4)                                  # only heavy models left: LRU among them
    # order: 2 (clock 3) < 0 (4) < 3 (6); evicting 2 leaves the 400 B gap 600..1000
    assert r["evicted"] == [2] and r["offset"] == 600
    a.register(5, 700, heavy=True)
    r = a.request(5)                                  # 0 (clock 4), then 3 (6): gaps 0..300, then 0..600
    assert r["evicted"] == [0, 3, 4] and r["offset"] == 0


def test_heaviness_policy_with_all_models_of_one_class_is_lru():
    for heavy in (False, True):
        lru, hv = ArenaSim(900, align=1), ArenaSim(900, align=1, policy="heaviness")
        for m in range(5):
            lru.register(m, 300)
            hv.register(m, 300, heavy=heavy)
        for m in (0, 1, 2, 0, 3, 4, 1, 2, 0, 4, 3):
            assert lru.request(m) == hv.request(m)


def test_heaviness_class_change_applies_to_later_evictions():
    a = ArenaSim(600, align=1, policy="heaviness")
    for m in range(3):
        a.register(m, 300, heavy=True)
    a.request(0); a.request(1)
    a.set_heavy(1, False)
    assert a.request(2)["evicted"] == [1]             # LRU would have taken model 0


# ------------------------------------------------------------------ SLO-aware queueing

from oracle import slo_queue


def test_rrc_solves_its_defining_equation():
    # (m + RRC) / (n + RRC) = p, multiplied out: m + RRC = p (n + RRC)
    for n, m, p in [(0, 0, 0.98), (10, 10, 0.98), (10, 7, 0.9), (50, 49, 0.98), (100, 60, 0.5), (3, 0, 0.99)]:
        r = slo_queue.rrc(n, m, p)
        assert m + r == pytest.approx(p * (n + r), abs=1e-9)
    # a function already above its percentile needs nothing more: RRC <= 0
    assert slo_queue.rrc(100, 99, 0.98) < 0 and slo_queue.rrc(100, 98, 0.98) == pytest.approx(0)
    assert slo_queue.rrc(100, 90, 0.98) == pytest.approx((98 - 90) / 0.02)


def test_high_group_threshold():
    rr = [5.0, -2.0, 1.0, 3.0, 0.0]          # sorted: f1 (-2), f4 (0), f2 (1), f3 (3), f0 (5); total 9
    assert slo_queue.high_group(rr, 0.0) == [False, True, False, False, True]   # only non-positive
    assert slo_queue.high_group(rr, 1 / 9) == [False, True, True, False, True]  # prefix 1 <= 1
    assert slo_queue.high_group(rr, 4 / 9) == [False, True, True, True, True]   # prefix 4 <= 4
    assert slo_queue.high_group(rr, 0.4) == [False, True, True, False, True]    # 4 > 3.6
    assert slo_queue.high_group(rr, 1.0) == [True] * 5
    assert slo_queue.high_group([-1.0, -3.0], 0.0) == [True, True]             # no positive RRC


def test_pick_order_within_and_across_groups():
    rr = [5.0, -2.0, 1.0, 3.0, 0.0]
    high = slo_queue.high_group(rr, 4 / 9)    # f1, f2, f3, f4 high; f0 low
    # high group first, largest RRC first: f3; its earliest queued request
    assert slo_queue.pick(rr, high, [0, 1, 3, 2, 3]) == 2
    assert slo_queue.pick(rr, high, [0, 4, 1]) == 1          # f4 (0) before f1 (-2)
    assert slo_queue.pick(rr, high, [0, 0]) == 0             # only the low group: f0
    low = [False] * 5                                        # all low: smallest RRC first
    assert slo_queue.pick(rr, low, [0, 3, 1, 2]) == 2
    assert slo_queue.pick([1.0, 1.0], [True, True], [1, 0]) == 1   # tie: lower index
    assert slo_queue.pick(rr, high, []) == -1


def test_alpha_auto_configuration_steps():
    assert slo_queue.alpha_update(0.25, 0.50, 0.60) == 0.5          # rose by 0.10 > 0.04
    assert slo_queue.alpha_update(0.75, 0.50, 0.60) == 1.0          # capped at 1
    assert slo_queue.alpha_update(0.5, 0.60, 0.50) == 0.25          # fell
    assert slo_queue.alpha_update(0.5, 0.60, 0.63) == 0.5           # within the threshold
    assert slo_queue.alpha_update(0.5, 0.60, 0.63, scalar=3.0, threshold=-0.01) == 1.0
