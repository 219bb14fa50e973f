"""Host-side checks of the C ABI (no GPU): exported symbols, descriptor validation, the
chunk plan and the arena bookkeeping against the oracle's reference rules."""
import os
import re
import subprocess

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import paper_2306_03622_amd as tp
import synth
from oracle import chunks as ref_chunks
from oracle.arena_sim import ArenaSim, NoSpace
from oracle.partition_sim import PartitionArenaSim

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    names = set()
    for h in ("torpor.h", "torpor_plan.h"):
        src = open(os.path.join(ROOT, "include", h)).read()
        names |= set(re.findall(r"^TP_API\s+[\w\s\*]+?\b(tph?_\w+)\s*\(", src, re.M))
    return names


def test_library_exports_every_declared_symbol():
    names = declared_symbols()
    assert len(names) == 40, sorted(names)
    L = tp.lib()
    for n in names:
        assert hasattr(L, n), n
    out = subprocess.run(["nm", "-D", "--defined-only", tp.torpor.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r" T (tph?_\w+)", out))
    assert exported == names, exported ^ names
    host = subprocess.run(["nm", "-D", "--defined-only", tp.torpor.HOST_LIB_PATH], capture_output=True, text=True).stdout
    assert set(re.findall(r" T (tph?_\w+)", host)) == {n for n in names if n.startswith("tph_")} | {"tp_last_error"}


def test_probe_library_exports_its_header():
    src = open(os.path.join(ROOT, "include", "torpor_probe.h")).read()
    declared = set(re.findall(r"^TPP_API\s+[\w\s\*]+?\b(tpp_\w+)\s*\(", src, re.M))
    assert declared == {"tpp_mfma_bf16", "tpp_hbm_read", "tpp_gather_h2d"}
    out = subprocess.run(["nm", "-D", "--defined-only", tp.torpor.PROBE_LIB_PATH], capture_output=True, text=True).stdout
    assert set(re.findall(r" T (tpp_\w+)", out)) == declared
    L = tp.torpor.probe_lib()
    for n in declared:
        assert hasattr(L, n)


def _desc(model, mutate=None, dims=None, dtype=None):
    tensors = [[t.layer, t.role, t.offset, t.nbytes, list(t.shape)] for t in model.tensors]
    if mutate:
        mutate(tensors)
    d = tp.ModelDesc.of(model)
    return tp.ModelDesc(model.arch, dtype or model.dtype, dims or list(d.desc.dims), [tuple(t) for t in tensors])


@pytest.mark.parametrize("case", ["shape", "missing", "dup", "misaligned", "overlap", "order", "bounds", "bytes",
                                  "dims", "dtype", "role"])
def test_validation_rejects_malformed_layouts(case):
    m = synth.bert(seed=1, layers=2, d=128, heads=2, ffn=256, seq=64, vocab=100, maxpos=64)
    kw = {}
    mut = None
    if case == "shape":
        mut = lambda t: t[3].__setitem__(4, [2, 128 * 3])
    elif case == "missing":
        mut = lambda t: t.pop(7)
    elif case == "dup":
        mut = lambda t: t[6].__setitem__(1, t[5][1])
    elif case == "misaligned":
        mut = lambda t: t[3].__setitem__(2, t[3][2] + 2)
    elif case == "overlap":
        mut = lambda t: t[3].__setitem__(2, t[2][2])
    elif case == "order":
        mut = lambda t: t.insert(0, t.pop(10))
    elif case == "bounds":
        mut = lambda t: t[-1].__setitem__(2, m.total_bytes + 256)
    elif case == "bytes":
        mut = lambda t: t[5].__setitem__(3, t[5][3] + 2)
    elif case == "dims":
        kw["dims"] = [2, 128, 3, 256, 64, 100, 64]
    elif case == "dtype":
        kw["dtype"] = "f32"
    elif case == "role":
        mut = lambda t: t[0].__setitem__(1, "w")
    d = _desc(m, mut, **kw)
    with pytest.raises(tp.TorporError) as e:
        tp.tph_validate(d, m.total_bytes)
    assert e.value.status == tp.TP_E_INVAL
    assert tp.lib().tp_last_error().decode()
    tp.tph_validate(tp.ModelDesc.of(m), m.total_bytes)        # the unmodified layout passes


def test_validation_accepts_all_workloads():
    for cfg in (1, 2, 3, 4):
        m = synth.config_model(cfg)
        tp.tph_validate(tp.ModelDesc.of(m), m.total_bytes)


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
@pytest.mark.parametrize("g", [0, 64 << 10, 2 << 20, 16 << 20, 1 << 40])
@pytest.mark.parametrize("per_tensor", [False, True])
def test_chunk_plan_matches_reference(cfg, g, per_tensor):
    m = synth.config_model(cfg)
    want = ref_chunks.plan([(t.layer, t.offset, t.nbytes) for t in m.tensors], m.total_bytes, g, per_tensor)
    flags = tp.TP_FLAG_PER_TENSOR if per_tensor else 0
    for L in (tp.lib(), tp.host_lib()):
        got = tp.tph_plan(tp.ModelDesc.of(m), m.total_bytes, g, flags, L=L)
        assert [(c["begin"], c["end"], c["first_layer"]) for c in got] == \
            [(c["begin"], c["end"], c["first_layer"]) for c in want]


def test_workspace_grows_with_batch():
    for cfg in (1, 2, 3, 4):
        d = tp.ModelDesc.of(synth.config_model(cfg))
        w = [tp.tp_workspace_bytes(d, b) for b in (1, 2, 8)]
        assert 0 < w[0] <= w[1] <= w[2]


def _replay(trace, sizes, cap, L, policy="lru", heavy=None):
    sim = ArenaSim(cap, align=256, policy=policy)
    ha = tp.HostArena(cap, 256, L=L, policy={"lru": tp.TP_EVICT_LRU, "heaviness": tp.TP_EVICT_HEAVINESS,
                                             "lru_window": tp.TP_EVICT_LRU_WINDOW}[policy])
    heavy = heavy or [False] * len(sizes)
    for i, nb in enumerate(sizes):
        sim.register(i, nb, heavy=heavy[i])
        ha.register(i, nb, heavy=heavy[i])
    for op, k in trace:
        if op == "evict":
            sim.evict(k)
            ha.evict(k)
            continue
        if op == "flip":
            sim.set_heavy(k, not sim.heavy[k])
            ha.set_heavy(k, sim.heavy[k])
            continue
        try:
            want = sim.request(k)
        except NoSpace:
            with pytest.raises(tp.TorporError) as e:
                ha.request(k)
            assert e.value.status == tp.TP_E_NOSPC
            continue
        assert ha.request(k) == want
    got = ha.stats()
    assert {k: got[k] for k in sim.stats()} == sim.stats() and got["registered"] == len(sizes)
    assert got["admit_calls"] == 0       # admissions are timed by the runtime, not the bookkeeping


@settings(max_examples=80, deadline=None)
@given(base=st.lists(st.integers(1, 90).map(lambda x: x * 100), min_size=1, max_size=4),
       picks=st.lists(st.integers(0, 40), min_size=2, max_size=10),
       ops=st.lists(st.tuples(st.sampled_from(["req"] * 6 + ["evict", "reg"]), st.integers(0, 9)), max_size=100),
       part_units=st.integers(1, 40), n_parts=st.integers(1, 6), tail=st.integers(0, 5),
       policy=st.sampled_from(["lru", "heaviness"]), bits=st.integers(0, 1023), consolidate=st.booleans())
def test_partitioned_arena_matches_simulator(base, picks, ops, part_units, n_parts, tail, policy, bits,
                                             consolidate):
    """tph_arena with two-tier partitions, with and without consolidation, against the
    oracle's partition simulator: offsets, victims, moves and counters, with models
    registered and unregistered on the way (a size class is common only while two
    registered models share it)."""
    sizes = [base[p % len(base)] if p < 30 else p * 170 for p in picks]
    part = part_units * 256
    cap = n_parts * part + tail * 256
    for L in (tp.lib(), tp.host_lib()):
        sim = PartitionArenaSim(cap, part, 256, policy, consolidate=consolidate)
        ha = tp.HostArena(cap, 256, L=L, partition=part, consolidate=consolidate,
                          policy=tp.TP_EVICT_HEAVINESS if policy == "heaviness" else tp.TP_EVICT_LRU)
        live = set()
        for i, nb in enumerate(sizes):
            sim.register(i, nb, bool(bits >> i & 1))
            ha.register(i, nb, bool(bits >> i & 1))
            live.add(i)
        for op, k in ops:
            k %= len(sizes)
            if op == "reg":
                if k in live:
                    sim.unregister(k)
                    ha.unregister(k)
                    live.discard(k)
                else:
                    sim.register(k, sizes[k], bool(bits >> k & 1))
                    ha.register(k, sizes[k], bool(bits >> k & 1))
                    live.add(k)
                continue
            if k not in live:
                continue
            if op == "evict":
                sim.evict(k)
                ha.evict(k)
                continue
            try:
                want = sim.request(k)
            except NoSpace:
                with pytest.raises(tp.TorporError) as e:
                    ha.request(k)
                assert e.value.status == tp.TP_E_NOSPC
                continue
            assert ha.request(k) == want
        got, want = ha.stats(), sim.stats()
        assert {k: got[k] for k in want} == want


def test_partitioned_arena_seeded_sweep():
    """3000 seeded traces against the oracle: registration churn makes size classes switch
    between common and irregular while their models are resident (so evacuated models may
    change tier), partitions of 1 to 64 units with and without a short tail, both eviction
    policies, consolidation on half of them; every decision, move order and counter equal."""
    import random
    L = tp.host_lib()
    evacuations = 0
    for seed in range(3000):
        r = random.Random(seed)
        part = 256 * r.choice([1, 2, 3, 4, 8, 16, 12, 40, 64])
        cap = part * r.randint(1, 6) + 256 * r.choice([0, 0, 1, 3, 7])
        n = r.randint(2, 10)
        base = [r.choice([1, 2, 3, 5, 8, 13, 20, 40, 70]) * 100 for _ in range(4)]
        sizes = [r.choice(base) if r.random() < 0.6 else r.randint(1, 80) * 100 for _ in range(n)]
        policy = r.choice(["lru", "heaviness"])
        consolidate = r.random() < 0.5
        heavy = [r.random() < 0.3 for _ in range(n)]
        sim = PartitionArenaSim(cap, part, 256, policy, consolidate=consolidate)
        ha = tp.HostArena(cap, 256, L=L, partition=part, consolidate=consolidate,
                          policy=tp.TP_EVICT_HEAVINESS if policy == "heaviness" else tp.TP_EVICT_LRU)
        live = set(range(n))
        for i in range(n):
            sim.register(i, sizes[i], heavy[i])
            ha.register(i, sizes[i], heavy[i])
        for _ in range(120):
            op, k = r.choice(["req"] * 6 + ["evict", "reg"]), r.randrange(n)
            if op == "reg":
                if k in live:
                    sim.unregister(k)
                    ha.unregister(k)
                    live.discard(k)
                else:
                    sim.register(k, sizes[k], heavy[k])
                    ha.register(k, sizes[k], heavy[k])
                    live.add(k)
            elif k in live and op == "evict":
                sim.evict(k)
                ha.evict(k)
            elif k in live:
                try:
                    want = sim.request(k)
                except NoSpace:
                    with pytest.raises(tp.TorporError):
                        ha.request(k)
                    continue
                assert ha.request(k) == want, seed
        got, want = ha.stats(), sim.stats()
        assert {k: got[k] for k in want} == want, seed
        evacuations += got["evacuations"]
    assert evacuations > 100


def test_partitioned_arena_errors():
    ha = tp.HostArena(1 << 20, 256, L=tp.host_lib())
    with pytest.raises(tp.TorporError) as e:
        ha.set_partitioned(1000)                    # not a multiple of the alignment
    assert e.value.status == tp.TP_E_INVAL
    ha.register(0, 5000)
    ha.request(0)
    with pytest.raises(tp.TorporError) as e:
        ha.set_partitioned(4096)                    # a model is resident
    assert e.value.status == tp.TP_E_STATE
    ha.evict(0)
    ha.set_partitioned(4096)
    assert ha.request(0)["offset"] == 0             # 5120 bytes > 4096: a run of two partitions, lowest first
    st_ = ha.stats()
    assert st_["partitions"] == 256 and st_["partitions_free"] == 254
    assert st_["evacuations"] == 0 and st_["bytes_moved"] == 0


@settings(max_examples=60, deadline=None)
@given(sizes=st.lists(st.integers(1, 40) .map(lambda x: x * 1000), min_size=2, max_size=10),
       ops=st.lists(st.tuples(st.sampled_from(["req", "req", "req", "evict"]), st.integers(0, 9)), max_size=80),
       frac=st.floats(0.2, 1.2))
def test_arena_matches_simulator_random_traces(sizes, ops, frac):
    cap = max(int(sum(sizes) * frac), 256) // 256 * 256
    trace = [(op, k % len(sizes)) for op, k in ops]
    _replay(trace, sizes, cap, tp.lib())
    _replay(trace, sizes, cap, tp.host_lib())


@settings(max_examples=60, deadline=None)
@given(sizes=st.lists(st.integers(1, 40).map(lambda x: x * 1000), min_size=2, max_size=10),
       ops=st.lists(st.tuples(st.sampled_from(["req", "req", "req", "req", "evict", "flip"]), st.integers(0, 9)),
                    max_size=80),
       frac=st.floats(0.2, 1.2), heavy_bits=st.integers(0, 1023))
def test_arena_heaviness_policy_matches_simulator(sizes, ops, frac, heavy_bits):
    cap = max(int(sum(sizes) * frac), 256) // 256 * 256
    heavy = [bool((heavy_bits >> i) & 1) for i in range(len(sizes))]
    trace = [(op, k % len(sizes)) for op, k in ops]
    _replay(trace, sizes, cap, tp.lib(), "heaviness", heavy)
    _replay(trace, sizes, cap, tp.host_lib(), "heaviness", heavy)


@settings(max_examples=60, deadline=None)
@given(sizes=st.lists(st.integers(1, 40).map(lambda x: x * 1000), min_size=2, max_size=12),
       ops=st.lists(st.tuples(st.sampled_from(["req", "req", "req", "req", "evict"]), st.integers(0, 11)),
                    max_size=100),
       frac=st.floats(0.2, 1.2))
def test_arena_window_policy_matches_simulator(sizes, ops, frac):
    cap = max(int(sum(sizes) * frac), 256) // 256 * 256
    trace = [(op, k % len(sizes)) for op, k in ops]
    _replay(trace, sizes, cap, tp.lib(), "lru_window")
    _replay(trace, sizes, cap, tp.host_lib(), "lru_window")


def test_arena_policy_errors():
    ha = tp.HostArena(10_000, 256)
    with pytest.raises(tp.TorporError) as e:
        tp.torpor._check(ha.L, ha.L.tph_arena_set_policy(ha.h, 7))
    assert e.value.status == tp.TP_E_INVAL
    with pytest.raises(tp.TorporError) as e:
        ha.set_heavy(3, True)
    assert e.value.status == tp.TP_E_NOENT


def test_arena_unregister_and_errors():
    ha = tp.HostArena(10_000, 256)
    ha.register(1, 5000)
    with pytest.raises(tp.TorporError) as e:
        ha.register(1, 10)
    assert e.value.status == tp.TP_E_STATE
    with pytest.raises(tp.TorporError) as e:
        ha.request(7)
    assert e.value.status == tp.TP_E_NOENT
    ha.request(1)
    ha.unregister(1)
    assert ha.stats()["used"] == 0 and ha.stats()["registered"] == 0


def test_blocked_layout_definition():
    # the test-side definition of the blocked order, pinned on a small matrix by hand
    from tests.common import pack_rows16x128
    w = np.arange(16 * 128, dtype=np.uint16).reshape(16, 128)
    p = pack_rows16x128(w)
    # first 8 elements: row 0, columns 0..7; next 8: row 1, columns 0..7
    assert p[:8].tolist() == list(range(8)) and p[8:16].tolist() == list(range(128, 136))
    # slot q = 1 starts after 16 rows: row 0, columns 8..15
    assert p[128:136].tolist() == list(range(8, 16))
    # group j = 1 starts at 512: row 0, columns 32..39
    assert p[512:520].tolist() == list(range(32, 40))
    assert sorted(p.tolist()) == list(range(16 * 128))


def _random_instance(rng, n):
    sizes = rng.integers(1, 200, size=n) * 256
    begin = np.concatenate([[0], np.cumsum(sizes)[:-1]]).tolist()
    total = int(sizes.sum()) + int(rng.integers(0, 4)) * 256
    us = (rng.random(n) * rng.choice([1.0, 30.0, 300.0])).tolist()
    return begin, total, us


@pytest.mark.parametrize("seed", range(40))
def test_cost_plan_is_optimal_against_exhaustion(seed):
    from oracle import pipeline
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 11))
    begin, total, us = _random_instance(rng, n)
    rate, o, h = float(rng.choice([50.0, 500.0, 5000.0])), float(rng.choice([1.0, 15.0, 200.0])), float(rng.random() * 10)
    want_first, want_t = pipeline.best_grouping(begin, total, us, rate, o, h)
    for L in (tp.lib(), tp.host_lib()):
        first, est = tp.tph_plan_cost(begin, us, total, rate, o, h, L=L)
        # the library's modelled time is the oracle's time of the library's grouping, and no
        # grouping is faster; the number of groups is the fewest among the fastest
        assert est == pytest.approx(pipeline.simulate(begin, total, us, first, rate, o, h), rel=1e-9, abs=1e-9)
        assert est <= want_t * (1 + 1e-9) + 1e-9
        assert len(first) <= len(want_first)


def test_cost_plan_errors():
    bad = [([5, 10], [1.0, 1.0], 20),        # unit 0 must start at byte 0
           ([0, 10, 10], [1.0] * 3, 20),     # offsets must increase
           ([0, 10], [1.0, -1.0], 20),       # negative time
           ([0, 10], [1.0, 1.0], 10)]        # the buffer must extend past the last unit
    for begin, us, total in bad:
        with pytest.raises(tp.TorporError) as e:
            tp.tph_plan_cost(begin, us, total, 10.0, 1.0, 1.0, L=tp.host_lib())
        assert e.value.status == tp.TP_E_INVAL
    with pytest.raises(tp.TorporError):
        tp.tph_plan_cost([0], [1.0], 10, 0.0, 1.0, 1.0, L=tp.host_lib())


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
@pytest.mark.parametrize("batch", [1, 8])
def test_cost_plan_of_workloads(cfg, batch):
    from oracle import pipeline
    m = synth.config_model(cfg)
    d = tp.ModelDesc.of(m)
    plan, est = tp.tph_plan_cost_model(d, m.total_bytes, batch, 57.0, 15.0, L=tp.host_lib())
    # chunks tile the buffer at layer starts, in first-use order
    assert plan[0]["begin"] == 0 and plan[-1]["end"] == m.total_bytes
    assert all(a["end"] == b["begin"] for a, b in zip(plan, plan[1:]))
    layer_start = {}
    for t in m.tensors:
        layer_start.setdefault(t.layer, t.offset)
    assert all(c["begin"] == layer_start[c["first_layer"]] for c in plan[1:])
    # the modelled time is the oracle's simulation of this grouping, and it is no worse than
    # the greedy plan at the default group size under the same model
    us = tp.tph_layer_costs(d, m.total_bytes, batch, L=tp.host_lib())
    begin = [0] + [layer_start[l] for l in range(1, len(us))]
    first = [c["first_layer"] for c in plan]
    assert est == pytest.approx(pipeline.simulate(begin, m.total_bytes, us, first, 57e3, 15.0, 5.0), rel=1e-9)
    greedy = tp.tph_plan(d, m.total_bytes, tp.DEFAULT_CHUNK, 0, L=tp.host_lib())
    g_first = [c["first_layer"] for c in greedy]
    assert est <= pipeline.simulate(begin, m.total_bytes, us, g_first, 57e3, 15.0, 5.0) + 1e-6
    # the transfer alone bounds the modelled time from below
    assert est >= m.total_bytes / 57e3
    assert all(u > 0 for u in us)


@settings(max_examples=200, deadline=None)
@given(counts=st.lists(st.tuples(st.integers(0, 60), st.integers(0, 60)), min_size=1, max_size=12),
       alpha=st.sampled_from([0.0, 0.03125, 0.125, 0.25, 0.5, 0.75, 1.0]),
       p=st.sampled_from([0.5, 0.9, 0.98, 0.99]), pend=st.lists(st.integers(0, 11), max_size=20))
def test_sched_pick_matches_oracle(counts, alpha, p, pend):
    from oracle import slo_queue
    n = [max(a, b) for a, b in counts]
    m = [min(a, b) for a, b in counts]
    pend = [f % len(n) for f in pend]
    rr = [slo_queue.rrc(a, b, p) for a, b in zip(n, m)]
    want_high = slo_queue.high_group(rr, alpha)
    want = slo_queue.pick(rr, want_high, pend)
    for L in (tp.lib(), tp.host_lib()):
        got, high = tp.tph_sched_pick(n, m, p, alpha, pend, L=L)
        assert high == want_high and got == want
        assert tp.tph_rrc(n[0], m[0], p, L=L) == pytest.approx(rr[0])


@pytest.mark.parametrize("alpha,last,new", [(0.25, 0.5, 0.6), (0.75, 0.5, 0.6), (0.5, 0.6, 0.5), (0.5, 0.6, 0.63),
                                            (1.0, 0.2, 0.9), (0.01, 0.9, 0.1)])
def test_alpha_update_matches_oracle(alpha, last, new):
    from oracle import slo_queue
    for L in (tp.lib(), tp.host_lib()):
        assert tp.tph_alpha_update(alpha, last, new, 2.0, 0.04, L=L) == slo_queue.alpha_update(alpha, last, new, 2.0, 0.04)
    with pytest.raises(tp.TorporError):
        tp.tph_alpha_update(alpha, last, new, 1.0, 0.04, L=tp.host_lib())
