"""Multi-tenant open-loop replay (tp_run_trace) on the GPU, scaled down: 9 models of the
three families, an arena that holds about a third of them, Poisson/Zipf arrivals, under
LRU, heaviness-aware and contiguous-window eviction.

Checks: every request's hit flag and the arena's counters equal the reference simulator
replayed on the same request sequence; every model's first output matches the oracle."""
import numpy as np
import pytest

import paper_2306_03622_amd as tp
import synth
from oracle import forward as oracle
from oracle.arena_sim import ArenaSim
from oracle.partition_sim import PartitionArenaSim
from tests.common import log, out_shape, to_device, torch_dev

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("policy", ["lru", "heaviness", "lru_window"])
def test_tenant_trace_lru_and_first_outputs(policy):
    torch, dev = torch_dev()
    specs = synth.tenant_models(9)
    models = [m for _, m in synth.build_models(specs, workers=9)]
    trace = synth.tenant_trace(120, n_models=9)
    cap = (models[0].total_bytes + models[1].total_bytes + models[2].total_bytes) // 256 * 256 + (64 << 20)
    ws = max(tp.tp_workspace_bytes(tp.ModelDesc.of(m), 1) for m in models)
    rt = tp.Runtime(cap, ws, evict_policy={"lru": tp.TP_EVICT_LRU, "heaviness": tp.TP_EVICT_HEAVINESS,
                                           "lru_window": tp.TP_EVICT_LRU_WINDOW}[policy])
    ids = [rt.register(tp.ModelDesc.of(m), m.blob()) for m in models]
    heavy = [bool(rt.info(i)["heavy"]) for i in ids]
    # the cost model classes the transfer-bound families heavy and ResNet-50 (whose compute
    # hides most of its transfer) light
    assert heavy == [m.arch != "resnet50" for m in models], heavy
    xs_np, reqs, outs = [], [], []
    for r in range(len(trace.model)):
        m = models[int(trace.model[r])]
        x_np = synth.request_input(m, int(trace.input_seed[r]))
        xs_np.append(x_np)
        y = torch.full(out_shape(m, 1), float("nan"), dtype=torch.float32, device=dev)
        outs.append(y)
        reqs.append((ids[int(trace.model[r])], 1, to_device(x_np), y, int(trace.arrival_s[r] * 1e9)))
    torch.cuda.synchronize()
    log(f"replaying {len(reqs)} requests over {trace.arrival_s[-1]:.2f} s")
    res = rt.run_trace(reqs)
    torch.cuda.synchronize()
    assert all(r["status"] == 0 for r in res)
    assert all(r["done_ns"] >= r["issue_ns"] for r in res)

    sim = ArenaSim(cap, align=256, policy=policy)
    for i, m, h in zip(ids, models, heavy):
        sim.register(i, m.total_bytes, heavy=h)
    want_hits = [sim.request(q[0])["hit"] for q in reqs]
    assert [r["hit"] for r in res] == want_hits
    got = rt.stats()
    for k, v in sim.stats().items():
        assert got[k] == v, (k, got[k], v)
    log(f"hit rate {np.mean(want_hits):.3f}, evictions {got['evictions']}")

    seen = set()
    for r, q in enumerate(reqs):
        k = int(trace.model[r])
        if k in seen:
            continue
        seen.add(k)
        y = outs[r].cpu().numpy()
        err = oracle.normwise_error(y, oracle.forward(models[k], xs_np[r])).max()
        log(f"  model {k} ({models[k].arch}) first request {r}: error {err:.2e}")
        assert np.all(np.isfinite(y)) and err <= 2e-2
    rt.close()


@pytest.mark.parametrize("policy", [tp.TP_QUEUE_FIFO, tp.TP_QUEUE_SLO])
def test_scheduled_replay(policy):
    # the same scaled workload at 4x the arrival rate with a host-side queue: every request
    # completes after its arrival and issue, at most max_inflight are outstanding, FIFO issues
    # in arrival order, and the first output of every model matches the oracle
    torch, dev = torch_dev()
    specs = synth.tenant_models(9)
    models = [m for _, m in synth.build_models(specs, workers=9)]
    trace = synth.tenant_trace(120, rate_per_s=200.0, n_models=9)
    cap = (models[0].total_bytes + models[1].total_bytes + models[2].total_bytes) // 256 * 256 + (64 << 20)
    ws = max(tp.tp_workspace_bytes(tp.ModelDesc.of(m), 1) for m in models)
    rt = tp.Runtime(cap, ws)
    ids = [rt.register(tp.ModelDesc.of(m), m.blob()) for m in models]
    deadline_ms = {"mlp": 40.0, "resnet50": 3.0, "bert": 12.0}
    xs_np, reqs, outs, dls = [], [], [], []
    for r in range(len(trace.model)):
        m = models[int(trace.model[r])]
        x_np = synth.request_input(m, int(trace.input_seed[r]))
        xs_np.append(x_np)
        y = torch.full(out_shape(m, 1), float("nan"), dtype=torch.float32, device=dev)
        outs.append(y)
        reqs.append((ids[int(trace.model[r])], 1, to_device(x_np), y, int(trace.arrival_s[r] * 1e9)))
        dls.append(int(deadline_ms[m.arch] * 1e6))
    torch.cuda.synchronize()
    res, stats = rt.run_trace_sched(reqs, dls, policy=policy, max_inflight=2, period_ns=100_000_000)
    torch.cuda.synchronize()
    log(f"policy {policy}: stats {stats}")
    assert all(r["status"] == 0 for r in res)
    for r, q in zip(res, reqs):
        assert q[4] <= r["issue_ns"] <= r["done_ns"]
    events = sorted([(r["issue_ns"], 1) for r in res] + [(r["done_ns"], -1) for r in res], key=lambda e: (e[0], e[1]))
    live = 0
    for _, d in events:
        live += d
        assert live <= 2
    if policy == tp.TP_QUEUE_FIFO:
        assert [r["issue_ns"] for r in res] == sorted(r["issue_ns"] for r in res)
    assert stats["functions"] == len(set(int(v) for v in trace.model)) and stats["compliant"] <= stats["functions"]
    assert 0 < stats["alpha"] <= 1 and stats["periods"] >= 1
    seen = set()
    for r, q in enumerate(reqs):
        k = int(trace.model[r])
        if k in seen:
            continue
        seen.add(k)
        y = outs[r].cpu().numpy()
        err = oracle.normwise_error(y, oracle.forward(models[k], xs_np[r])).max()
        assert np.all(np.isfinite(y)) and err <= 2e-2, (k, err)
    rt.close()


@pytest.mark.parametrize("alloc", [tp.TP_ALLOC_PARTITION, tp.TP_ALLOC_PARTITION_CONSOLIDATE])
def test_partitioned_arena_trace(alloc):
    # The scaled workload on a 1100 MiB arena of two 512 MiB partitions and a short one:
    # MLPs take runs of both full partitions, ResNet-50 and BERT-base slots of partitions of
    # their class; with consolidation the trace makes 11 evacuations (1171 MiB moved) where
    # the arena would otherwise evict. Retired extents are poisoned (NaN in bf16). Checks:
    # hit flags and counters (moves included) equal the oracle's partition simulator, and
    # every request's output equals the same request's on an arena that holds all models.
    torch, dev = torch_dev()
    specs = synth.tenant_models(9)
    models = [m for _, m in synth.build_models(specs, workers=9)]
    trace = synth.tenant_trace(120, n_models=9)
    cap, part = 1100 << 20, 512 << 20
    ws = max(tp.tp_workspace_bytes(tp.ModelDesc.of(m), 1) for m in models)
    xs, outs, ref_outs = [], [], []
    for r in range(len(trace.model)):
        m = models[int(trace.model[r])]
        xs.append(to_device(synth.request_input(m, int(trace.input_seed[r]))))
        outs.append(torch.full(out_shape(m, 1), float("nan"), dtype=torch.float32, device=dev))
        ref_outs.append(torch.full(out_shape(m, 1), float("nan"), dtype=torch.float32, device=dev))

    def replay(rt, ys):
        ids = [rt.register(tp.ModelDesc.of(m), m.blob()) for m in models]
        reqs = [(ids[int(trace.model[r])], 1, xs[r], ys[r], int(trace.arrival_s[r] * 1e9))
                for r in range(len(trace.model))]
        torch.cuda.synchronize()
        res = rt.run_trace(reqs)
        torch.cuda.synchronize()
        assert all(q["status"] == 0 for q in res)
        return ids, res

    big = sum(m.total_bytes for m in models) + (64 << 20)
    rt = tp.Runtime(big // 256 * 256, ws)
    replay(rt, ref_outs)
    rt.close()

    rt = tp.Runtime(cap, ws, alloc=alloc, partition_bytes=part, flags=tp.TP_FLAG_POISON)
    ids, res = replay(rt, outs)
    consolidate = alloc == tp.TP_ALLOC_PARTITION_CONSOLIDATE
    sim = PartitionArenaSim(cap, part, 256, consolidate=consolidate)
    for i, m in zip(ids, models):
        sim.register(i, m.total_bytes)
    want_hits = [sim.request(ids[int(k)])["hit"] for k in trace.model]
    assert [q["hit"] for q in res] == want_hits
    got, want = rt.stats(), sim.stats()
    for k, v in want.items():
        assert got[k] == v, (k, got[k], v)
    if consolidate:
        assert got["evacuations"] == 11
    assert all((q["admit_ns"] > 0) == (not q["hit"]) for q in res)
    log(f"alloc {alloc}: hit rate {np.mean(want_hits):.3f}, evictions {got['evictions']}, "
        f"evacuations {got['evacuations']}, moved {got['bytes_moved'] >> 20} MiB")
    worst = 0.0
    for r in range(len(outs)):
        y, ref = outs[r].cpu().numpy(), ref_outs[r].cpu().numpy()
        assert np.all(np.isfinite(y)), r
        err = float(np.abs(y - ref).max() / max(np.abs(ref).max(), 1e-30))
        worst = max(worst, err)
        assert err <= 1e-5, (r, int(trace.model[r]), err)
    log(f"  largest relative difference from the all-resident run: {worst:.1e}")
    rt.close()
