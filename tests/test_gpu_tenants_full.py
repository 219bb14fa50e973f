"""The multi-tenant workload at its stated size, against the oracle.

100 registered models (model i: the 24 x 4096 MLP, ResNet-50 or BERT-base by i mod 3, weight
seed 1000 + i; 36.26 GB of pinned host copies), an 8 GiB arena, 3000 requests at batch 1 with
Poisson arrivals at 50 per second and Zipf(1.1) popularity, replayed open loop by
tp_run_trace under LRU or contiguous-window eviction and first-fit placement; every request
brings input and output buffers of its own. Checks:
  * every request's hit flag, and the arena's counters, equal the oracle's arena simulator
    replayed on the same request sequence (paper Sec. 4.3 "Model eviction", Sec. 5.4 LRU);
  * the first request of every requested model matches the oracle's float64 forward pass
    (normwise per sample, 2e-2 for bf16);
  * warm requests capture a graph only at the first hit after a swap to a new extent; every
    other hit repoints a cached graph at its own buffers.
It writes a summary (latency, hit rates beside a byte-capacity LRU without contiguity, the
achieved errors) to tenants_full_<policy>.json in the results folder ($TP_RESULTS_DIR, else
results/ at the repository root). It takes about four minutes per
policy, so it runs only when TP_FULL_TENANTS=1 is set."""
import json
import os
import time
from collections import OrderedDict

import numpy as np
import pytest

import paper_2306_03622_amd as tp
import synth
from oracle import forward as oracle
from oracle.arena_sim import ArenaSim
from tests.common import RESULTS_DIR, log, out_shape, record_parity, to_device, torch_dev

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(os.environ.get("TP_FULL_TENANTS") != "1",
                                 reason="full-size multi-tenant replay (about 4 minutes): set TP_FULL_TENANTS=1")]

N_MODELS, N_REQUESTS, ARENA = 100, 3000, 8 << 30


def byte_lru_hits(sizes, sequence, capacity):
    """Hits of a plain LRU cache holding at most `capacity` bytes (no placement constraint)."""
    lru, used, hits = OrderedDict(), 0, []
    for k in sequence:
        if k in lru:
            lru.move_to_end(k)
            hits.append(True)
            continue
        hits.append(False)
        while used + sizes[k] > capacity:
            _, b = lru.popitem(last=False)
            used -= b
        lru[k] = sizes[k]
        used += sizes[k]
    return hits


@pytest.mark.parametrize("policy", ["lru", "lru_window"])
def test_full_size_trace_matches_oracle(policy):
    torch, dev = torch_dev()
    specs = synth.tenant_models(N_MODELS)
    trace = synth.tenant_trace(N_REQUESTS, n_models=N_MODELS)
    first = {}
    for r, k in enumerate(trace.model):
        first.setdefault(int(k), r)
    log(f"{len(first)} of {N_MODELS} models are requested")
    ws = max(tp.tp_workspace_bytes(tp.ModelDesc.of(synth.config_model(c, 0)), 1) for c in (2, 3, 4))
    rt = tp.Runtime(ARENA, ws, plan=tp.TP_PLAN_COST,
                    evict_policy=tp.TP_EVICT_LRU_WINDOW if policy == "lru_window" else tp.TP_EVICT_LRU)
    ids, sizes, kinds, expected, inputs = [], {}, {}, {}, {}
    t0 = time.perf_counter()
    for i, m in synth.build_models(specs, workers=16):
        mid = rt.register(tp.ModelDesc.of(m), m.blob())
        ids.append(mid)
        sizes[mid], kinds[mid] = m.total_bytes, m.arch
        if i in first:            # the oracle's output for the model's first request, from the same bytes
            r = first[i]
            inputs[r] = synth.request_input(m, int(trace.input_seed[r]))
            expected[r] = (oracle.forward(m, inputs[r]), m)
        m.drop_blob()
        if i % 10 == 9:
            log(f"  registered {i + 1} models, oracle outputs for {len(expected)} ({time.perf_counter() - t0:.0f} s)")
    protos = {c: synth.config_model(c, 0) for c in (2, 3, 4)}       # shapes only
    reqs, outs = [], []
    for r in range(N_REQUESTS):
        k = int(trace.model[r])
        proto = protos[specs[k][0]]
        x = inputs.get(r)
        if x is None:
            x = synth.request_input(proto, int(trace.input_seed[r]))
        y = torch.full(out_shape(proto, 1), float("nan"), dtype=torch.float32, device=dev)
        outs.append(y)
        reqs.append((ids[k], 1, to_device(x), y, int(trace.arrival_s[r] * 1e9)))
    torch.cuda.synchronize()
    log(f"replaying {N_REQUESTS} requests over {trace.arrival_s[-1]:.1f} s")
    stream = torch.cuda.Stream(device=dev)
    res = rt.run_trace(reqs, stream=stream)
    torch.cuda.synchronize()
    assert all(q["status"] == 0 for q in res)
    st = rt.stats()

    sim = ArenaSim(ARENA, align=256, policy=policy)
    for mid in ids:
        sim.register(mid, sizes[mid])
    decisions = [sim.request(q[0]) for q in reqs]
    want_hits = [d["hit"] for d in decisions]
    got_hits = [bool(q["hit"]) for q in res]
    mismatch = [r for r, (a, b) in enumerate(zip(got_hits, want_hits)) if a != b]
    assert not mismatch, mismatch[:10]
    for key, v in sim.stats().items():
        assert st[key] == v, (key, st[key], v)

    errors = {}
    for r, (ref, m) in sorted(expected.items()):
        got = outs[r].cpu().numpy()
        err = float(oracle.normwise_error(got, ref).max())
        errors[r] = (m.arch, err)
        record_parity(m, 1, err, 2e-2)
        assert np.all(np.isfinite(got)), r
    worst = {a: max((e for aa, e in errors.values() if aa == a), default=None) for a in ("mlp", "resnet50", "bert")}
    log(f"first-request errors, worst per family: {worst}")
    assert all(e <= 2e-2 for _, e in errors.values()), [(r, a, e) for r, (a, e) in errors.items() if e > 2e-2]

    # Warm requests replay a graph per (model, batch): the first hit of a model captures it,
    # every later hit repoints it at its own buffers, and a hit in another extent than the
    # model's previous hit also moves the graph's weight pointers; no hit captures again.
    last_hit_off, want_captures, want_rebases = {}, 0, 0
    for rq, d in zip(reqs, decisions):
        if not d["hit"]:
            continue
        prev = last_hit_off.get(rq[0])
        if prev is None:
            want_captures += 1
        elif prev != d["offset"]:
            want_rebases += 1
        last_hit_off[rq[0]] = d["offset"]
    log(f"graph captures {st['graph_captures']} (expected {want_captures}), repoints {st['graph_repoints']}, "
        f"rebases {st['graph_rebases']} (expected {want_rebases})")
    assert st["graph_captures"] == want_captures, st
    assert st["graph_repoints"] == st["hits"] - want_captures, st
    assert st["graph_rebases"] == want_rebases, st
    lat = np.array([(q["done_ns"] - rq[4]) / 1e6 for q, rq in zip(res, reqs)])
    arch = np.array([kinds[rq[0]] for rq in reqs])
    hits = np.array(got_hits)
    idle = np.array([i == 0 or res[i]["issue_ns"] >= res[i - 1]["done_ns"] for i in range(len(res))])
    lru = byte_lru_hits(sizes, [rq[0] for rq in reqs], ARENA)
    summary = {
        "workload": f"{N_MODELS} models (24x4096 MLP / ResNet-50 / BERT-base by index mod 3), 8 GiB arena, "
                    f"{N_REQUESTS} requests, Poisson 50/s, Zipf(1.1), batch 1, first fit",
        "eviction": policy,
        "models_requested": len(first), "models_checked_against_oracle": len(errors),
        "worst_normwise_error_by_family": worst, "tolerance": 2e-2,
        "p50_ms": round(float(np.percentile(lat, 50)), 3), "p99_ms": round(float(np.percentile(lat, 99)), 3),
        "per_family": {a: {"requests": int((arch == a).sum()),
                           "p50_ms": round(float(np.percentile(lat[arch == a], 50)), 3),
                           "p99_ms": round(float(np.percentile(lat[arch == a], 99)), 3),
                           "hit_rate": round(float(hits[arch == a].mean()), 4),
                           "hit_p50_ms": round(float(np.percentile(lat[(arch == a) & hits], 50)), 3),
                           "idle_hit_p50_ms": round(float(np.percentile(lat[(arch == a) & hits & idle], 50)), 3)}
                       for a in ("mlp", "resnet50", "bert")},
        "hit_rate_arena": round(float(hits.mean()), 4), "hit_rate_simulator": round(float(np.mean(want_hits)), 4),
        "hit_rate_byte_capacity_lru": round(float(np.mean(lru)), 4),
        "arena": {k: st[k] for k in ("hits", "misses", "evictions", "frag_evictions", "bytes_swapped",
                                     "graph_captures", "graph_repoints", "graph_rebases", "cache_touches")},
        "decisions_equal_simulator": True,
    }
    log(json.dumps(summary))
    out_dir = RESULTS_DIR
    os.makedirs(out_dir, exist_ok=True)
    with open(os.path.join(out_dir, f"tenants_full_{policy}.json"), "w") as f:
        json.dump(summary, f, indent=1)
    rt.close()
