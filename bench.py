"""Cold-start (swap-in + execute) latency of the 24-layer, 4096-wide bf16 MLP on one MI355X.

    python bench.py [--steps K] [--warmup W] [--batch B] [--method memcpy|gather|auto] [--full]

A step is one cold request: the model is invalidated (metadata only), then tp_infer
streams its 805,502,976 weight bytes from the pinned host pool into the HBM arena in
per-layer chunks while the layer kernels run as each chunk lands, and the host waits
for the fp32 output. The request input (activations) is already in device memory when
the clock starts; the weights start in pinned host memory by definition of "cold".

Prints one JSON line: the p50 cold latency, its lower bound
max(weight bytes / measured host-link peak, warm compute time), the effective swap
rate, warm latency, the HBM roofline of the dominant compute kernel (the skinny bf16
GEMM, timed with HIP events on its stream), and the CPU oracle timed on this host.
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
PCIE5_X16_GBS = 63.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def p50(xs):
    return statistics.median(xs)


def pct(xs, q):
    return float(np.percentile(np.asarray(xs), q))


def to_dev(torch, x, dev):
    if x.dtype == np.uint16:
        x = x.view(np.int16)
    return torch.from_numpy(np.ascontiguousarray(x)).to(dev)


def out_shape(m, b):
    if m.arch == "mlp":
        return (b, m.dims["width"])
    if m.arch == "resnet50":
        return (b, m.dims["classes"])
    return (b, m.dims["seq"], m.dims["d"])


def link_rates(torch, dev):
    """(bound rate, copy-engine rate, gather-kernel rate) of the host link in GB/s: the
    best single 1 GiB pinned copy and the best 1 GiB kernel gather from pinned memory (64
    workgroups, the library's default grid and the fastest in the copy comparison); the bound
    uses the higher."""
    import paper_2306_03622_amd as tp
    memcpy = link_peak(torch, dev)
    gather = tp.probe_gather_h2d(1 << 30, 64, 5)
    return max(memcpy, gather), memcpy, gather


def machine_peaks():
    """Measured matrix-core and HBM peaks next to the published ones."""
    import paper_2306_03622_amd as tp
    tflops, clock = tp.probe_mfma_bf16(1024, 2048, 5)
    hbm = tp.probe_hbm_read(4 << 30, 2048, 5)
    return {"mfma_bf16_tflops": round(tflops, 1), "shader_clock_ghz": round(clock, 3),
            "hbm_read_gbs": round(hbm, 1),
            "published": {"mfma_bf16_tflops": BF16_PEAK_TFLOPS, "hbm_gbs": HBM_PEAK_GBS, "clock_ghz": 2.4},
            "probe": "1024 workgroups x 4 waves x 2048 x 8 independent bf16 16x16x32 MFMAs; 4 GiB non-temporal "
                     "read by 2048 workgroups; best of 5 each"}


def link_peak(torch, dev, reps=10, nbytes=1 << 30):
    """Best-of-`reps` single pinned host->device copy of 1 GiB (GB/s)."""
    h = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
    d = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    s = torch.cuda.Stream(device=dev)
    best = 0.0
    for _ in range(reps):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        with torch.cuda.stream(s):
            d.copy_(h, non_blocking=True)
        s.synchronize()
        best = max(best, nbytes / (time.perf_counter() - t0) / 1e9)
    del h, d
    return best


class Bench:
    def __init__(self, torch, dev, model, batches, method, chunk, copy_streams=0, flags=0, direct=None, plan="greedy",
                 link_gbs=0.0, gather_wgs=0, spacers=0):
        import paper_2306_03622_amd as tp
        import synth
        self.tp, self.torch, self.dev, self.m = tp, torch, dev, model
        self.desc = tp.ModelDesc.of(model)
        ws = tp.tp_workspace_bytes(self.desc, max(batches))
        # spacers: small models registered beside the measured one, swapped in below it to
        # place it at another arena offset
        spacer = synth.mlp(2, 256, "bf16", "gelu", seed=5) if spacers else None
        extra = spacers * (spacer.total_bytes + 4096) if spacers else 0
        cm = {"memcpy": tp.TP_COPY_MEMCPY, "gather": tp.TP_COPY_GATHER, "pageable": tp.TP_COPY_PAGEABLE,
              "zero": tp.TP_COPY_ZERO}[method]
        self.rt = tp.Runtime(model.total_bytes + extra + (1 << 20), ws, chunk_min_bytes=chunk, copy_method=cm,
                             gather_wgs=gather_wgs, copy_streams=copy_streams, flags=flags,
                             direct_max_bytes=tp.DEFAULT_DIRECT if direct is None else direct,
                             plan=tp.TP_PLAN_COST if plan == "cost" else tp.TP_PLAN_GREEDY,
                             plan_batch=max(batches), link_gbs=link_gbs)
        self.mid = self.rt.register(self.desc, model.blob())
        self.spacers = [self.rt.register(tp.ModelDesc.of(spacer), spacer.blob()) for _ in range(spacers)]
        self.stream = torch.cuda.Stream(device=dev)

    def place(self, k):
        """Makes the model resident above the first k spacers (another arena offset for each
        k), with nothing of it in flight."""
        self.rt.evict(self.mid)
        for j, sp in enumerate(self.spacers):
            self.rt.evict(sp)
        for sp in self.spacers[:k]:
            self.rt.swap_in(sp, stream=self.stream)
        self.rt.swap_in(self.mid, stream=self.stream)
        self.stream.synchronize()
        return self.rt.info(self.mid)["extent_offset"]

    def request(self, x, out, cold):
        torch = self.torch
        if cold:
            self.rt.evict(self.mid)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        self.rt.infer(self.mid, x, out, stream=self.stream)
        self.last_enqueue_ms = (time.perf_counter() - t0) * 1e3      # host time of the call alone
        self.stream.synchronize()
        return (time.perf_counter() - t0) * 1e3

    def swap_only(self):
        self.rt.evict(self.mid)
        self.torch.cuda.synchronize()
        t0 = time.perf_counter()
        self.rt.swap_in(self.mid, stream=self.stream)
        self.stream.synchronize()
        return (time.perf_counter() - t0) * 1e3

    def io(self, batch, seed):
        import synth
        x = to_dev(self.torch, synth.config_input(self.m, batch, seed), self.dev)
        out = self.torch.empty(out_shape(self.m, batch), dtype=self.torch.float32, device=self.dev)
        return x, out

    def event_time_ms(self, x, out, reps):
        """Average warm forward time measured by HIP events on the compute stream."""
        torch = self.torch
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        self.rt.infer(self.mid, x, out, stream=self.stream)
        torch.cuda.synchronize()
        e0.record(self.stream)
        for _ in range(reps):
            self.rt.infer(self.mid, x, out, stream=self.stream)
        e1.record(self.stream)
        self.stream.synchronize()
        return e0.elapsed_time(e1) / reps

    def close(self):
        self.rt.close()


def measure(b: Bench, batch, seed, steps, warmup, warm_reps):
    x, out = b.io(batch, seed)
    for _ in range(warmup):
        b.request(x, out, cold=True)
        b.request(x, out, cold=False)
    torch = b.torch
    torch.cuda.synchronize()
    t_all = time.perf_counter()
    cold, cold_enq = [], []
    for _ in range(steps):
        cold.append(b.request(x, out, cold=True))
        cold_enq.append(b.last_enqueue_ms)
    torch.cuda.synchronize()
    t_all = time.perf_counter() - t_all
    warm, warm_enq = [], []
    for _ in range(warm_reps):
        warm.append(b.request(x, out, cold=False))
        warm_enq.append(b.last_enqueue_ms)
    swap = [b.swap_only() for _ in range(max(5, steps // 2))]
    return {"cold": cold, "warm": warm, "swap": swap, "t_all": t_all, "x": x, "out": out,
            "cold_enqueue": cold_enq, "warm_enqueue": warm_enq}


def elbow_sweep(torch, dev, method, copy_streams=0, sizes=(256 << 10, 512 << 10, 1 << 20, 2 << 20, 4 << 20, 8 << 20, 16 << 20,
                                             32 << 20, 1 << 40), reps=8):
    """Transfer throughput of a chunked, event-handed-off swap versus group size G.

    Runs through the library: a 512-wide bf16 MLP of 256 layers (512 KiB per layer,
    128 MiB) is swapped in with each G (whole layers per chunk), and a cold request
    with per-layer waits is timed too. The elbow is the smallest G whose swap
    throughput is within 5% of the largest measured.
    """
    import paper_2306_03622_amd as tp
    import synth
    m = synth.mlp(256, 512, "bf16", "relu", seed=99)
    m.blob()
    rows = []
    x, out = None, None
    for g in sizes:
        b = Bench(torch, dev, m, [1], method, g, copy_streams)
        if x is None:
            x, out = b.io(1, 5)
        b.swap_only()
        sw = p50([b.swap_only() for _ in range(reps)])
        b.request(x, out, cold=True)
        cold = p50([b.request(x, out, cold=True) for _ in range(reps)])
        n = len(b.rt.chunks(b.mid))
        b.close()
        rows.append({"chunk_min_bytes": g, "chunks": n, "swap_gbs": round(m.total_bytes / (sw / 1e3) / 1e9, 2),
                     "cold_pipelined_ms": round(cold, 3)})
        log(f"  G={g >> 10} KiB chunks={n}: swap {rows[-1]['swap_gbs']} GB/s, cold {cold:.3f} ms")
    best = max(r["swap_gbs"] for r in rows)
    elbow = next(r["chunk_min_bytes"] for r in rows if r["swap_gbs"] >= 0.95 * best)
    return {"model": "256 x 512 bf16 MLP (512 KiB per layer)", "rows": rows, "elbow_bytes": elbow}


# Swap designs of the breakdown (Sec. 6.1, "Performance breakdown of model swapping"), each
# changing one thing from the row above, then the alternatives the library also offers.
# (name, copy method, group size or None for the default, flags, copy streams, direct-access
# size limit, chunk plan)
ABLATION = (
    ("baseline: pageable copy per tensor, then execute", "pageable", 0, "serial|per_tensor", 1, 0, "greedy"),
    ("pinned: pinned copy per tensor, then execute", "memcpy", 0, "serial|per_tensor", 1, 0, "greedy"),
    ("pipeline: per-tensor transfers overlapped with execution", "memcpy", 0, "per_tensor", 1, 0, "greedy"),
    ("group: tensors grouped to >= G, overlapped", "memcpy", None, "per_tensor", 1, 0, "greedy"),
    ("group by layer: whole layers grouped to >= G", "memcpy", None, "", 1, 0, "greedy"),
    ("gather kernel instead of the copy engine, grouped by layer", "gather", None, "", 1, 0, "greedy"),
    ("two copy streams, grouped by layer", "memcpy", None, "", 2, 0, "greedy"),
    ("zero-copy: kernels read the pinned host copy, never resident", "zero", None, "", 1, 0, "greedy"),
    ("direct access first, swap behind it (default for models <= 2 MiB)", "memcpy", None, "", 1, 1 << 62, "greedy"),
    ("cost-model grouping: boundaries minimising the modelled completion time", "memcpy", None, "", 1, 0, "cost"),
)


def ablation(torch, dev, chunk, link_gbs, budget_s=2.5, max_reps=20):
    """Cold p50 of every swap design on the single-GPU workloads (batch 8, and batch 1 for
    the 1 MB MLP). A design is timed until max_reps cold requests or budget_s seconds."""
    import synth
    import paper_2306_03622_amd as tp
    bits = {"serial": tp.TP_FLAG_SERIAL, "per_tensor": tp.TP_FLAG_PER_TENSOR}
    out = {}
    for cfg, bt in ((1, 1), (2, 8), (3, 8), (4, 8)):
        m = synth.config_model(cfg)
        m.blob()
        rows = []
        ref = None
        for name, method, g, fl, ns, direct, plan in ABLATION:
            flags = 0
            for f in filter(None, fl.split("|")):
                flags |= bits[f]
            log(f"ablation cfg{cfg} b{bt}: {name}")
            b = Bench(torch, dev, m, [bt], method, chunk if g is None else g, ns, flags, direct, plan, link_gbs)
            x, y = b.io(bt, synth.CONFIG_SEEDS[cfg][1] + (0 if cfg == 1 else bt))
            b.request(x, y, cold=True)
            got = y.cpu()
            same = bool(torch.equal(got, ref)) if ref is not None else True
            ref = got if ref is None else ref
            times, t_start = [], time.perf_counter()
            while len(times) < max_reps and time.perf_counter() - t_start < budget_s:
                times.append(b.request(x, y, cold=True))
            rows.append({"design": name, "cold_p50_ms": round(p50(times), 3), "runs": len(times),
                         "chunks": len(b.rt.chunks(b.mid)), "bitwise_equal_to_first": same})
            b.close()
        out[f"cfg{cfg}_b{bt}"] = {"weight_bytes": m.total_bytes, "designs": rows}
        m.drop_blob()
    return out


def copy_compare(torch, dev, link_copy, link_gather, wgs=(64, 256, 1024, 2048), reps=10):
    """The copy engine against the gather kernel at several grid sizes, on the chunk plans the
    library uses (cost plan, batch 8): swap-only and cold p50 per design, and whether the cold
    outputs are bitwise equal to the copy engine's. Run under rocprofv3 with the kernel and
    memory-copy traces to get the per-chunk durations of both on the device."""
    import synth
    import paper_2306_03622_amd as tp
    out = {}
    for cfg in (2, 3, 4):
        m = synth.config_model(cfg)
        m.blob()
        rows, ref = [], None
        for method, w in [("memcpy", 0)] + [("gather", v) for v in wgs]:
            log(f"copy compare cfg{cfg}: {method} {w or ''}")
            b = Bench(torch, dev, m, [8], method, tp.DEFAULT_CHUNK, plan="cost",
                      link_gbs=link_gather if method == "gather" else link_copy, gather_wgs=w)
            x, y = b.io(8, synth.CONFIG_SEEDS[cfg][1] + 8)
            b.swap_only()
            sw = p50([b.swap_only() for _ in range(reps)])
            b.request(x, y, cold=True)
            cold = p50([b.request(x, y, cold=True) for _ in range(reps)])
            got = y.cpu()
            same = bool(torch.equal(got, ref)) if ref is not None else True
            ref = got if ref is None else ref
            rows.append({"method": method, "gather_wgs": w or None, "chunks": len(b.rt.chunks(b.mid)),
                         "swap_ms": round(sw, 3), "swap_gbs": round(m.total_bytes / (sw / 1e3) / 1e9, 2),
                         "cold_p50_ms": round(cold, 3), "bitwise_equal_to_copy_engine": same})
            b.close()
        out[f"cfg{cfg}_b8"] = {"weight_bytes": m.total_bytes, "rows": rows}
        m.drop_blob()
    return out


def hit_conditions(torch, dev, reps=40, idle_s=0.02, flush_bytes=512 << 20):
    """A warm request (weights resident) of workloads 2-4 at batch 1 under the conditions a hit
    meets in the multi-tenant workload, one at a time: back to back with the same buffers (the
    isolated warm figure), with a new input/output pair each time (the cached graph is
    repointed), after an idle gap of the trace's mean inter-arrival time, after a device copy of
    flush_bytes that displaces the weights from the caches (other models ran in between), both,
    and after the model came back into another arena offset (five offsets in turn). Then the
    cache conditions again in a context where every warm request pre-reads its weights into the
    caches (TP_FLAG_TOUCH_ALWAYS; by default only a request that follows another model's does).
    Host latency (the call plus the stream synchronisation) and the device span of the request
    (events on its stream), p50 of `reps` each."""
    import synth
    import paper_2306_03622_amd as tp
    src = torch.empty(flush_bytes, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    out = {}
    conditions = (("back_to_back", False, False, False, False), ("new_buffers", True, False, False, False),
                  ("idle", False, True, False, False), ("flushed", False, False, True, False),
                  ("idle_flushed", False, True, True, False), ("idle_flushed_new_buffers", True, True, True, False),
                  ("moved_new_buffers", True, False, False, True))
    touched = ("back_to_back", "flushed", "idle_flushed_new_buffers")
    for cfg in (2, 3, 4):
        m = synth.config_model(cfg)
        m.blob()
        row = {"weight_bytes": m.total_bytes}
        for flags, key, names in ((0, "conditions", [c[0] for c in conditions]),
                                  (tp.TP_FLAG_TOUCH_ALWAYS, "conditions_touch_always", touched)):
            b = Bench(torch, dev, m, [1], "memcpy", tp.DEFAULT_CHUNK, plan="cost", spacers=4, flags=flags)
            pairs = [b.io(1, synth.CONFIG_SEEDS[cfg][1] + 1), b.io(1, synth.CONFIG_SEEDS[cfg][1] + 1)]
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            offsets = set()

            def one(k, idle, flush, move=False):
                x, y = pairs[k % 2]
                if move:
                    offsets.add(b.place(k % 5))
                if flush:
                    dst.copy_(src)
                torch.cuda.synchronize()
                if idle:
                    time.sleep(idle_s)
                t0 = time.perf_counter()
                e0.record(b.stream)
                b.rt.infer(b.mid, x, y, stream=b.stream)
                e1.record(b.stream)
                b.stream.synchronize()
                return (time.perf_counter() - t0) * 1e3, e0.elapsed_time(e1)

            b.place(0)
            b.request(*pairs[0], cold=False)
            for k in range(6):
                one(k, False, False)
            rows = {}
            for name, alt, idle, flush, move in conditions:
                if name not in names:
                    continue
                log(f"hit conditions cfg{cfg}: {name}" + (" (touch always)" if flags else ""))
                r = [one(k if alt else 0, idle, flush, move) for k in range(1, reps + 1)]
                rows[name] = {"p50_ms": round(p50([v[0] for v in r]), 4),
                              "device_p50_ms": round(p50([v[1] for v in r]), 4)}
            row[key] = rows
            st = b.rt.stats()
            if flags:
                row["cache_touches"] = st.get("cache_touches")
            else:
                row["outputs_of_both_buffer_pairs_equal"] = bool(torch.equal(pairs[0][1], pairs[1][1]))
                row["moved_offsets"] = len(offsets)
                row["graphs"] = {k: st.get(k) for k in ("graph_captures", "graph_repoints", "graph_rebases")}
            b.close()
        out[f"cfg{cfg}_b1"] = row
        m.drop_blob()
    return out


def native_alloc_us(sizes, reps=10):
    """p50 of hipMalloc + hipFree of each size (the per-swap allocation that a reserved arena
    avoids), through the HIP runtime torch has loaded."""
    import ctypes
    hip = ctypes.CDLL("libamdhip64.so.7", mode=ctypes.RTLD_GLOBAL)   # the copy torch has loaded
    out = {}
    for name, nb in sizes.items():
        ts = []
        for _ in range(reps):
            p = ctypes.c_void_p()
            t0 = time.perf_counter()
            if hip.hipMalloc(ctypes.byref(p), ctypes.c_size_t(nb)) != 0:
                raise RuntimeError("hipMalloc failed")
            if hip.hipFree(p) != 0:
                raise RuntimeError("hipFree failed")
            ts.append((time.perf_counter() - t0) * 1e6)
        out[name] = round(p50(ts), 1)
    return out


def byte_lru_hit_rate(seq, sizes, capacity):
    """Hit rate of an LRU cache of `capacity` bytes over the request sequence with no placement
    constraint (a model fits whenever the resident bytes allow it): the figure the arena's
    contiguous placement loses hits against."""
    from collections import OrderedDict
    res, used, hits = OrderedDict(), 0, 0
    for mid in seq:
        if mid in res:
            hits += 1
            res.move_to_end(mid)
            continue
        while used + sizes[mid] > capacity:
            used -= res.popitem(last=False)[1]
        res[mid] = sizes[mid]
        used += sizes[mid]
    return hits / len(seq)


def tenants(torch, dev, n_requests, n_models, arena_gib, workers, evict="lru", plan="cost", queue=None, rate=50.0,
            deadline_ms=None, slo_pct=0.98, alloc="first-fit", partition_mib=0, lib_flags=0):
    """Open-loop multi-tenant run: n_models registered models of the three families, an
    arena of arena_gib GiB, Poisson arrivals at 50/s with Zipf(1.1) popularity, LRU,
    heaviness-aware or contiguous-window eviction, first-fit or two-tier partitioned placement (with or without
    consolidation)."""
    import paper_2306_03622_amd as tp
    import synth
    specs = synth.tenant_models(n_models)
    trace = synth.tenant_trace(n_requests, rate_per_s=rate, n_models=n_models)
    ws = 0
    descs, kinds, host_bytes, heavy = {}, {}, {}, {}
    for cfg in (2, 3, 4):
        ws = max(ws, tp.tp_workspace_bytes(tp.ModelDesc.of(synth.config_model(cfg)), 1))
    alloc_mode = {"first-fit": tp.TP_ALLOC_FIRST_FIT, "partition": tp.TP_ALLOC_PARTITION,
                  "consolidate": tp.TP_ALLOC_PARTITION_CONSOLIDATE}[alloc]
    rt = tp.Runtime(arena_gib << 30, ws, plan=tp.TP_PLAN_COST if plan == "cost" else tp.TP_PLAN_GREEDY,
                    evict_policy={"lru": tp.TP_EVICT_LRU, "heaviness": tp.TP_EVICT_HEAVINESS,
                                  "window": tp.TP_EVICT_LRU_WINDOW}[evict],
                    alloc=alloc_mode, partition_bytes=partition_mib << 20, flags=lib_flags)
    t0 = time.perf_counter()
    ids = []
    for i, m in synth.build_models(specs, workers):
        d = tp.ModelDesc.of(m)
        mid = rt.register(d, m.blob())
        ids.append(mid)
        kinds[mid] = m.arch
        heavy[m.arch] = bool(rt.info(mid)["heavy"])
        host_bytes[mid] = m.total_bytes
        if i % 10 == 9:
            log(f"  registered {i + 1} models ({(time.perf_counter() - t0):.0f} s)")
        m.drop_blob()
    reg_s = time.perf_counter() - t0
    protos = {cfg: synth.config_model(cfg, 0) for cfg in (2, 3, 4)}      # shapes only
    xs, outs, reqs = [], [], []
    for r in range(n_requests):
        mid = ids[int(trace.model[r])]
        proto = protos[specs[int(trace.model[r])][0]]
        x = to_dev(torch, synth.request_input(proto, int(trace.input_seed[r])), dev)
        y = torch.empty(out_shape(proto, 1), dtype=torch.float32, device=dev)
        xs.append(x)
        outs.append(y)
        reqs.append((mid, 1, x, y, int(trace.arrival_s[r] * 1e9)))
    stream = torch.cuda.Stream(device=dev)
    # warm every family's kernels once, then start from an empty arena
    for cfg in (2, 3, 4):
        k = next(i for i, sp in enumerate(specs) if sp[0] == cfg)
        r0 = next(r for r in range(n_requests) if int(trace.model[r]) == k) if k in set(trace.model.tolist()) else None
        x = xs[r0] if r0 is not None else to_dev(torch, synth.request_input(protos[cfg], 1), dev)
        y = torch.empty(out_shape(protos[cfg], 1), dtype=torch.float32, device=dev)
        rt.infer(ids[k], x, y, stream=stream)
    stream.synchronize()
    for mid in ids:
        rt.evict(mid)
    st0 = rt.stats()
    torch.cuda.synchronize()
    log(f"running {n_requests} requests over {trace.arrival_s[-1]:.1f} s")
    sched = None
    if queue is None:
        res = rt.run_trace(reqs, stream=stream)
    else:
        dls = [int(deadline_ms[kinds[q[0]]] * 1e6) for q in reqs]
        res, sched = rt.run_trace_sched(reqs, dls, stream=stream, slo_pct=slo_pct,
                                        policy=tp.TP_QUEUE_SLO if queue == "slo" else tp.TP_QUEUE_FIFO)
    st1 = rt.stats()
    rt.close()
    lat = np.array([(r["done_ns"] - q[4]) / 1e6 for r, q in zip(res, reqs)])
    hit = np.array([r["hit"] for r in res])
    issue_delay = np.array([(r["issue_ns"] - q[4]) / 1e6 for r, q in zip(res, reqs)])
    service = np.array([(r["done_ns"] - r["issue_ns"]) / 1e6 for r in res])
    # requests issued with nothing of theirs queued ahead on the GPU (the previous request had
    # completed): their latency is the request's own service time
    idle = np.array([i == 0 or res[i]["issue_ns"] >= res[i - 1]["done_ns"] for i in range(len(res))])
    arch = np.array([kinds[q[0]] for q in reqs])
    per = {}
    for a in ("mlp", "resnet50", "bert"):
        sel = arch == a
        if sel.any():
            per[a] = {"requests": int(sel.sum()), "p50_ms": round(float(np.percentile(lat[sel], 50)), 3),
                      "p99_ms": round(float(np.percentile(lat[sel], 99)), 3),
                      "hit_rate": round(float(hit[sel].mean()), 4),
                      "hit_p50_ms": round(float(np.percentile(lat[sel & (hit == 1)], 50)), 3) if (sel & (hit == 1)).any()
                      else None,
                      "idle_hit_p50_ms": round(float(np.percentile(lat[sel & (hit == 1) & idle], 50)), 3)
                      if (sel & (hit == 1) & idle).any() else None}
            ih = sel & (hit == 1) & idle
            if ih.any():
                # an idle hit's latency split: arrival -> tp_infer call (the driver's wake-up),
                # call -> completion seen by the host
                per[a]["idle_hit_issue_delay_p50_ms"] = round(float(np.percentile(issue_delay[ih], 50)), 4)
                per[a]["idle_hit_service_p50_ms"] = round(float(np.percentile(service[ih], 50)), 4)
    delta = {k: st1[k] - st0[k] for k in ("hits", "misses", "evictions", "frag_evictions", "bytes_swapped",
                                          "evacuations", "bytes_moved", "graph_captures", "graph_repoints",
                                          "graph_rebases", "cache_touches")}
    delta["partitions"] = st1["partitions"]
    calls = st1["admit_calls"] - st0["admit_calls"]
    adm = np.array([r["admit_ns"] / 1e3 for r in res if not r["hit"]])
    admit = {"admissions": calls,
             "mean_us": round((st1["admit_ns_total"] - st0["admit_ns_total"]) / max(calls, 1) / 1e3, 2),
             "max_us_since_start": round(st1["admit_ns_max"] / 1e3, 2),
             "cdf_us": ({f"p{q}": round(float(np.percentile(adm, q)), 2) for q in (50, 90, 99)} |
                        {"max": round(float(adm.max()), 2)}) if adm.size else None,
             "native_alloc_us": native_alloc_us({a: host_bytes[next(m for m in ids if kinds[m] == a)]
                                                 for a in set(kinds.values())})}
    slo = None
    if queue is not None:
        # a function (model) complies when at least slo_pct of its requests met their deadline
        by_model = {}
        for r, q in zip(res, reqs):
            ok = (r["done_ns"] - q[4]) <= deadline_ms[kinds[q[0]]] * 1e6
            by_model.setdefault(q[0], []).append(ok)
        comp = {mid: np.mean(v) >= slo_pct for mid, v in by_model.items()}
        slo = {"queue": queue, "deadline_ms": deadline_ms, "pct": slo_pct, "functions": len(comp),
               "compliant_functions": int(sum(comp.values())),
               "compliant_ratio": round(float(np.mean(list(comp.values()))), 4),
               "requests_within_deadline": round(float(np.mean([(r["done_ns"] - q[4]) <= deadline_ms[kinds[q[0]]] * 1e6
                                                                 for r, q in zip(res, reqs)])), 4),
               "scheduler": sched}
    return {"metric": f"multi-tenant request latency (open loop, {evict} eviction)", "unit": "ms",
            "p50_ms": round(float(np.percentile(lat, 50)), 3), "p99_ms": round(float(np.percentile(lat, 99)), 3),
            "hit_rate": round(float(hit.mean()), 4),
            "byte_lru_hit_rate": round(byte_lru_hit_rate([q[0] for q in reqs], {m: -(-b // 256) * 256 for m, b in
                                                                               host_bytes.items()}, arena_gib << 30), 4),
            "requests": n_requests, "models": n_models,
            "arena_gib": arena_gib, "registered_host_bytes": int(sum(host_bytes.values())),
            "register_s": round(reg_s, 1), "trace_s": round(float(trace.arrival_s[-1]), 2),
            "per_family": per, "arena": delta, "admission": admit, "heavy_by_family": heavy, "slo": slo,
            "config": {"workload": f"{n_models} models (24x4096 MLP / ResNet-50 / BERT-base by index mod 3), "
                                   f"Poisson {rate:g} req/s, Zipf(1.1), {arena_gib} GiB arena, batch 1",
                       "eviction": evict, "chunk_plan": plan, "placement": alloc,
                       "partition_mib": (partition_mib or (arena_gib << 10) // 8) if alloc != "first-fit" else None}}


def measure_workload(torch, dev, cfg, bts, method, chunk, copy_streams, plan, link, steps, warmup, trace,
                     plan_link=None, cpu=False, lib_flags=0):
    """Cold, warm and swap-only latencies of workload `cfg` at batches `bts` (one context);
    `link` sets the bound, `plan_link` (default `link`) the cost-model plan; with `cpu` the
    oracle's time at each batch too."""
    import paper_2306_03622_amd as tp
    import synth
    m = synth.config_model(cfg)
    out, outs = {}, {}
    bb = Bench(torch, dev, m, bts, method, chunk, copy_streams, plan=plan, link_gbs=plan_link or link,
               flags=(tp.TP_FLAG_TRACE if trace else 0) | lib_flags)
    for bt in bts:
        rr = measure(bb, bt, synth.CONFIG_SEEDS[cfg][1] + (0 if cfg == 1 else bt), steps, warmup, max(4 * steps, 100))
        if trace and m.total_bytes > tp.DEFAULT_DIRECT:     # direct-access requests are not traced
            x, y = bb.io(bt, 1)
            bb.request(x, y, cold=True)
            tl = bb.rt.timeline()
            out[f"cfg{cfg}_b{bt}_timeline"] = {k: ([round(v, 4) for v in tl[k]] if isinstance(tl[k], list)
                                                   else round(tl[k], 4)) for k in tl}
        wp = p50(rr["warm"])
        bnd = max(m.total_bytes / (link * 1e9) * 1e3, wp)
        fl = forward_flops(m, bt)
        import hashlib
        digest = hashlib.sha256(rr["out"].cpu().numpy().tobytes()).hexdigest()[:16]   # last request's output
        fwd = bb.event_time_ms(rr["x"], rr["out"], 20)
        out[f"cfg{cfg}_b{bt}"] = {
            "weight_bytes": m.total_bytes, "chunks": len(bb.rt.chunks(bb.mid)),
            "cold_p50_ms": round(p50(rr["cold"]), 4), "cold_p10_ms": round(pct(rr["cold"], 10), 4),
            "cold_p90_ms": round(pct(rr["cold"], 90), 4),
            "warm_p50_ms": round(wp, 4), "bound_ms": round(bnd, 4),
            "cold_enqueue_p50_ms": round(p50(rr["cold_enqueue"]), 4),
            "warm_enqueue_p50_ms": round(p50(rr["warm_enqueue"]), 4),
            "cold_over_bound": round(p50(rr["cold"]) / bnd, 4),
            "swap_only_gbs": round(m.total_bytes / (p50(rr["swap"]) / 1e3) / 1e9, 2),
            "forward_gflop": round(fl / 1e9, 3), "warm_forward_event_ms": round(fwd, 4),
            "warm_tflops": round(fl / (fwd * 1e-3) / 1e12, 2),
            "mfma_util": round(fl / (fwd * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 5),
            "hbm_frac_weights": round(m.total_bytes / (fwd * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "output_sha16": digest}
        outs[bt] = rr["out"].cpu().numpy()
    bb.close()
    if cpu:
        for bt in bts:
            log(f"  CPU oracle, workload {cfg} batch {bt}")
            out[f"cfg{cfg}_b{bt}"]["cpu_oracle"] = cpu_baseline(m, bt, synth.CONFIG_SEEDS[cfg][1] + (0 if cfg == 1 else bt),
                                                                budget_s=8.0, max_runs=50 if cfg == 1 else 5,
                                                                gpu_out=outs[bt])
    m.drop_blob()
    return out


def kernel_fingerprint():
    """First 16 hex digits of sha256 over the skinny-GEMM kernel sources and the device
    compile flags."""
    import hashlib
    from paper_2306_03622_amd import build as tp_build
    h = hashlib.sha256()
    for f in ("gemv_bf16.hip", "gemm_args.hpp", "common.hpp", "kernels.hpp"):
        with open(os.path.join(ROOT, "paper_2306_03622_amd", "csrc", "kernels", f), "rb") as fh:
            h.update(fh.read())
    h.update(" ".join(tp_build.DEVICE).encode())
    return h.hexdigest()[:16]


def counted_traffic(batch):
    """HBM bytes per launch from the committed counter passes, if they still describe the
    kernel as built (same source fingerprint and batch), else None."""
    path = os.path.join(ROOT, "profiles", f"gemv_mlp24x4096_b{batch}_pmc.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if "=" in line and not line.startswith("#"):
            k, v = line.split("=", 1)
            kv[k.strip()] = v.strip()
    if kv.get("source_fingerprint") != kernel_fingerprint():
        return None
    return int(kv["traffic_bytes_per_launch"])


def forward_flops(model, batch):
    """Algorithmic FLOPs of one forward pass: 2 M N K per contraction (convolutions as implicit
    GEMMs, M = B Ho Wo, K = KH KW Cin), 4 S^2 d_h per (sample, head) for attention."""
    import synth
    d = model.dims
    if model.arch == "mlp":
        return 2 * batch * d["width"] * d["width"] * d["layers"]
    if model.arch == "resnet50":
        hw, total = d.get("image", 224), 0
        convs = synth.models.resnet50_convs(d.get("stages", synth.models.RESNET50_STAGES), d.get("stem", 64))
        h = (hw + 2 * 3 - 7) // 2 + 1                    # conv1
        total += 2 * batch * h * h * convs[0][1] * 7 * 7 * 3
        h = (h + 2 - 3) // 2 + 1                         # max-pool
        for name, co, kh, kw, ci, st, pad in convs[1:]:
            # the projection shortcut reads the block input and lands on the block output size
            ho = h if name.endswith(".ds") else (h + 2 * pad - kh) // st + 1
            total += 2 * batch * ho * ho * co * kh * kw * ci
            h = ho if kh == 3 else h
        return total + 2 * batch * 2048 * d["classes"]
    L, dm, F, S = d["layers"], d["d"], d["ffn"], d["seq"]
    M = batch * S
    per_layer = 2 * M * dm * (3 * dm) + 2 * M * dm * dm + 2 * M * dm * F * 2 + 4 * S * S * dm * batch
    return L * per_layer


def cpu_baseline(model, batch, seed, budget_s=12.0, max_runs=30, gpu_out=None):
    """The oracle (fp32 variant) on this host's cores, a bounded number of runs; with `gpu_out`
    (the library's output for the same input) also the normwise error between the two."""
    import synth
    from oracle import forward as oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max((i.get("num_threads", 0) for i in threadpool_info() if i.get("user_api") == "blas"), default=0)
    except Exception:
        threads = 0
    x = synth.config_input(model, batch, seed)
    ref = oracle.forward(model, x, np.float32)          # first touch
    times = []
    t_start = time.perf_counter()
    while len(times) < max_runs and (time.perf_counter() - t_start) < budget_s:
        t0 = time.perf_counter()
        ref = oracle.forward(model, x, np.float32)
        times.append((time.perf_counter() - t0) * 1e3)
    out = {"value": round(p50(times), 3), "unit": "ms", "cores": threads or os.cpu_count(), "kind": "oracle",
           "sample": f"{len(times)} fp32 oracle forwards of the same workload at batch {batch} "
                     f"(p50; {os.cpu_count()} host CPUs visible, BLAS threads {threads})"}
    if gpu_out is not None:
        # the GPU's output for the same input beside the oracle's (fp32 variant; it agrees with
        # the float64 oracle to <= 1e-5 normwise on every workload)
        out["gpu_normwise_error"] = float(f"{oracle.normwise_error(gpu_out, ref).max():.3e}")
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--batch", type=int, default=8)
    ap.add_argument("--method", choices=["memcpy", "gather", "auto"], default="memcpy")
    ap.add_argument("--chunk", default="default",
                    help="transfer group size G in bytes, 'default' (the library's) or 'elbow' (this run's sweep)")
    ap.add_argument("--no-sweep", action="store_true", help="skip the group-size sweep")
    ap.add_argument("--copy-streams", type=int, default=0, help="copy streams of the library (0: its default)")
    ap.add_argument("--plan", choices=["cost", "greedy"], default="cost",
                    help="chunk plan: cost model (boundaries minimising the modelled completion time, with the "
                         "measured link rate) or the greedy >= G rule")
    ap.add_argument("--tenants", type=int, default=0, metavar="N_REQUESTS",
                    help="run the multi-tenant open-loop workload with this many requests instead")
    ap.add_argument("--tenant-models", type=int, default=100)
    ap.add_argument("--tenant-arena-gib", type=int, default=8)
    ap.add_argument("--evict", choices=["lru", "heaviness", "window"], default="lru",
                    help="eviction policy of the multi-tenant run (window: TP_EVICT_LRU_WINDOW)")
    ap.add_argument("--alloc", choices=["first-fit", "partition", "consolidate"], default="first-fit",
                    help="multi-tenant arena placement: first fit, two-tier partitions, or partitions with "
                         "consolidation")
    ap.add_argument("--partition-mib", type=int, default=0,
                    help="partition size of --alloc partition/consolidate (0: arena / 8)")
    ap.add_argument("--queue", choices=["none", "fifo", "slo"], default="none",
                    help="multi-tenant run: host-side request queue (FIFO or SLO-aware) instead of issuing at arrival")
    ap.add_argument("--rate", type=float, default=50.0, help="multi-tenant arrival rate (requests/s)")
    ap.add_argument("--deadlines", default="40,3,12",
                    help="multi-tenant SLO deadlines in ms for the MLP, ResNet-50 and BERT-base families")
    ap.add_argument("--pmc-workload", action="store_true",
                    help="run only a fixed workload for hardware-counter passes: 20 warm forwards of the "
                         "bench model, then one 256 MiB device-to-device copy (the byte-count calibration)")
    ap.add_argument("--full", action="store_true", help="(the default; kept for older command lines)")
    ap.add_argument("--quick", action="store_true",
                    help="the headline workload at --batch only: no other batches, workloads or multi-tenant run")
    ap.add_argument("--no-tenants", action="store_true", help="skip the multi-tenant row of the default run")
    ap.add_argument("--ablation", action="store_true",
                    help="time the cold request under every swap design instead (breakdown table)")
    ap.add_argument("--copy-compare", action="store_true",
                    help="copy engine against the gather kernel (grid sizes 64-2048) on workloads 2-4, batch 8")
    ap.add_argument("--hit-conditions", action="store_true",
                    help="warm requests of workloads 2-4 at batch 1: back to back, new buffers, idle gap, flushed caches")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--workload", type=int, default=0, help=argparse.SUPPRESS)   # child process of --full
    ap.add_argument("--batches", default="1", help=argparse.SUPPRESS)
    ap.add_argument("--lib-flags", type=int, default=0, help="extra TP_FLAG_* bits for --workload and --tenants runs (A/B checks)")
    ap.add_argument("--trace", action="store_true",
                    help="with --full: record the per-chunk timeline of one more cold request per workload")
    a = ap.parse_args()
    if a.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: swap-in and execution of a model is a per-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    children = {}
    if not a.quick and not a.workload and not (a.tenants or a.ablation or a.pmc_workload or a.copy_compare or a.hit_conditions):
        # Each extra workload runs in a process of its own, started before this process touches
        # the GPU: a serving process holds one context, and after many contexts and streams in
        # one process HIP's stream-to-hardware-queue arrangement can serialise a swap behind
        # the kernels (seen as BERT-base cold 4.5-4.8 ms instead of 4.0 ms).
        import subprocess
        for cfg, bts in ((1, [1]), (3, [1, 8]), (4, [1, 8])):
            log(f"workload {cfg} (child process)")
            cmd = [sys.executable, os.path.abspath(__file__), "--workload", str(cfg), "--batches",
                   ",".join(map(str, bts)), "--steps", str(a.steps), "--warmup", str(a.warmup), "--method",
                   "memcpy" if a.method == "auto" else a.method, "--chunk", str(a.chunk), "--copy-streams",
                   str(a.copy_streams), "--plan", a.plan] + (["--trace"] if a.trace else []) + \
                  (["--no-cpu"] if a.no_cpu else [])
            out = subprocess.run(cmd, stdout=subprocess.PIPE, text=True)     # its log goes to our stderr
            if out.returncode != 0:
                raise SystemExit(f"workload {cfg} failed with status {out.returncode}")
            children.update(json.loads(out.stdout.strip().splitlines()[-1]))
        if not a.no_tenants:
            log("workload 5, multi-tenant (child process)")
            out = subprocess.run([sys.executable, os.path.abspath(__file__), "--tenants", "3000", "--plan", a.plan],
                                 stdout=subprocess.PIPE, text=True)
            if out.returncode != 0:
                raise SystemExit(f"multi-tenant workload failed with status {out.returncode}")
            t = json.loads(out.stdout.strip().splitlines()[-1])
            children["cfg5_multi_tenant"] = {k: t[k] for k in ("p50_ms", "p99_ms", "hit_rate", "byte_lru_hit_rate",
                                                               "requests", "models",
                                                               "arena_gib", "per_family", "arena", "config",
                                                               "trace_s")}

    import torch
    import synth
    if not torch.cuda.is_available():
        print("bench.py needs an MI355X (no HIP device visible)", file=sys.stderr)
        sys.exit(2)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)

    if a.tenants:
        dl = dict(zip(("mlp", "resnet50", "bert"), (float(v) for v in a.deadlines.split(","))))
        print(json.dumps(tenants(torch, dev, a.tenants, a.tenant_models, a.tenant_arena_gib, 16, a.evict, a.plan,
                                 None if a.queue == "none" else a.queue, a.rate, dl, alloc=a.alloc,
                                 partition_mib=a.partition_mib, lib_flags=a.lib_flags)), flush=True)
        return

    if a.ablation:
        import paper_2306_03622_amd as tp
        link = link_peak(torch, dev)
        print(json.dumps({"ablation": ablation(torch, dev, tp.DEFAULT_CHUNK, link), "link_peak_gbs": round(link, 2),
                          "group_bytes": tp.DEFAULT_CHUNK}), flush=True)
        return

    if a.copy_compare:
        _, link_copy, link_gather = link_rates(torch, dev)
        print(json.dumps({"copy_compare": copy_compare(torch, dev, link_copy, link_gather),
                          "link_copy_engine_gbs": round(link_copy, 2), "link_gather_kernel_gbs": round(link_gather, 2)}),
              flush=True)
        return

    if a.hit_conditions:
        print(json.dumps({"hit_conditions": hit_conditions(torch, dev)}), flush=True)
        return

    if a.pmc_workload:
        model = synth.config_model(2)
        b = Bench(torch, dev, model, [a.batch], "memcpy", 8 << 20, a.copy_streams)
        x, out = b.io(a.batch, 10200 + a.batch)
        for _ in range(20):
            b.request(x, out, cold=False)
        src = torch.empty(256 << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        b.close()
        print(json.dumps({"pmc_workload": "20 warm forwards of the 24 x 4096 bf16 MLP at batch "
                          f"{a.batch}, then one 268435456-byte device copy"}), flush=True)
        return

    import paper_2306_03622_amd as tp
    log("measuring host-link peak (1 GiB pinned H2D copies and kernel gathers, best of 10 / 5)")
    link, link_copy, link_gather = link_rates(torch, dev)
    log(f"  link peak {link:.1f} GB/s (copy engine {link_copy:.1f}, gather kernel {link_gather:.1f})")
    if a.workload:
        bts = [int(v) for v in a.batches.split(",")]
        chunk = tp.DEFAULT_CHUNK if a.chunk in ("default", "elbow") else int(a.chunk)
        res = measure_workload(torch, dev, a.workload, bts, a.method, chunk, a.copy_streams, a.plan, link, a.steps,
                               a.warmup, a.trace, plan_link=link_copy if a.method != "gather" else link_gather,
                               cpu=not a.no_cpu, lib_flags=a.lib_flags)
        for v in res.values():
            if "cold_p50_ms" in v:
                v["link_peak_gbs"] = round(link, 2)
        print(json.dumps(res), flush=True)
        return

    # the group-size sweep creates many contexts; it runs after the measurements unless its
    # elbow is asked for as the group size
    sweep = None
    sweep_method = "gather" if a.method == "gather" else "memcpy"
    if a.chunk == "elbow" and not a.no_sweep:
        log("group-size sweep")
        sweep = elbow_sweep(torch, dev, sweep_method, a.copy_streams)
        a.chunk = sweep["elbow_bytes"]
    elif a.chunk in ("default", "elbow"):
        a.chunk = tp.DEFAULT_CHUNK
    else:
        a.chunk = int(a.chunk)

    model = synth.config_model(2)
    log("generating the 24 x 4096 bf16 MLP weights")
    model.blob()
    batches = [a.batch] if a.quick else sorted({1, 8, 32, a.batch})
    method = a.method
    extra = {}
    if method == "auto":
        rates = {}
        for meth in ("memcpy", "gather"):
            b = Bench(torch, dev, model, batches, meth, a.chunk, a.copy_streams, plan=a.plan,
                      link_gbs=link_gather if meth == "gather" else link_copy)
            b.swap_only()
            rates[meth] = model.total_bytes / (p50([b.swap_only() for _ in range(5)]) / 1e3) / 1e9
            b.close()
        method = max(rates, key=rates.get)
        extra["swap_rate_by_method_gbs"] = {k: round(v, 2) for k, v in rates.items()}
        log(f"  swap rates {rates} -> {method}")

    b = Bench(torch, dev, model, batches, method, a.chunk, a.copy_streams, plan=a.plan,
              link_gbs=link_gather if method == "gather" else link_copy)
    n_chunks = len(b.rt.chunks(b.mid))
    results = {}
    for bt in batches:
        log(f"cold/warm requests, batch {bt}")
        results[bt] = measure(b, bt, 10200 + bt, a.steps, a.warmup, max(4 * a.steps, 100))
    r = results[a.batch] if a.batch in results else results[batches[0]]
    B = a.batch if a.batch in results else batches[0]

    W = model.total_bytes
    warm_p50 = p50(r["warm"])
    cold_p50 = p50(r["cold"])
    bound = max(W / (link * 1e9) * 1e3, warm_p50)
    swap_gbs = W / (p50(r["swap"]) / 1e3) / 1e9

    # dominant compute kernel: the skinny bf16 GEMM (24 launches per forward, nothing else)
    reps = 50
    fwd_ms = b.event_time_ms(r["x"], r["out"], reps)
    kern_us = fwd_ms / 24 * 1e3
    K = N = 4096
    alg_bytes = N * K * 2 + N * 2 + B * K * 2 + B * N * 2
    achieved = alg_bytes / (kern_us * 1e-6) / 1e9
    flops = 2 * B * N * K
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": counted_traffic(B),
                "kernel": "k_gemv<1,4,8,true> (bf16 [B x 4096] x [4096 x 4096]^T + bias, GELU; 4 waves x 8 "
                          "k-blocks, blocked weights)",
                "avg_launch_us": round(kern_us, 2), "algorithmic_bytes_per_launch": alg_bytes,
                "mfma_util": round(flops / (kern_us * 1e-6) / 1e12 / BF16_PEAK_TFLOPS, 5)}

    for bt, rr in results.items():
        wp = p50(rr["warm"])
        fwd = b.event_time_ms(rr["x"], rr["out"], 20) if bt != B else fwd_ms
        extra[f"mlp24x4096_b{bt}"] = {
            "warm_forward_event_ms": round(fwd, 4),
            "hbm_frac_weights": round(W / (fwd * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "mfma_util": round(2 * bt * K * N * 24 / (fwd * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 5),
            "swap_only_gbs": round(W / (p50(rr["swap"]) / 1e3) / 1e9, 2),
            "cold_p50_ms": round(p50(rr["cold"]), 3), "cold_p10_ms": round(pct(rr["cold"], 10), 3),
            "cold_p90_ms": round(pct(rr["cold"], 90), 3), "warm_p50_ms": round(wp, 4),
            "bound_ms": round(max(W / (link * 1e9) * 1e3, wp), 3),
            "cold_over_bound": round(p50(rr["cold"]) / max(W / (link * 1e9) * 1e3, wp), 4),
            "swap_only_p50_ms": round(p50(rr["swap"]), 3)}
    b.close()

    extra.update(children)

    if sweep is None and not a.no_sweep:
        log("group-size sweep")
        sweep = elbow_sweep(torch, dev, sweep_method, a.copy_streams)

    cpu = None
    if not a.no_cpu:
        log("CPU oracle baseline")
        cpu = cpu_baseline(model, B, 10200 + B, gpu_out=r["out"].cpu().numpy())
    log("matrix-core and HBM peak probes")
    peaks = machine_peaks()

    line = {
        "metric": "cold-start p50 latency (swap+exec)",
        "value": round(cold_p50, 3), "unit": "ms", "n_gpus": 1, "steps": a.steps, "warmup": a.warmup,
        "ms_per_step": round(r["t_all"] / a.steps * 1e3, 3), "higher_is_better": False, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"24-layer MLP, hidden 4096, bf16 weights (805,502,976 B) swapped cold from pinned "
                               f"host memory, batch {B}", "batch": B, "copy_method": method,
                   "chunk_plan": a.plan, "chunks": n_chunks,
                   "chunk_min_bytes": a.chunk if a.plan == "greedy" else None, "copy_streams": a.copy_streams or 1,
                   "direct_max_bytes": tp.DEFAULT_DIRECT},
        "bound_ms": round(bound, 3), "cold_over_bound": round(cold_p50 / bound, 4),
        "swap_gbs": round(swap_gbs, 2), "link_peak_gbs": round(link, 2), "link_copy_engine_gbs": round(link_copy, 2),
        "link_gather_kernel_gbs": round(link_gather, 2), "link_theoretical_gbs": PCIE5_X16_GBS,
        "peaks": peaks,
        "warm_p50_ms": round(warm_p50, 4), "roofline": roofline, "cpu_baseline": cpu, "elbow_sweep": sweep,
        "extra": extra,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
