"""Swap-in invariants on the GPU (exact): swapped bytes equal the host copy for both copy
methods; pipelined output equals preloaded output bit for bit; relocation after a
different eviction history does not change the output; throttled copies with poisoned
evicted extents give the same bits; arena decisions follow the reference simulator."""
import numpy as np
import pytest

import paper_2306_03622_amd as tp
import synth
from oracle.arena_sim import ArenaSim
from tests.common import (check_parity, expected_host_image, infer, log, make_runtime, out_shape, to_device,
                          torch_dev)


def infer_shape(m):
    return out_shape(m, 1)[1:]

pytestmark = pytest.mark.gpu


def _models():
    return [synth.mlp(6, 512, "bf16", "gelu", seed=61),
            synth.bert(seed=62, layers=2, d=128, heads=2, ffn=256, seq=64, vocab=500, maxpos=64),
            synth.resnet50(seed=63, classes=10, image=32)]


def _inputs(ms, batch=2):
    return [synth.config_input(m, batch, 70 + i) for i, m in enumerate(ms)]


@pytest.mark.parametrize("method", [tp.TP_COPY_MEMCPY, tp.TP_COPY_GATHER])
@pytest.mark.parametrize("chunk", [0, 64 << 10, 2 << 20, 1 << 40])
def test_swapped_bytes_identical(method, chunk):
    ms = _models()
    rt, ids = make_runtime(ms, batch_max=2, copy_method=method, chunk_min_bytes=chunk)
    torch, dev = torch_dev()
    s = torch.cuda.Stream(device=dev)
    for mid, m in zip(ids, ms):
        rt.swap_in(mid, stream=s)
        s.synchronize()
        assert rt.resident(mid)
        image = rt.host_image(mid)
        assert np.array_equal(image, expected_host_image(m)), m.arch
        assert np.array_equal(rt.extent(mid).cpu().numpy(), image), (method, chunk, m.arch)
    rt.close()


@pytest.mark.parametrize("method", [tp.TP_COPY_MEMCPY, tp.TP_COPY_GATHER])
@pytest.mark.parametrize("streams", [1, 2])
def test_pipelined_equals_preloaded(method, streams):
    ms, xs = _models(), None
    xs = _inputs(ms)
    rt, ids = make_runtime(ms, batch_max=2, copy_method=method, chunk_min_bytes=0, copy_streams=streams,
                           flags=tp.TP_FLAG_NO_GRAPH)
    torch, dev = torch_dev()
    s = torch.cuda.Stream(device=dev)
    for mid, m, x in zip(ids, ms, xs):
        log(f"pipelined vs preloaded: {m.arch}")
        pipelined = infer(rt, mid, m, x, stream=s)          # cold: per-layer waits
        rt.evict(mid)
        rt.swap_in(mid, stream=s)                           # preloaded: swap, sync, run
        s.synchronize()
        preloaded = infer(rt, mid, m, x, stream=s)
        assert np.array_equal(pipelined, preloaded)
    rt.close()


@pytest.mark.parametrize("cfg", [2, 3, 4])
def test_cost_plan_pipelined_equals_preloaded_full_size(cfg):
    # the cost-model plan groups layers unevenly (tiny head chunks, one large middle chunk);
    # the pipelined cold request must compute the same bits as the preloaded one, and match
    # the oracle
    m = synth.config_model(cfg)
    batch = 2
    x = synth.config_input(m, batch, 777)
    rt, ids = make_runtime([m], batch_max=batch, plan=tp.TP_PLAN_COST, plan_batch=8, link_gbs=57.0)
    chunks = rt.chunks(ids[0])
    log(f"cost plan cfg{cfg}: {len(chunks)} chunks, first layers {[c['first_layer'] for c in chunks]}")
    torch, dev = torch_dev()
    s = torch.cuda.Stream(device=dev)
    pipelined = infer(rt, ids[0], m, x, stream=s)
    rt.evict(ids[0])
    rt.swap_in(ids[0], stream=s)
    s.synchronize()
    preloaded = infer(rt, ids[0], m, x, stream=s)
    assert np.array_equal(pipelined, preloaded)
    got = rt.extent(ids[0]).cpu().numpy()
    assert np.array_equal(got, rt.host_image(ids[0]))
    rt.close()
    check_parity(pipelined, m, x, 2e-2)
    m.drop_blob()


def test_warm_graph_replay_equals_kernel_by_kernel():
    # every family with a forward pass long enough (>= 16 launches) to be replayed as a graph
    ms = [synth.mlp(18, 256, "bf16", "gelu", seed=61),
          synth.bert(seed=62, layers=3, d=128, heads=2, ffn=256, seq=64, vocab=500, maxpos=64),
          synth.resnet50(seed=63, classes=10, image=32)]
    torch, dev = torch_dev()
    eager_rt, eager_ids = make_runtime(ms, batch_max=3, flags=tp.TP_FLAG_NO_GRAPH)
    rt, ids = make_runtime(ms, batch_max=3)
    s = torch.cuda.Stream(device=dev)
    for k, m in enumerate(ms):
        # same buffers, new contents each request; then a different output buffer and batch
        x_np = synth.config_input(m, 3, 200 + k)
        x = torch.empty_like(to_device(x_np))
        outs = [torch.empty((3,) + tuple(infer_shape(m)), dtype=torch.float32, device=dev) for _ in range(2)]
        for rep in range(5):
            x_np = synth.config_input(m, 3, 300 + 10 * k + rep)
            x.copy_(to_device(x_np))
            want = infer(eager_rt, eager_ids[k], m, x_np)
            out = outs[rep % 2]
            torch.cuda.synchronize()
            rt.infer(ids[k], x, out, stream=s)
            s.synchronize()
            assert np.array_equal(out.cpu().numpy(), want), (m.arch, rep)
        # a smaller batch makes a new graph
        got = infer(rt, ids[k], m, x_np[:1])
        assert np.array_equal(got, infer(eager_rt, eager_ids[k], m, x_np[:1]))
    st = rt.stats()
    # per family: one capture at batch 3 (the cold request launches eagerly) and one at
    # batch 1; the batch-3 graph was repointed at the other output buffer on every second
    # request, then the batch-1 request's new buffers were captured fresh
    assert st["graph_captures"] == 2 * len(ms), st
    assert st["graph_repoints"] == 3 * len(ms), st
    eager_rt.close()
    rt.close()


def test_warm_hits_with_new_buffers_repoint_the_graph():
    # every warm request brings buffers of its own (as a server does): each must compute the
    # kernel-by-kernel bits, and only the first warm request per (model, batch) may capture
    ms = [synth.mlp(18, 256, "bf16", "gelu", seed=64),
          synth.bert(seed=65, layers=3, d=128, heads=2, ffn=256, seq=64, vocab=500, maxpos=64),
          synth.resnet50(seed=66, classes=10, image=32)]
    torch, dev = torch_dev()
    eager_rt, eager_ids = make_runtime(ms, batch_max=4, flags=tp.TP_FLAG_NO_GRAPH)
    rt, ids = make_runtime(ms, batch_max=4)
    s = torch.cuda.Stream(device=dev)
    keep = []                     # every buffer stays allocated, so no address comes back
    for k, m in enumerate(ms):
        for batch in (4, 2):
            for rep in range(4):
                x_np = synth.config_input(m, batch, 500 + 31 * k + 7 * rep + batch)
                want = infer(eager_rt, eager_ids[k], m, x_np)
                x = to_device(x_np)
                out = torch.full(out_shape(m, batch), float("nan"), dtype=torch.float32, device=dev)
                keep += [x, out]
                torch.cuda.synchronize()
                rt.infer(ids[k], x, out, stream=s)
                s.synchronize()
                got = out.cpu().numpy()
                assert np.array_equal(got, want), (m.arch, batch, rep)
                if rep == 0 and batch == 4:
                    check_parity(got, m, x_np, 2e-2)
    st = rt.stats()
    log(f"graph captures {st['graph_captures']}, repoints {st['graph_repoints']}")
    # per family: the very first request is cold (eager); batch 4 then captures once and
    # repoints twice, batch 2 captures once and repoints three times
    assert st["graph_captures"] == 2 * len(ms), st
    assert st["graph_repoints"] == 5 * len(ms), st
    eager_rt.close()
    rt.close()


def test_warm_hits_after_a_move_rebase_the_graph():
    # a model that comes back into another extent keeps its graph: the nodes holding weight
    # pointers are moved to the new extent (retired extents are poisoned, so a node left
    # pointing at the old one reads poison); the bits stay the kernel-by-kernel ones
    ms = [synth.mlp(18, 256, "bf16", "gelu", seed=71),
          synth.bert(seed=72, layers=3, d=128, heads=2, ffn=256, seq=64, vocab=500, maxpos=64),
          synth.resnet50(seed=73, classes=10, image=32)]
    spacer = synth.mlp(2, 256, "bf16", "gelu", seed=74)
    eager_rt, eager_ids = make_runtime(ms, batch_max=2, flags=tp.TP_FLAG_NO_GRAPH)
    arena = max(m.total_bytes for m in ms) + spacer.total_bytes + (1 << 20)
    rt, ids = make_runtime(ms + [spacer], batch_max=2, arena_bytes=arena, flags=tp.TP_FLAG_POISON)
    sp = ids[-1]
    torch, dev = torch_dev()
    s = torch.cuda.Stream(device=dev)
    rebases, keep = 0, []
    for k, m in enumerate(ms):
        x_np = synth.config_input(m, 2, 700 + k)
        want = infer(eager_rt, eager_ids[k], m, x_np)
        for mid in ids:
            rt.evict(mid)
        seen = []
        # resident at the arena's base, then after the spacer, then at the base again
        for step, with_spacer in enumerate((False, False, True, True, False)):
            if step:
                rt.evict(ids[k])
                rt.evict(sp)
                if with_spacer:
                    rt.swap_in(sp, stream=s)
            rt.swap_in(ids[k], stream=s)
            s.synchronize()
            off = rt.info(ids[k])["extent_offset"]
            if seen and off != seen[-1]:
                rebases += 1
            seen.append(off)
            # a warm hit with buffers of its own (kept allocated, so no address comes back)
            x = to_device(x_np)
            out = torch.full(out_shape(m, 2), float("nan"), dtype=torch.float32, device=dev)
            keep += [x, out]
            torch.cuda.synchronize()
            rt.infer(ids[k], x, out, stream=s)
            s.synchronize()
            assert np.array_equal(out.cpu().numpy(), want), (m.arch, step, off)
        log(f"{m.arch}: offsets {seen}")
        assert len(set(seen)) == 2, seen
    st = rt.stats()
    log(f"graph captures {st['graph_captures']}, repoints {st['graph_repoints']}, rebases {st['graph_rebases']}")
    # one capture per model (its first hit); every later hit repoints, those after a move also
    # move the weight pointers
    assert st["graph_captures"] == len(ms), st
    assert st["graph_repoints"] == 4 * len(ms), st
    assert st["graph_rebases"] == rebases == 2 * len(ms), st
    eager_rt.close()
    rt.close()


def test_eviction_order_and_placement_do_not_change_outputs():
    ms = _models()
    xs = _inputs(ms)
    small_arena = max(m.total_bytes for m in ms) + sum(sorted(m.total_bytes for m in ms)[:1]) + 4096
    ref_rt, ref_ids = make_runtime(ms, batch_max=2)
    ref = [infer(ref_rt, i, m, x) for i, m, x in zip(ref_ids, ms, xs)]
    ref_rt.close()
    for r, m, x in zip(ref, ms, xs):
        check_parity(r, m, x, 2e-2)
    rt, ids = make_runtime(ms, batch_max=2, arena_bytes=small_arena, flags=tp.TP_FLAG_POISON)
    offsets = {i: set() for i in range(3)}
    order = [0, 1, 2, 1, 0, 2, 2, 0, 1, 0]
    for k in order:
        got = infer(rt, ids[k], ms[k], xs[k])
        offsets[k].add(rt.info(ids[k])["extent_offset"])
        assert np.array_equal(got, ref[k]), (k, order)
    log(f"offsets seen: {offsets}")
    assert rt.stats()["evictions"] > 0
    assert any(len(v) > 1 for v in offsets.values())
    rt.close()


@pytest.mark.parametrize("plan", [tp.TP_PLAN_GREEDY, tp.TP_PLAN_COST])
def test_throttled_poisoned_swaps_are_bit_identical(plan):
    ms = _models()
    xs = _inputs(ms)
    ref_rt, ref_ids = make_runtime(ms, batch_max=2)
    ref = [infer(ref_rt, i, m, x) for i, m, x in zip(ref_ids, ms, xs)]
    ref_rt.close()
    for r, m, x in zip(ref, ms, xs):
        check_parity(r, m, x, 2e-2)
    # each chunk waits ~200 us on the copy stream; a layer that did not wait for its chunk
    # would read 0xFF bytes (NaN) left by the poisoned eviction of the previous tenant
    arena = max(m.total_bytes for m in ms) + 4096
    rt, ids = make_runtime(ms, batch_max=2, arena_bytes=arena, chunk_min_bytes=0,
                           flags=tp.TP_FLAG_POISON | tp.TP_FLAG_THROTTLE, throttle_us=200, plan=plan,
                           link_gbs=0.5, chunk_us=1.0)
    for rep in range(2):
        for k in range(3):
            got = infer(rt, ids[k], ms[k], xs[k])
            assert np.array_equal(got, ref[k]), (rep, k)
    assert rt.stats()["misses"] == 6
    rt.close()


def test_arena_decisions_match_simulator():
    rng = np.random.default_rng(5)
    ms = [synth.mlp(int(rng.integers(1, 5)), int(rng.choice([64, 128, 256])), "bf16", "relu", seed=80 + i)
          for i in range(8)]
    cap = max(int(sum(m.total_bytes for m in ms) * 0.45), max(m.total_bytes for m in ms)) // 256 * 256
    rt, ids = make_runtime(ms, batch_max=1, arena_bytes=cap)
    sim = ArenaSim(cap, align=256)
    for i, m in zip(ids, ms):
        sim.register(i, m.total_bytes)
    xs = [synth.mlp_input(1, m.dims["width"], "bf16", 90 + i) for i, m in enumerate(ms)]
    for step in range(60):
        k = int(rng.integers(0, len(ms)))
        if rng.random() < 0.1:
            rt.evict(ids[k]); sim.evict(ids[k])
            continue
        want = sim.request(ids[k])
        infer(rt, ids[k], ms[k], xs[k])
        assert rt.info(ids[k])["extent_offset"] == want["offset"]
        assert [rt.resident(i) for i in ids] == [i in sim.where for i in ids], step
    got = rt.stats()
    for key, v in sim.stats().items():
        assert got[key] == v, (key, got[key], v)
    rt.close()


def test_single_chunk_swaps_over_previous_tenant():
    # one chunk per model and an arena that holds one model at a time: every request swaps
    # over the extent the previous tenant was still reading
    ms = _models()
    xs = _inputs(ms)
    ref_rt, ref_ids = make_runtime(ms, batch_max=2, flags=tp.TP_FLAG_NO_GRAPH)
    ref = [infer(ref_rt, i, m, x) for i, m, x in zip(ref_ids, ms, xs)]
    ref_rt.close()
    for r, m, x in zip(ref, ms, xs):
        check_parity(r, m, x, 2e-2)
    arena = max(m.total_bytes for m in ms) + 4096
    rt, ids = make_runtime(ms, batch_max=2, arena_bytes=arena, chunk_min_bytes=1 << 40)
    torch, dev = torch_dev()
    s = torch.cuda.Stream(device=dev)
    for rep in range(3):
        for k in range(3):
            assert len(rt.chunks(ids[k])) == 1
            got = infer(rt, ids[k], ms[k], xs[k], stream=s)
            assert np.array_equal(got, ref[k]), (rep, k)
            assert np.array_equal(rt.extent(ids[k]).cpu().numpy(), expected_host_image(ms[k])), (rep, k)
    assert rt.stats()["misses"] == 9
    rt.close()


# the swap designs of the breakdown: every one computes the same bits as the default
ABLATION = {
    "pageable-serial-per-tensor": dict(copy_method=tp.TP_COPY_PAGEABLE, chunk_min_bytes=0,
                                       flags=tp.TP_FLAG_SERIAL | tp.TP_FLAG_PER_TENSOR),
    "pinned-serial-per-tensor": dict(chunk_min_bytes=0, flags=tp.TP_FLAG_SERIAL | tp.TP_FLAG_PER_TENSOR),
    "pipelined-per-tensor": dict(chunk_min_bytes=0, flags=tp.TP_FLAG_PER_TENSOR),
    "grouped-by-tensor": dict(chunk_min_bytes=96 << 10, flags=tp.TP_FLAG_PER_TENSOR),
    "pageable-pipelined": dict(copy_method=tp.TP_COPY_PAGEABLE, chunk_min_bytes=96 << 10),
    "zero-copy": dict(copy_method=tp.TP_COPY_ZERO),
}


@pytest.mark.parametrize("name", sorted(ABLATION))
def test_swap_designs_compute_the_same_bits(name):
    ms = _models()
    xs = _inputs(ms)
    ref_rt, ref_ids = make_runtime(ms, batch_max=2, flags=tp.TP_FLAG_NO_GRAPH)
    ref = [infer(ref_rt, i, m, x) for i, m, x in zip(ref_ids, ms, xs)]
    ref_rt.close()
    for r, m, x in zip(ref, ms, xs):                    # the reference itself matches the oracle
        check_parity(r, m, x, 2e-2)
    arena = max(m.total_bytes for m in ms) + 4096       # one model at a time
    rt, ids = make_runtime(ms, batch_max=2, arena_bytes=arena, **ABLATION[name])
    zero = ABLATION[name].get("copy_method") == tp.TP_COPY_ZERO
    for rep in range(2):
        for k in range(3):
            log(f"{name}: rep {rep} {ms[k].arch}")
            got = infer(rt, ids[k], ms[k], xs[k])
            assert np.array_equal(got, ref[k]), (name, rep, k)
            if zero:
                assert not rt.resident(ids[k])
            else:
                assert np.array_equal(rt.extent(ids[k]).cpu().numpy(), expected_host_image(ms[k])), (name, rep, k)
    st = rt.stats()
    assert st["misses"] == (0 if zero else 6) and st["hits"] == 0
    if zero:
        # an explicit swap-in still makes the model resident; the request then hits
        rt.swap_in(ids[0])
        got = infer(rt, ids[0], ms[0], xs[0])
        assert np.array_equal(got, ref[0]) and rt.stats()["hits"] == 1
    rt.close()


@pytest.mark.parametrize("flags", [0, tp.TP_FLAG_NO_GRAPH])
def test_direct_access_then_background_swap(flags):
    # cold requests read the pinned host copy; the swap runs behind them with a ~200 us
    # delay per chunk and evicted extents poisoned, so a later request that did not wait
    # for the swap would read NaN bytes
    ms = _models()
    xs = _inputs(ms)
    ref_rt, ref_ids = make_runtime(ms, batch_max=2, flags=tp.TP_FLAG_NO_GRAPH)
    ref = [infer(ref_rt, i, m, x) for i, m, x in zip(ref_ids, ms, xs)]
    ref_rt.close()
    for r, m, x in zip(ref, ms, xs):                    # the reference itself matches the oracle
        check_parity(r, m, x, 2e-2)
    arena = max(m.total_bytes for m in ms) + 4096
    rt, ids = make_runtime(ms, batch_max=2, arena_bytes=arena, chunk_min_bytes=0, direct_max_bytes=1 << 40,
                           flags=flags | tp.TP_FLAG_POISON | tp.TP_FLAG_THROTTLE, throttle_us=200)
    torch, dev = torch_dev()
    s = torch.cuda.Stream(device=dev)
    for rep in range(2):
        for k in range(3):
            log(f"direct access: rep {rep} {ms[k].arch}")
            cold = infer(rt, ids[k], ms[k], xs[k], stream=s)
            warm = infer(rt, ids[k], ms[k], xs[k], stream=s)
            assert np.array_equal(cold, ref[k]) and np.array_equal(warm, ref[k]), (rep, k)
            assert np.array_equal(rt.extent(ids[k]).cpu().numpy(), expected_host_image(ms[k])), (rep, k)
    st = rt.stats()
    assert st["misses"] == 6 and st["hits"] == 6
    rt.close()


def test_traced_timeline_is_causal():
    # chunk c's first kernel passes its wait only after its copy ended; copies run in order
    m = synth.resnet50(seed=63, classes=10, image=32)
    x = synth.config_input(m, 2, 71)
    rt, ids = make_runtime([m], batch_max=2, chunk_min_bytes=2 << 20, flags=tp.TP_FLAG_TRACE)
    ref_rt, ref_ids = make_runtime([m], batch_max=2)
    want = infer(ref_rt, ref_ids[0], m, x)
    ref_rt.close()
    check_parity(want, m, x, 2e-2)
    for rep in range(3):
        rt.evict(ids[0])
        assert np.array_equal(infer(rt, ids[0], m, x), want)
        tl = rt.timeline()
        n = len(rt.chunks(ids[0]))
        assert n > 3 and len(tl["copy_begin_ms"]) == n
        cb, ce, xb = tl["copy_begin_ms"], tl["copy_end_ms"], tl["exec_begin_ms"]
        log(f"timeline rep {rep}: total {tl['total_ms']:.3f} ms, last copy end {ce[-1]:.3f} ms")
        for c in range(n):
            assert cb[c] <= ce[c] <= xb[c] + 1e-3 <= tl["total_ms"] + 2e-3, (c, cb[c], ce[c], xb[c])
            if c:
                assert ce[c - 1] <= cb[c] + 1e-3 and xb[c - 1] <= xb[c] + 1e-3
    rt.close()
