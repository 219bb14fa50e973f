"""Error paths of the runtime on the GPU. No device work fails: a host-side test hook
(tp_debug_fail_copy) makes the n-th copy a context enqueues fail before anything is
enqueued for it, as if the HIP runtime had rejected the call. A failed request must return
TP_E_HIP, leave its model non-resident with consistent counters and retired extents, and a
retry must swap the model in again and compute the undisturbed run's bits (which match the
oracle)."""
import numpy as np
import pytest

import paper_2306_03622_amd as tp
import synth
from oracle.partition_sim import PartitionArenaSim
from tests.common import check_parity, expected_host_image, infer, log, make_runtime, out_shape, to_device, torch_dev

pytestmark = pytest.mark.gpu


def _bert():
    return synth.bert(seed=91, layers=4, d=128, heads=2, ffn=256, seq=64, vocab=500, maxpos=64)


def _reference(m, x):
    rt, (mid,) = make_runtime([m], batch_max=x.shape[0], flags=tp.TP_FLAG_NO_GRAPH)
    want = infer(rt, mid, m, x)
    rt.close()
    check_parity(want, m, x, 2e-2)
    return want


def _expect_hip_error(fn):
    torch, _ = torch_dev()
    with pytest.raises(tp.TorporError) as ei:
        fn()
    torch.cuda.synchronize()
    assert ei.value.status == tp.TP_E_HIP, ei.value
    log(f"  failed as expected: {ei.value}")


@pytest.mark.parametrize("nth", [1, 2, 4])
@pytest.mark.parametrize("caller_stream", [False, True])
def test_failed_chunk_copy_of_a_cold_request(nth, caller_stream):
    # one chunk per layer (5 chunks): the first, second or fourth chunk's copy fails while
    # the layers before it are already enqueued
    m, x = _bert(), synth.config_input(_bert(), 2, 92)
    want = _reference(m, x)
    flags = tp.TP_FLAG_POISON | (tp.TP_FLAG_CALLER_STREAM if caller_stream else 0)
    rt, (mid,) = make_runtime([m], batch_max=2, chunk_min_bytes=0, flags=flags)
    assert len(rt.chunks(mid)) == 5
    rt.fail_copy(nth)
    _expect_hip_error(lambda: infer(rt, mid, m, x))
    st = rt.stats()
    assert not rt.resident(mid)
    assert (st["misses"], st["hits"], st["resident"], st["used"]) == (1, 0, 0, 0), st
    got = infer(rt, mid, m, x)                 # the retry swaps the whole model again
    assert rt.resident(mid) and rt.stats()["misses"] == 2
    assert np.array_equal(got, want)
    assert np.array_equal(rt.extent(mid).cpu().numpy(), expected_host_image(m))
    assert np.array_equal(infer(rt, mid, m, x), want)       # and a warm request after it
    rt.close()


def test_failed_swap_in():
    m, x = _bert(), synth.config_input(_bert(), 2, 93)
    want = _reference(m, x)
    rt, (mid,) = make_runtime([m], batch_max=2, chunk_min_bytes=0, flags=tp.TP_FLAG_POISON)
    torch, dev = torch_dev()
    s = torch.cuda.Stream(device=dev)
    rt.fail_copy(3)
    _expect_hip_error(lambda: rt.swap_in(mid, stream=s))
    assert not rt.resident(mid) and rt.stats()["resident"] == 0
    rt.swap_in(mid, stream=s)
    s.synchronize()
    assert rt.resident(mid)
    assert np.array_equal(rt.extent(mid).cpu().numpy(), expected_host_image(m))
    assert np.array_equal(infer(rt, mid, m, x), want)
    assert rt.stats()["hits"] == 1
    rt.close()


def test_failed_background_swap_behind_direct_access():
    # a small model read over the host link by its cold request, with the swap behind it:
    # the swap's copy fails after the request's kernels were enqueued
    m = synth.mlp(4, 256, "bf16", "gelu", seed=94)
    x = synth.config_input(m, 3, 95)
    want = _reference(m, x)
    rt, (mid,) = make_runtime([m], batch_max=3, direct_max_bytes=1 << 40, flags=tp.TP_FLAG_POISON)
    rt.fail_copy(1)
    _expect_hip_error(lambda: infer(rt, mid, m, x))
    assert not rt.resident(mid)
    assert np.array_equal(infer(rt, mid, m, x), want)      # direct access again, swap behind it
    assert rt.resident(mid)
    assert np.array_equal(infer(rt, mid, m, x), want)      # warm, after the swap
    assert np.array_equal(rt.extent(mid).cpu().numpy(), expected_host_image(m))
    rt.close()


def test_failed_swap_in_kernel_of_a_small_fp32_model():
    # a small fp32 MLP's cold request swaps it in with its first layer kernel; that launch
    # counts as the copy, fails, and leaves the model non-resident for the retry
    m = synth.config_model(1)
    x = synth.config_input(m, 2, 97)
    rt, (mid,) = make_runtime([m], batch_max=2, direct_max_bytes=1 << 40)
    rt.fail_copy(1)
    _expect_hip_error(lambda: infer(rt, mid, m, x))
    st = rt.stats()
    assert not rt.resident(mid)
    assert (st["misses"], st["hits"], st["resident"]) == (1, 0, 0), st
    got = infer(rt, mid, m, x)
    check_parity(got, m, x, 1e-4)
    assert rt.resident(mid) and rt.stats()["misses"] == 2
    assert np.array_equal(rt.extent(mid).cpu().numpy(), m.blob())
    assert np.array_equal(infer(rt, mid, m, x), got)
    rt.close()


def test_armed_failure_counts_only_copies():
    # the countdown passes over warm requests (no copies) and fires on the next swap
    m, x = _bert(), synth.config_input(_bert(), 1, 96)
    want = _reference(m, x)
    rt, (mid,) = make_runtime([m], batch_max=1, chunk_min_bytes=0)
    assert np.array_equal(infer(rt, mid, m, x), want)
    rt.fail_copy(2)
    for _ in range(3):
        assert np.array_equal(infer(rt, mid, m, x), want)
    rt.evict(mid)
    _expect_hip_error(lambda: infer(rt, mid, m, x))
    rt.fail_copy(0)
    assert np.array_equal(infer(rt, mid, m, x), want)
    with pytest.raises(tp.TorporError) as ei:
        rt.fail_copy(-1)
    assert ei.value.status == tp.TP_E_INVAL
    rt.close()


def test_failed_consolidation_move_rolls_back_the_admission():
    # The scaled multi-tenant workload on a partitioned arena with consolidation. At the first
    # request whose admission moves a model (found with the oracle's partition simulator),
    # the move's copy fails: the request fails, the requester and the moved models are left
    # non-resident, and every later request still computes the all-resident run's bits.
    torch, dev = torch_dev()
    specs = synth.tenant_models(9)
    models = [m for _, m in synth.build_models(specs, workers=9)]
    trace = synth.tenant_trace(120, n_models=9)
    cap, part = 1100 << 20, 512 << 20
    sim = PartitionArenaSim(cap, part, 256, consolidate=True)
    for i, m in enumerate(models):
        sim.register(i + 1, m.total_bytes)            # the ids the runtime will assign
    first_move = next(r for r, k in enumerate(trace.model)
                      if any(st[0] == "move" for st in sim.request(int(k) + 1).get("steps", [])))
    n = min(len(trace.model), first_move + 40)
    log(f"first consolidation move at request {first_move}; replaying {n} requests")
    xs = [synth.request_input(models[int(trace.model[r])], int(trace.input_seed[r])) for r in range(n)]
    ws = max(tp.tp_workspace_bytes(tp.ModelDesc.of(m), 1) for m in models)

    big = sum(m.total_bytes for m in models) + (64 << 20)
    ref_rt = tp.Runtime(big // 256 * 256, ws)
    ref_ids = [ref_rt.register(tp.ModelDesc.of(m), m.blob()) for m in models]
    ref = [infer(ref_rt, ref_ids[int(trace.model[r])], models[int(trace.model[r])], xs[r]) for r in range(n)]
    ref_rt.close()

    rt = tp.Runtime(cap, ws, alloc=tp.TP_ALLOC_PARTITION_CONSOLIDATE, partition_bytes=part, flags=tp.TP_FLAG_POISON)
    ids = [rt.register(tp.ModelDesc.of(m), m.blob()) for m in models]
    assert ids == list(range(1, len(models) + 1))
    for r in range(n):
        k = int(trace.model[r])
        if r == first_move:
            before = {i: rt.resident(i) for i in ids}
            rt.fail_copy(1)
            _expect_hip_error(lambda: infer(rt, ids[k], models[k], xs[r]))
            after = {i: rt.resident(i) for i in ids}
            assert not after[ids[k]]
            lost = [i for i in ids if before[i] and not after[i]]
            log(f"  request {r}: models left non-resident {lost}")
            assert lost, "the failed move's model stays resident"
            assert rt.stats()["resident"] == sum(after.values())
            continue
        got = infer(rt, ids[k], models[k], xs[r])
        assert np.array_equal(got, ref[r]), (r, k)
    rt.close()
