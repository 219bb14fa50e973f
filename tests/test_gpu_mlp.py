"""MLP family through the C ABI on the GPU vs the oracle, plus the swap invariants.

fp32 (the 4 x 256 workload): normwise error <= 1e-4. bf16: <= 2e-2.
"""
import numpy as np
import pytest

import synth
from tests.common import check_parity, expected_host_image, infer, log, make_runtime, to_device, torch_dev

pytestmark = pytest.mark.gpu


def test_cfg1_fp32_cold_then_warm():
    m = synth.config_model(1)
    x = synth.config_input(m, 1, 10101)
    rt, (mid,) = make_runtime([m])
    log("cfg1 cold")
    cold = infer(rt, mid, m, x)
    assert rt.resident(mid)
    warm = infer(rt, mid, m, x)
    check_parity(cold, m, x, 1e-4)
    assert np.array_equal(cold, warm)
    # swapped bytes are the host bytes (fp32 weights are stored as registered)
    assert np.array_equal(rt.host_image(mid), m.blob())
    assert np.array_equal(rt.extent(mid).cpu().numpy(), m.blob())
    st = rt.stats()
    assert (st["hits"], st["misses"], st["bytes_swapped"]) == (1, 1, m.total_bytes)
    rt.close()


@pytest.mark.parametrize("width,batch", [(256, 1), (256, 8), (264, 3), (1024, 2), (256, 9), (1032, 2)])
def test_fp32_cold_request_swaps_in_with_its_first_kernel(width, batch):
    # Small fp32 MLPs under direct access: up to width 1024 and batch 8 the cold request's
    # first layer kernel also copies the whole image into the arena (run_mlp_swapin); batch 9
    # and width 1032 take direct access with the swap behind it. Two models share an arena that
    # holds one, so each cold request reuses the extent the other just used, from a new
    # stream (first pass) or the same one (second pass).
    a = synth.mlp(4, width, "f32", "relu", seed=40 + width)
    b = synth.mlp(4, width, "f32", "gelu", seed=41 + width, bias_std=0.1)
    xa = synth.mlp_input(batch, width, "f32", 50 + batch)
    xb = synth.mlp_input(batch, width, "f32", 60 + batch)
    arena = max(a.total_bytes, b.total_bytes) + 4096
    rt, (ia, ib) = make_runtime([a, b], batch_max=batch, arena_bytes=arena, direct_max_bytes=1 << 40)
    torch, dev = torch_dev()
    same = torch.cuda.Stream(device=dev)
    for rep in range(2):
        for mid, m, x in ((ia, a, xa), (ib, b, xb)):
            log(f"fp32 swap-in: width {width} batch {batch} rep {rep} model {mid}")
            s = same if rep else None
            cold = infer(rt, mid, m, x, stream=s)
            assert rt.resident(mid)
            warm = infer(rt, mid, m, x, stream=s)
            check_parity(cold, m, x, 1e-4)
            assert np.array_equal(cold, warm)
            assert np.array_equal(rt.extent(mid).cpu().numpy(), m.blob())
    st = rt.stats()
    assert (st["misses"], st["hits"], st["bytes_swapped"]) == (4, 4, 2 * (a.total_bytes + b.total_bytes))
    rt.close()


@pytest.mark.parametrize("layers,dtype", [(1, "f32"), (2, "f32"), (1, "bf16"), (2, "bf16")])
def test_shallow_mlps(layers, dtype):
    # one- and two-layer models (the first layer is also the last) through the swap path and
    # under direct access (for fp32 the swap-in kernel): oracle parity, cold == warm bitwise,
    # the extent equals the library's host image
    m = synth.mlp(layers, 256, dtype, "relu", seed=80 + layers)
    x = synth.mlp_input(3, 256, dtype, 81)
    tol = 1e-4 if dtype == "f32" else 2e-2
    for direct in (0, 1 << 40):
        log(f"mlp {layers} x 256 {dtype}, direct limit {direct}")
        rt, (mid,) = make_runtime([m], batch_max=3, direct_max_bytes=direct)
        cold = infer(rt, mid, m, x)
        warm = infer(rt, mid, m, x)
        check_parity(cold, m, x, tol)
        assert np.array_equal(cold, warm)
        assert np.array_equal(rt.extent(mid).cpu().numpy(), expected_host_image(m))
        rt.close()


def test_infer_rejects_malformed_requests():
    # argument errors come back as TP_E_INVAL / TP_E_NOSPC before anything is enqueued, and
    # leave the context serving
    import paper_2306_03622_amd as tp
    m = synth.mlp(2, 256, "f32", "relu", seed=91)
    x_np = synth.mlp_input(2, 256, "f32", 92)
    rt, (mid,) = make_runtime([m], batch_max=2)
    torch, dev = torch_dev()
    x = to_device(x_np)
    out = torch.empty((2, 256), dtype=torch.float32, device=dev)
    for batch, xi, oi, want in ((0, x, out, tp.TP_E_INVAL), (2, None, out, tp.TP_E_INVAL),
                                (2, x, None, tp.TP_E_INVAL), (64, x, out, tp.TP_E_NOSPC)):
        with pytest.raises(tp.TorporError) as ei:
            tp.tp_infer(rt.ctx, mid, xi, batch, oi, torch.cuda.current_stream(dev))
        assert ei.value.status == want, (batch, ei.value)
    with pytest.raises(tp.TorporError) as ei:
        tp.tp_infer(rt.ctx, mid + 100, x, 2, out, torch.cuda.current_stream(dev))
    assert ei.value.status == tp.TP_E_NOENT
    assert rt.stats()["misses"] == 0 and not rt.resident(mid)
    got = infer(rt, mid, m, x_np)
    check_parity(got, m, x_np, 1e-4)
    rt.close()


@pytest.mark.parametrize("batch", [1, 5, 16, 17, 32, 33, 100])
def test_mlp_bf16_ragged(batch):
    m = synth.mlp(3, 200, "bf16", "gelu", seed=7)
    x = synth.mlp_input(batch, 200, "bf16", 100 + batch)
    rt, (mid,) = make_runtime([m], batch_max=batch)
    log(f"mlp bf16 width 200 batch {batch}")
    got = infer(rt, mid, m, x)
    check_parity(got, m, x, 2e-2)
    rt.close()


@pytest.mark.parametrize("batch", [1, 16, 17, 32, 33, 100])
def test_mlp_bf16_blocked_weights(batch):
    # width % 128 == 0: weights stored blocked; batches up to 32 take the skinny kernel,
    # larger ones the tiled kernel, both reading the blocked layout
    m = synth.mlp(3, 384, "bf16", "gelu", seed=17)
    x = synth.mlp_input(batch, 384, "bf16", 300 + batch)
    rt, (mid,) = make_runtime([m], batch_max=batch)
    check_parity(infer(rt, mid, m, x), m, x, 2e-2)
    rt.close()


@pytest.mark.parametrize("width,batch", [(320, 100), (1088, 1030)])
def test_mlp_bf16_row_major_epilogue_prefetch(width, batch):
    # row-major weights (width % 128 != 0) whose width is a multiple of the tile: the tiled
    # kernel fetches bias values with its first operands (32 x 32 tiles at width 320, 64 x 64
    # at 1088), on batches that leave a partial tile of rows
    m = synth.mlp(3, width, "bf16", "gelu", seed=27)
    x = synth.mlp_input(batch, width, "bf16", 700 + batch)
    rt, (mid,) = make_runtime([m], batch_max=batch)
    log(f"mlp bf16 width {width} batch {batch}")
    check_parity(infer(rt, mid, m, x), m, x, 2e-2)
    rt.close()


@pytest.mark.parametrize("act", ["relu", "none", "gelu"])
def test_mlp_f32_acts(act):
    # gelu: the kernels' fp32 erf (Abramowitz-Stegun 7.1.26, |error| <= 1.5e-7) against the
    # oracle's exact one at the fp32 tolerance
    m = synth.mlp(2, 264, "f32", act, seed=3, bias_std=0.1)
    x = synth.mlp_input(3, 264, "f32", 4)
    rt, (mid,) = make_runtime([m], batch_max=3)
    check_parity(infer(rt, mid, m, x), m, x, 1e-4)
    rt.close()


@pytest.mark.parametrize("batch", [1, 8, 32])
def test_cfg2_full(batch):
    m = synth.config_model(2)
    x = synth.config_input(m, batch, 10200 + batch)
    rt, (mid,) = make_runtime([m], batch_max=batch)
    log(f"cfg2 batch {batch}: cold")
    cold = infer(rt, mid, m, x)
    warm = infer(rt, mid, m, x)
    assert np.array_equal(cold, warm)
    check_parity(cold, m, x, 2e-2)
    rt.close()


@pytest.mark.parametrize("width,batch", [(2000, 8200), (2048, 8192)])
def test_mlp_bf16_large_tiles(width, batch):
    # ceil(width/128) * ceil(batch/128) >= 1024 tiles of 128 x 128: the contraction takes the
    # 128 x 128 tile kernel; width 2000 (row-major weights, ragged in both tile dimensions)
    # and 2048 (blocked weights)
    m = synth.mlp(2, width, "bf16", "gelu", seed=23)
    x = synth.mlp_input(batch, width, "bf16", 500 + width)
    rt, (mid,) = make_runtime([m], batch_max=batch)
    log(f"mlp bf16 width {width} batch {batch}: 128 x 128 tiles")
    check_parity(infer(rt, mid, m, x), m, x, 2e-2)
    rt.close()
