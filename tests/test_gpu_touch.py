"""The warm requests' cache touch (a read of the model's weights on the execution stream,
alongside the request's own kernels) through the C ABI: which requests touch, under the
default policy, TP_FLAG_TOUCH_ALWAYS and TP_FLAG_NO_TOUCH, and that it changes no result."""
import numpy as np
import pytest

import paper_2306_03622_amd as tp
import synth
from tests.common import check_parity, infer, log, make_runtime, out_shape, to_device, torch_dev

pytestmark = pytest.mark.gpu


def _models():
    # ResNet-50 (47 MB at 10 classes) and a 4-layer BERT (25 MB past its token table) lie within
    # the touch bounds; MLPs are never touched
    return [synth.resnet50(seed=61, classes=10, image=32),
            synth.bert(seed=62, layers=4, d=512, heads=8, ffn=2048, seq=64, vocab=1000, maxpos=64),
            synth.mlp(2, 1024, "bf16", "gelu", seed=63)]


def _inputs(ms):
    return [synth.resnet_input(1, 64, image=32), synth.bert_input(1, 65, seq=64, vocab=1000),
            synth.mlp_input(1, 1024, "bf16", 66)]


# model index per request: misses at the first request of each model
SEQUENCE = [0, 0, 1, 0, 1, 1, 2, 2, 0]
# requests that touch under the default policy: hits whose model differs from the previous
# request's (requests 3, 4 and 8); under TP_FLAG_TOUCH_ALWAYS every hit of ResNet or BERT
EXPECTED = {0: 3, tp.TP_FLAG_TOUCH_ALWAYS: 5, tp.TP_FLAG_NO_TOUCH: 0}


@pytest.mark.parametrize("flags", [0, tp.TP_FLAG_TOUCH_ALWAYS, tp.TP_FLAG_NO_TOUCH])
def test_cache_touch_policy_and_results(flags):
    ms, xs = _models(), _inputs(_models())
    rt, ids = make_runtime(ms, batch_max=1, flags=flags)
    log(f"cache touch, flags {flags}")
    outs = [[] for _ in ms]
    for k in SEQUENCE:
        outs[k].append(infer(rt, ids[k], ms[k], xs[k]))
    st = rt.stats()
    assert st["cache_touches"] == EXPECTED[flags], st
    assert (st["hits"], st["misses"]) == (6, 3), st
    for k, m in enumerate(ms):
        for o in outs[k][1:]:
            assert np.array_equal(o, outs[k][0])
        check_parity(outs[k][0], m, xs[k], 2e-2)
    rt.close()


def test_cache_touch_after_explicit_swap_in():
    # a model that tp_swap_in brought in was written by the copy engine and read by nothing, so
    # its next request touches even though the same model was served last; the touch waits for
    # the copies, which are still in flight when the request is made here
    ms, xs = _models()[:1], _inputs(_models())[:1]
    rt, (mid,) = make_runtime(ms, batch_max=1)
    torch, dev = torch_dev()
    s = torch.cuda.Stream(device=dev)
    want = infer(rt, mid, ms[0], xs[0])            # the miss: no touch
    assert np.array_equal(infer(rt, mid, ms[0], xs[0]), want)
    assert rt.stats()["cache_touches"] == 0
    x = to_device(xs[0])
    for rep in range(2):
        out = torch.full(out_shape(ms[0], 1), float("nan"), dtype=torch.float32, device=dev)
        torch.cuda.synchronize()
        rt.evict(mid)
        rt.swap_in(mid, stream=s)
        rt.infer(mid, x, out, stream=s)
        s.synchronize()
        assert np.array_equal(out.cpu().numpy(), want)
        assert rt.stats()["cache_touches"] == rep + 1
        assert np.array_equal(infer(rt, mid, ms[0], xs[0]), want)   # read since: no touch
        assert rt.stats()["cache_touches"] == rep + 1
    rt.close()


def test_cache_touch_leaves_noalloc_requests_alone():
    # tp_infer_noalloc (for callers that may be capturing their stream) never touches
    ms, xs = _models()[:2], _inputs(_models())[:2]
    rt, ids = make_runtime(ms, batch_max=1, flags=tp.TP_FLAG_TOUCH_ALWAYS)
    torch, dev = torch_dev()
    s = torch.cuda.Stream(device=dev)
    want = [infer(rt, ids[k], ms[k], xs[k]) for k in (0, 1)]
    touches = rt.stats()["cache_touches"]
    for k in (0, 1, 0):
        x = to_device(xs[k])
        out = torch.full(out_shape(ms[k], 1), float("nan"), dtype=torch.float32, device=dev)
        torch.cuda.synchronize()
        rt.infer_noalloc(ids[k], x, out, stream=s)
        s.synchronize()
        assert np.array_equal(out.cpu().numpy(), want[k])
    assert rt.stats()["cache_touches"] == touches
    rt.close()
