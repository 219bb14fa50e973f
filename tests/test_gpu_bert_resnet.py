"""BERT and ResNet families through the C ABI on the GPU vs the oracle (bf16: 2e-2)."""
import numpy as np
import pytest

import synth
from tests.common import check_parity, infer, log, make_runtime, out_shape, to_device, torch_dev

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("seq,batch", [(32, 1), (64, 3), (96, 2), (256, 1)])
def test_bert_small(seq, batch):
    m = synth.bert(seed=41, layers=2, d=128, heads=2, ffn=264, seq=seq, vocab=1000, maxpos=256)
    ids = synth.bert_input(batch, 42 + seq, seq=seq, vocab=1000)
    rt, (mid,) = make_runtime([m], batch_max=batch)
    log(f"bert small seq {seq} batch {batch}")
    check_parity(infer(rt, mid, m, ids), m, ids, 2e-2)
    rt.close()


@pytest.mark.parametrize("d", [128, 256, 512])
def test_bert_split_reduction_with_layernorm(d):
    # FFN2 (K = 2048: 32 k-stages over 2 x d/64 tiles) is split over k here, so the second
    # LayerNorm of each layer runs with its reduction: in registers for widths 256 and 512,
    # as the plain reduction followed by a LayerNorm launch for width 128. Cold and warm
    # requests agree bitwise; both match the oracle.
    m = synth.bert(seed=45, layers=2, d=d, heads=d // 64, ffn=2048, seq=64, vocab=500, maxpos=64)
    ids = synth.bert_input(2, 46, seq=64, vocab=500)
    rt, (mid,) = make_runtime([m], batch_max=2)
    log(f"bert d {d}: split FFN2 with LayerNorm")
    cold = infer(rt, mid, m, ids)
    assert np.array_equal(cold, infer(rt, mid, m, ids))
    check_parity(cold, m, ids, 2e-2)
    rt.close()


def test_bert_out_of_range_ids_are_clamped():
    m = synth.bert(seed=43, layers=1, d=64, heads=1, ffn=64, seq=32, vocab=50, maxpos=32)
    ids = synth.bert_input(1, 44, seq=32, vocab=50)
    bad = ids.copy()
    bad[0, :4] = [-5, 50, 1 << 30, -(1 << 30)]
    clamped = np.clip(bad, 0, 49).astype(np.int32)
    rt, (mid,) = make_runtime([m], batch_max=1)
    assert np.array_equal(infer(rt, mid, m, bad), infer(rt, mid, m, clamped))
    rt.close()


@pytest.mark.parametrize("batch", [1, 8])
def test_cfg4_full(batch):
    m = synth.config_model(4)
    ids = synth.config_input(m, batch, 10400 + batch)
    rt, (mid,) = make_runtime([m], batch_max=batch)
    log(f"cfg4 batch {batch}")
    cold = infer(rt, mid, m, ids)
    assert np.array_equal(cold, infer(rt, mid, m, ids))
    check_parity(cold, m, ids, 2e-2)
    rt.close()


@pytest.mark.parametrize("image,batch", [(32, 1), (64, 3), (96, 2), (160, 1)])
def test_resnet_small_images(image, batch):
    m = synth.resnet50(seed=51, classes=10, image=image)
    x = synth.resnet_input(batch, 52, image=image)
    rt, (mid,) = make_runtime([m], batch_max=batch)
    log(f"resnet image {image} batch {batch}")
    check_parity(infer(rt, mid, m, x), m, x, 2e-2)
    rt.close()


@pytest.mark.parametrize("image,batch", [(64, 2), (224, 1), (224, 8)])
def test_resnet_input_alignment_paths(image, batch):
    # the stem stages its input rows as 16-byte vectors when the image is 16-byte aligned and
    # element by element otherwise: an input one element into a buffer takes the second path;
    # both give the oracle's result and the same bits
    torch, dev = torch_dev()
    m = synth.resnet50(seed=53, classes=10, image=image)
    x = synth.resnet_input(batch, 54, image=image)
    rt, (mid,) = make_runtime([m], batch_max=batch)
    aligned = infer(rt, mid, m, x)
    check_parity(aligned, m, x, 2e-2)
    flat = to_device(x).reshape(-1)
    buf = torch.zeros(flat.numel() + 8, dtype=flat.dtype, device=dev)
    buf[1:1 + flat.numel()] = flat
    xs = buf[1:1 + flat.numel()].view(x.shape)
    assert xs.data_ptr() % 16 == 2
    s = torch.cuda.Stream(device=dev)
    # warm requests alternate between the unaligned and an aligned input: the cached graph
    # is captured afresh whenever the input's alignment changes (its stem kernel was chosen by
    # the captured one's), and repointed when it does not
    xa = to_device(x)
    assert xa.data_ptr() % 16 == 0
    for k, xin in enumerate((xs, xa, xs, xs)):
        out = torch.full(out_shape(m, batch), float("nan"), dtype=torch.float32, device=dev)
        torch.cuda.synchronize()
        rt.infer(mid, xin, out, stream=s)
        s.synchronize()
        assert np.array_equal(out.cpu().numpy(), aligned), k
    st = rt.stats()
    assert (st["graph_captures"], st["graph_repoints"]) == (3, 1), st
    rt.close()


@pytest.mark.parametrize("batch", [1, 8])
def test_cfg3_full(batch):
    m = synth.config_model(3)
    x = synth.config_input(m, batch, 10300 + batch)
    rt, (mid,) = make_runtime([m], batch_max=batch)
    log(f"cfg3 batch {batch}")
    cold = infer(rt, mid, m, x)
    assert np.array_equal(cold, infer(rt, mid, m, x))
    check_parity(cold, m, x, 2e-2)
    rt.close()
