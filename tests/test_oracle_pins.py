"""Pins of the CPU oracle against brute force, closed forms and special cases.

The paper prints no worked example or model output, so nothing here matches a
printed number; instead every oracle function is checked against float64 scalar
loops on tiny inputs (tests/brute.py), textbook identities, and invariants that a
dropped term, a wrong sign or index, or a transposed operand would break.
"""
import math

import numpy as np
import pytest
import torch

import synth
from oracle import ops, forward
from tests import brute

RNG = np.random.default_rng(1234)


def _r(*shape):
    return RNG.standard_normal(shape)


def _close(a, b, tol=1e-12):
    a, b = np.asarray(a, dtype=np.float64), np.asarray(b, dtype=np.float64)
    assert a.shape == b.shape, (a.shape, b.shape)
    assert np.max(np.abs(a - b)) <= tol * max(1.0, np.max(np.abs(b))), np.max(np.abs(a - b))


# ---------------------------------------------------------------- elementary ops

def test_linear_brute_3x5x7():
    x, w, b = _r(3, 5), _r(7, 5), _r(7)
    _close(ops.linear(x, w, b), brute.linear(x.tolist(), w.tolist(), b.tolist()))


def test_gelu_against_math_erf_and_identities():
    x = np.linspace(-6, 6, 97)
    _close(ops.gelu(x), [brute.gelu(v) for v in x])
    # GELU(x) - GELU(-x) = x (since Phi(x) + Phi(-x) = 1), GELU(0) = 0
    _close(ops.gelu(x) - ops.gelu(-x), x)
    assert ops.gelu(np.zeros(1))[0] == 0.0
    # Phi(1) = 0.8413447460685429 (standard normal CDF table value)
    _close(ops.gelu(np.array([1.0])), [0.8413447460685429], 1e-15)


def test_relu():
    x = np.array([-2.0, -0.0, 0.0, 3.5])
    assert ops.relu(x).tolist() == [0.0, 0.0, 0.0, 3.5]


@pytest.mark.parametrize("k,s,p", [(1, 1, 0), (1, 2, 0), (3, 1, 1), (3, 2, 1), (7, 2, 3), (3, 2, 0)])
def test_conv_brute(k, s, p):
    x, w, b = _r(2, 5, 6, 3), _r(4, k, k, 3), _r(4)
    _close(ops.conv2d_nhwc(x, w, b, s, p), brute.conv(x.tolist(), w.tolist(), b.tolist(), s, p))


def test_conv_1x1_is_gemm_and_delta_is_identity():
    x, w, b = _r(2, 4, 4, 6), _r(5, 1, 1, 6), _r(5)
    _close(ops.conv2d_nhwc(x, w, b, 1, 0), (x.reshape(-1, 6) @ w.reshape(5, 6).T + b).reshape(2, 4, 4, 5))
    d = np.zeros((6, 3, 3, 6))
    for c in range(6):
        d[c, 1, 1, c] = 1.0
    _close(ops.conv2d_nhwc(x, d, np.zeros(6), 1, 1), x)
    # stride 2 delta picks every second pixel
    _close(ops.conv2d_nhwc(x, d, np.zeros(6), 2, 1), x[:, ::2, ::2, :])


def test_maxpool_brute_with_negative_inputs():
    x = -np.abs(_r(2, 7, 6, 3)) - 0.5          # all negative: zero padding would win, -inf must not
    _close(ops.maxpool_nhwc(x, 3, 2, 1), brute.maxpool(x.tolist(), 3, 2, 1))
    assert ops.maxpool_nhwc(x, 3, 2, 1).max() < 0


def test_avgpool_brute():
    x = _r(2, 3, 5, 4)
    _close(ops.global_avgpool_nhwc(x), brute.avgpool(x.tolist()))


def test_layernorm_brute_width7_and_moments():
    x, g, b = _r(3, 7), _r(7), _r(7)
    _close(ops.layernorm(x, g, b, 1e-12), [brute.layernorm_row(r, g.tolist(), b.tolist(), 1e-12) for r in x.tolist()])
    y = ops.layernorm(x * 5 + 3, np.ones(7), np.zeros(7), 1e-12)
    _close(y.mean(axis=1), np.zeros(3), 1e-14)
    _close((y ** 2).mean(axis=1), np.ones(3), 1e-10)


def test_softmax_and_attention_brute():
    s = _r(5, 9)
    _close(ops.softmax(s).sum(axis=1), np.ones(5), 1e-15)
    _close(ops.softmax(s), [brute.softmax_row(r) for r in s.tolist()])
    q, k, v = _r(4, 3), _r(4, 3), _r(4, 3)
    _close(ops.attention(q, k, v), brute.attention(q.tolist(), k.tolist(), v.tolist()))
    # all keys equal -> uniform weights -> every output row is the mean of V
    ke = np.repeat(_r(1, 3), 4, axis=0)
    _close(ops.attention(q, ke, v), np.repeat(v.mean(axis=0, keepdims=True), 4, axis=0))


def test_multihead_head_split_brute():
    n, s, h, dh = 2, 4, 2, 3
    d = h * dh
    qkv = _r(n, s, 3 * d)
    got = ops.multihead_self_attention(qkv, h)
    for i in range(n):
        for hh in range(h):
            q = qkv[i, :, hh * dh:(hh + 1) * dh]
            k = qkv[i, :, d + hh * dh:d + (hh + 1) * dh]
            v = qkv[i, :, 2 * d + hh * dh:2 * d + (hh + 1) * dh]
            _close(got[i, :, hh * dh:(hh + 1) * dh], brute.attention(q.tolist(), k.tolist(), v.tolist()))


# ---------------------------------------------------------------- input generation

def test_bf16_round_matches_torch_and_ties_to_even():
    x = np.array([1.0, -2.5, 3.14159, 1e-30, 65504.0, 1 + 2 ** -8, 1 + 3 * 2 ** -8], dtype=np.float32)
    want = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert synth.bf16_round(x).tolist() == want.tolist()
    # 1 + 2^-8 is exactly half-way between bf16 neighbours 1 and 1 + 2^-7: ties go to the even one (1.0)
    assert synth.bf16_round(np.array([1 + 2 ** -8], np.float32))[0] == 0x3F80
    assert synth.bf16_round(np.array([1 + 3 * 2 ** -8], np.float32))[0] == 0x3F82
    y = np.random.default_rng(0).standard_normal(10000).astype(np.float32)
    assert np.array_equal(synth.bf16_round(y), torch.from_numpy(y).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16))


def test_layout_byte_counts():
    # derived by hand from the layer shapes (weights + biases, no padding)
    assert synth.config_model(1).param_bytes == 4 * (256 * 256 + 256) * 4 == 1_052_672
    assert synth.config_model(2).param_bytes == 24 * (4096 * 4096 + 4096) * 2 == 805_502_976
    r = synth.config_model(3)
    assert r.param_bytes == 25_530_472 * 2 and len(r.tensors) == 108
    assert r.param_bytes == 51_060_944
    b = synth.config_model(4)
    per_layer = (2304 * 768 + 2304 + 768 * 768 + 768 + 2 * 768 + 3072 * 768 + 3072 + 768 * 3072 + 768 + 2 * 768) * 2
    assert per_layer == 14_175_744
    assert b.param_bytes == (30522 + 512 + 2) * 768 * 2 + 2 * 768 * 2 + 12 * per_layer == 217_783_296
    for m in (synth.config_model(c) for c in (1, 2, 3, 4)):
        assert all(t.offset % synth.ALIGN == 0 for t in m.tensors)
        ends = [t.offset + t.nbytes for t in m.tensors]
        assert all(e <= o for e, o in zip(ends, [t.offset for t in m.tensors][1:]))


# ---------------------------------------------------------------- whole networks vs brute force

def _w(model, name):
    return forward._widen(model.tensor_bytes(name), model.tensor(name).dtype, np.float64).reshape(model.tensor(name).shape)


def test_mlp_tiny_brute():
    m = synth.mlp(3, 5, "f32", "relu", seed=9, bias_std=0.3)
    x = synth.mlp_input(2, 5, "f32", 11)
    h = x.astype(np.float64).tolist()
    for l in range(3):
        h = brute.linear(h, _w(m, f"l{l}.w").tolist(), _w(m, f"l{l}.b").tolist())
        if l < 2:
            h = brute.amap(brute.relu, h)
    _close(forward.mlp_forward(m, x), h)


def test_mlp_gelu_bf16_tiny_brute():
    m = synth.mlp(2, 8, "bf16", "gelu", seed=5)
    x = synth.mlp_input(3, 8, "bf16", 6)
    h = synth.bf16_to_f32(x).astype(np.float64).tolist()
    h = brute.amap(brute.gelu, brute.linear(h, _w(m, "l0.w").tolist(), _w(m, "l0.b").tolist()))
    h = brute.linear(h, _w(m, "l1.w").tolist(), _w(m, "l1.b").tolist())
    _close(forward.mlp_forward(m, x), h)


def test_mlp_identity_weights_pass_relu_through():
    m = synth.mlp(3, 4, "f32", "relu", seed=1)
    blob = m.blob()
    for l in range(3):
        t = m.tensor(f"l{l}.w")
        blob[t.offset:t.offset + t.nbytes] = np.eye(4, dtype=np.float32).reshape(-1).view(np.uint8)
    x = np.array([[1.5, -2.0, 0.25, -0.5]], np.float32)
    # two ReLU layers then a linear identity: negatives clamp to 0, positives pass
    _close(forward.mlp_forward(m, x), [[1.5, 0.0, 0.25, 0.0]])


def test_mlp_cfg1_positive_homogeneity():
    m = synth.config_model(1)
    x = synth.config_input(m, 1, 10101).astype(np.float64)   # scale in float64: no input rounding
    for a in (0.5, 3.0):
        _close(forward.mlp_forward(m, a * x), a * forward.mlp_forward(m, x), 1e-12)


def test_bert_tiny_brute():
    L, d, H, f, S, V, P = 2, 6, 2, 8, 4, 11, 7
    m = synth.bert(seed=21, layers=L, d=d, heads=H, ffn=f, seq=S, vocab=V, maxpos=P, std=0.5)
    blob = m.blob()   # non-trivial LN parameters so gamma/beta ordering is pinned
    for name in [t.name for t in m.tensors if t.role.endswith("_g") or t.role.endswith("_b") and "ln" in t.role]:
        t = m.tensor(name)
        vals = np.random.default_rng(len(name)).standard_normal(t.numel).astype(np.float32) * 0.3 + (1.0 if name.endswith(".g") else 0.0)
        blob[t.offset:t.offset + t.nbytes] = synth.bf16_round(vals).view(np.uint8)
    ids = synth.bert_input(2, 3, seq=S, vocab=V)
    g = lambda n: _w(m, n).tolist()
    out = []
    for b in range(2):
        h = [brute.add(brute.add(g("emb.tok")[ids[b, s]], g("emb.pos")[s]), g("emb.type")[0]) for s in range(S)]
        h = [brute.layernorm_row(r, g("emb.ln.g"), g("emb.ln.b"), 1e-12) for r in h]
        for l in range(1, L + 1):
            qkv = brute.linear(h, g(f"l{l}.qkv.w"), g(f"l{l}.qkv.b"))
            dh = d // H
            a = [[0.0] * d for _ in range(S)]
            for hh in range(H):
                q = [r[hh * dh:(hh + 1) * dh] for r in qkv]
                k = [r[d + hh * dh:d + (hh + 1) * dh] for r in qkv]
                v = [r[2 * d + hh * dh:2 * d + (hh + 1) * dh] for r in qkv]
                o = brute.attention(q, k, v)
                for s in range(S):
                    a[s][hh * dh:(hh + 1) * dh] = o[s]
            ao = brute.linear(a, g(f"l{l}.o.w"), g(f"l{l}.o.b"))
            h = [brute.layernorm_row(brute.add(h[s], ao[s]), g(f"l{l}.ln1.g"), g(f"l{l}.ln1.b"), 1e-12) for s in range(S)]
            f1 = brute.amap(brute.gelu, brute.linear(h, g(f"l{l}.ffn1.w"), g(f"l{l}.ffn1.b")))
            f2 = brute.linear(f1, g(f"l{l}.ffn2.w"), g(f"l{l}.ffn2.b"))
            h = [brute.layernorm_row(brute.add(h[s], f2[s]), g(f"l{l}.ln2.g"), g(f"l{l}.ln2.b"), 1e-12) for s in range(S)]
        out.append(h)
    _close(forward.bert_forward(m, ids), out, 1e-10)


def test_resnet_narrow_brute():
    stages = ((2, 2, 4, 1), (1, 3, 5, 2))
    m = synth.resnet50(seed=31, classes=3, image=16, stages=stages, stem=2, bias_std=0.3)
    x = synth.resnet_input(1, 32, image=16)
    g = lambda n: _w(m, n).tolist()

    def conv(name, t, s, p):
        return brute.conv(t, g(f"{name}.w"), g(f"{name}.b"), s, p)

    h = synth.bf16_to_f32(x).astype(np.float64).tolist()
    h = brute.amap(brute.relu, conv("conv1", h, 2, 3))
    h = brute.maxpool(h, 3, 2, 1)
    for si, (nblk, _mid, _out, _s) in enumerate(stages):
        for bi in range(nblk):
            p = f"s{si + 1}.b{bi}"
            st = 2 if (si > 0 and bi == 0) else 1      # v1.5: the stride sits on the 3x3
            t = brute.amap(brute.relu, conv(f"{p}.c1", h, 1, 0))
            t = brute.amap(brute.relu, conv(f"{p}.c2", t, st, 1))
            t = conv(f"{p}.c3", t, 1, 0)
            sc = conv(f"{p}.ds", h, st, 0) if bi == 0 else h
            h = brute.amap(brute.relu, brute.add(t, sc))
    h = brute.avgpool(h)
    y = brute.linear(h, g("fc.w"), g("fc.b"))
    _close(forward.resnet50_forward(m, x), y, 1e-10)


def test_resnet50_spatial_plan():
    # v1.5 at 224: 112 after conv1, 56 after maxpool, stage outputs 56, 28, 14, 7
    convs = synth.models.resnet50_convs()
    assert len(convs) == 53
    h = 224
    sizes = {}
    for name, co, kh, kw, ci, s, p in convs:
        if name.endswith(".ds"):
            continue
        h = (h + 2 * p - kh) // s + 1
        if name == "conv1":
            h = (h + 2 - 3) // 2 + 1  # maxpool
        sizes[name.split(".")[0]] = h
    assert sizes == {"conv1": 56, "s1": 56, "s2": 28, "s3": 14, "s4": 7}


# ---------------------------------------------------------------- precision of the oracle itself

@pytest.mark.slow
@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_oracle_fp32_matches_fp64(cfg):
    m = synth.config_model(cfg)
    x = synth.config_input(m, 1, synth.CONFIG_SEEDS[cfg][1] + (0 if cfg == 1 else 1))
    y64 = forward.forward(m, x, np.float64)
    y32 = forward.forward(m, x, np.float32)
    assert y32.dtype == np.float32
    err = forward.normwise_error(y32, y64).max()
    assert err <= 1e-5, err
    m.drop_blob()


# ---------------------------------------------------------------- the parity metric

def test_normwise_error_hand_computed():
    # Reading of "max relative error" for whole outputs: per sample (first axis),
    # ||got - ref||_inf / ||ref||_inf. Values below are worked by hand.
    ref = np.array([[1.0, -4.0, 2.0],          # sample 0: ||ref||_inf = 4 (a negative entry)
                    [0.5, 0.25, -0.125]])      # sample 1: ||ref||_inf = 0.5
    got = np.array([[1.5, -4.0, 2.0],          # |diff| max 0.5  -> 0.5 / 4   = 0.125
                    [0.5, 0.0, -0.125]])       # |diff| max 0.25 -> 0.25 / 0.5 = 0.5
    err = forward.normwise_error(got, ref)
    assert err.shape == (2,)
    assert err.tolist() == [0.125, 0.5]
    # a per-tensor denominator (4 for both samples) would give 0.0625 for sample 1,
    # and a signed maximum of ref (2 for sample 0) would give 0.25 for sample 0
    assert err[1] != 0.25 / 4.0 and err[0] != 0.5 / 2.0
    # errors of opposite sign count by magnitude: got below ref by 1 in sample 0
    got2 = ref.copy()
    got2[0, 1] = -5.0
    assert forward.normwise_error(got2, ref).tolist() == [0.25, 0.0]
    # exact agreement is exactly zero
    assert forward.normwise_error(ref, ref).tolist() == [0.0, 0.0]


def test_normwise_error_flattens_all_but_the_sample_axis():
    # [2][2][3] outputs (a BERT-like [batch][seq][d]); each sample's norm is over all its
    # elements, not per row. Sample 0: ||ref|| = 8, largest |diff| 2 -> 0.25. Sample 1:
    # ||ref|| = 3 (at -3), largest |diff| 0.75 in its second row -> 0.25.
    ref = np.zeros((2, 2, 3))
    ref[0, 0] = [8.0, 1.0, 1.0]
    ref[0, 1] = [1.0, 1.0, 1.0]
    ref[1, 0] = [1.0, -3.0, 1.0]
    ref[1, 1] = [0.5, 0.5, 0.5]
    got = ref.copy()
    got[0, 1, 2] += 2.0
    got[1, 1, 0] -= 0.75
    assert forward.normwise_error(got, ref).tolist() == [0.25, 0.25]
    # a per-row reading would have divided sample 0's error by 1 (its second row's norm)
    # and sample 1's by 0.5
    assert forward.normwise_error(got.reshape(4, 3), ref.reshape(4, 3)).tolist() == [0.0, 2.0, 0.0, 1.5]
    # float32 inputs (the GPU's outputs) are widened before the difference
    g32 = np.float32(1.0) + np.float32(2.0 ** -23)
    assert forward.normwise_error(np.array([[g32]], np.float32), np.array([[1.0]])).tolist() == [2.0 ** -23]
