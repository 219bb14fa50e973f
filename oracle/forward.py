"""Plain forward passes of the three model families (oracle; test infrastructure only).

The method executes each model exactly as written, only with its weights arriving
layer by layer (paper Sec. 4.3, "Model swapping and pipeline execution": transfer of
later layers overlaps compute of earlier ones within one forward pass). The result is
therefore the ordinary forward pass from the registered weight bytes, computed here
without intermediate rounding, in ``dt`` (float64 by default).

The model is given as a ``synth.Model`` (tensor names, shapes, dtypes and byte offsets
into its host buffer); each function checks every tensor against the shape the
architecture demands before using it.
"""
from __future__ import annotations

import numpy as np

from . import ops


def _widen(raw: np.ndarray, dtype: str, dt) -> np.ndarray:
    """Exact widening of stored bytes: fp32 as is, bf16 by placing the 16 bits on top."""
    if dtype == "f32":
        return raw.view(np.float32).astype(dt)
    u = raw.view(np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(dt)


class _Weights:
    def __init__(self, model, dt):
        self.m, self.dt, self.blob = model, dt, model.blob()

    def __call__(self, name: str, shape: tuple) -> np.ndarray:
        t = self.m.tensor(name)
        if tuple(t.shape) != tuple(shape):
            raise ValueError(f"{name}: layout shape {t.shape}, architecture needs {shape}")
        return _widen(self.blob[t.offset:t.offset + t.nbytes], t.dtype, self.dt).reshape(shape)


def _input(x: np.ndarray, model_dtype: str, dt) -> np.ndarray:
    if model_dtype == "bf16" and x.dtype == np.uint16:
        return _widen(x.reshape(-1).view(np.uint8), "bf16", dt).reshape(x.shape)
    return x.astype(dt)


def mlp_forward(model, x, dt=np.float64):
    """x_l = act(x_{l-1} W_l^T + b_l) for every layer but the last, which has no activation."""
    L, W, act = model.dims["layers"], model.dims["width"], model.dims["act"]
    w = _Weights(model, dt)
    h = _input(x, model.dtype, dt)
    f = {"relu": ops.relu, "gelu": ops.gelu, "none": (lambda t: t)}[act]
    for l in range(L):
        h = ops.linear(h, w(f"l{l}.w", (W, W)), w(f"l{l}.b", (W,)))
        if l < L - 1:
            h = f(h)
    return h


def resnet50_forward(model, x, dt=np.float64):
    """ResNet-50 v1.5 with batch-norm folded into conv biases, NHWC.

    conv1 7x7/2 pad 3 + ReLU, maxpool 3x3/2 pad 1, then stages of (3, 4, 6, 3)
    bottlenecks with (mid, out) widths (64, 256), (128, 512), (256, 1024), (512, 2048):
    1x1 -> ReLU -> 3x3 pad 1 carrying the stage stride (2 in the first block of
    stages 2-4) -> ReLU -> 1x1, plus an identity shortcut or, in each stage's first
    block, a 1x1 projection with the same stride; ReLU of the sum. Then global
    average pool and a fully connected layer to the class logits.
    """
    w = _Weights(model, dt)
    classes = model.dims["classes"]
    # narrow variants (for brute-force checks) carry their widths; the default is ResNet-50
    stages = [(n, mid, out) for n, mid, out, *_ in model.dims.get(
        "stages", ((3, 64, 256), (4, 128, 512), (6, 256, 1024), (3, 512, 2048)))]
    stem = model.dims.get("stem", 64)

    def conv(name, t, cout, k, stride, pad):
        cin = t.shape[-1]
        return ops.conv2d_nhwc(t, w(f"{name}.w", (cout, k, k, cin)), w(f"{name}.b", (cout,)), stride, pad)

    h = _input(x, "bf16", dt)
    h = ops.relu(conv("conv1", h, stem, 7, 2, 3))
    h = ops.maxpool_nhwc(h, 3, 2, 1)
    for si, (nblk, mid, out) in enumerate(stages):
        for bi in range(nblk):
            p = f"s{si + 1}.b{bi}"
            stride = 2 if (bi == 0 and si > 0) else 1
            t = ops.relu(conv(f"{p}.c1", h, mid, 1, 1, 0))
            t = ops.relu(conv(f"{p}.c2", t, mid, 3, stride, 1))
            t = conv(f"{p}.c3", t, out, 1, 1, 0)
            sc = conv(f"{p}.ds", h, out, 1, stride, 0) if bi == 0 else h
            h = ops.relu(t + sc)
    h = ops.global_avgpool_nhwc(h)
    return ops.linear(h, w("fc.w", (classes, h.shape[-1])), w("fc.b", (classes,)))


def bert_forward(model, ids, dt=np.float64):
    """BERT encoder, post-LN, no attention mask, token type 0 everywhere, LN eps 1e-12."""
    dm = model.dims
    L, d, H, f, V, P = dm["layers"], dm["d"], dm["heads"], dm["ffn"], dm["vocab"], dm["maxpos"]
    eps = 1e-12
    w = _Weights(model, dt)
    n, s = ids.shape
    h = w("emb.tok", (V, d))[ids] + w("emb.pos", (P, d))[:s][None] + w("emb.type", (2, d))[0][None, None]
    h = ops.layernorm(h, w("emb.ln.g", (d,)), w("emb.ln.b", (d,)), eps)
    for l in range(1, L + 1):
        p = f"l{l}"
        qkv = ops.linear(h, w(f"{p}.qkv.w", (3 * d, d)), w(f"{p}.qkv.b", (3 * d,)))
        a = ops.multihead_self_attention(qkv, H)
        h = ops.layernorm(h + ops.linear(a, w(f"{p}.o.w", (d, d)), w(f"{p}.o.b", (d,))),
                          w(f"{p}.ln1.g", (d,)), w(f"{p}.ln1.b", (d,)), eps)
        g = ops.gelu(ops.linear(h, w(f"{p}.ffn1.w", (f, d)), w(f"{p}.ffn1.b", (f,))))
        h = ops.layernorm(h + ops.linear(g, w(f"{p}.ffn2.w", (d, f)), w(f"{p}.ffn2.b", (d,))),
                          w(f"{p}.ln2.g", (d,)), w(f"{p}.ln2.b", (d,)), eps)
    return h


def forward(model, x, dt=np.float64):
    return {"mlp": mlp_forward, "resnet50": resnet50_forward, "bert": bert_forward}[model.arch](model, x, dt)


def normwise_error(got: np.ndarray, ref: np.ndarray) -> np.ndarray:
    """Per-sample ||got - ref||_inf / ||ref||_inf (first axis = samples)."""
    g = np.asarray(got, dtype=np.float64).reshape(got.shape[0], -1)
    r = np.asarray(ref, dtype=np.float64).reshape(ref.shape[0], -1)
    return np.abs(g - r).max(axis=1) / np.abs(r).max(axis=1)
