"""Plain definitions of the layer operations (oracle; test infrastructure only).

The paper runs stock framework layers (appendix A.1, Table "cuda_api": cuBLAS GEMMs,
cuDNN convolutions, batch-norm inference, framework elementwise kernels). Each function
here is the textbook definition of one such layer, written for readability, in the
precision of its inputs (callers pass float64 or float32 arrays).
"""
from __future__ import annotations

import numpy as np
from scipy.special import erf


def linear(x, w, b):
    """y = x W^T + b, W stored [out][in] (the layout of a framework linear layer)."""
    return x @ w.T + b


def relu(x):
    return np.maximum(x, 0)


def gelu(x):
    """Exact GELU: x * Phi(x) = x/2 * (1 + erf(x / sqrt 2))."""
    return 0.5 * x * (1.0 + erf(x / np.sqrt(x.dtype.type(2.0))))


def conv2d_nhwc(x, w, b, stride: int, pad: int):
    """2-D cross-correlation with zero padding, NHWC input, OHWI weights.

    y[n, i, j, o] = b[o] + sum_{p, q, c} xpad[n, i*stride + p, j*stride + q, c] * w[o, p, q, c],
    with output size floor((H + 2 pad - k) / stride) + 1. The sum over the kernel taps
    (p, q) is taken one tap at a time; the sum over channels c is a matrix product.
    """
    n, h, wd, c = x.shape
    o, kh, kw, c2 = w.shape
    assert c == c2, (x.shape, w.shape)
    ho = (h + 2 * pad - kh) // stride + 1
    wo = (wd + 2 * pad - kw) // stride + 1
    xp = np.zeros((n, h + 2 * pad, wd + 2 * pad, c), dtype=x.dtype)
    xp[:, pad:pad + h, pad:pad + wd, :] = x
    y = np.zeros((n, ho, wo, o), dtype=x.dtype)
    for p in range(kh):
        for q in range(kw):
            patch = xp[:, p:p + stride * (ho - 1) + 1:stride, q:q + stride * (wo - 1) + 1:stride, :]
            y += patch @ w[:, p, q, :].T
    return y + b


def maxpool_nhwc(x, k: int, stride: int, pad: int):
    """Max over k x k windows; padded positions never win (they are -inf)."""
    n, h, wd, c = x.shape
    ho = (h + 2 * pad - k) // stride + 1
    wo = (wd + 2 * pad - k) // stride + 1
    xp = np.full((n, h + 2 * pad, wd + 2 * pad, c), -np.inf, dtype=x.dtype)
    xp[:, pad:pad + h, pad:pad + wd, :] = x
    y = np.full((n, ho, wo, c), -np.inf, dtype=x.dtype)
    for p in range(k):
        for q in range(k):
            y = np.maximum(y, xp[:, p:p + stride * (ho - 1) + 1:stride, q:q + stride * (wo - 1) + 1:stride, :])
    return y


def global_avgpool_nhwc(x):
    """Mean over the spatial positions: [N, H, W, C] -> [N, C]."""
    return x.mean(axis=(1, 2))


def layernorm(x, g, b, eps: float):
    """(x - mean) / sqrt(var + eps) * g + b over the last axis, population variance."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * g + b


def softmax(s):
    """Row softmax exp(s_j) / sum_k exp(s_k); the row max is subtracted first (exact identity)."""
    e = np.exp(s - s.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def attention(q, k, v):
    """Scaled dot-product attention softmax(Q K^T / sqrt(d)) V over the last two axes, no mask."""
    d = q.shape[-1]
    s = (q @ np.swapaxes(k, -1, -2)) / np.sqrt(q.dtype.type(d))
    return softmax(s) @ v


def multihead_self_attention(qkv, heads: int):
    """qkv [N, S, 3*D] with columns Q (heads x dh), K, V -> [N, S, D] heads concatenated."""
    n, s, three_d = qkv.shape
    d = three_d // 3
    dh = d // heads

    def split(t):  # [N, S, D] -> [N, heads, S, dh]
        return t.reshape(n, s, heads, dh).transpose(0, 2, 1, 3)

    q, k, v = split(qkv[..., :d]), split(qkv[..., d:2 * d]), split(qkv[..., 2 * d:])
    a = attention(q, k, v)                       # [N, heads, S, dh]
    return a.transpose(0, 2, 1, 3).reshape(n, s, d)
