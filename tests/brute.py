"""Scalar-loop float64 implementations used to pin the oracle on tiny inputs.

Every sum is a ``math.fsum`` over explicitly indexed terms; nothing here is vectorised,
so a dropped term, a transposed operand or a wrong stride in the oracle shows up as a
mismatch.
"""
import math


def linear(x, w, b):
    n, k = len(x), len(x[0])
    o = len(w)
    return [[math.fsum([x[i][c] * w[j][c] for c in range(k)]) + b[j] for j in range(o)] for i in range(n)]


def relu(v):
    return v if v > 0 else 0.0


def gelu(v):
    return 0.5 * v * (1.0 + math.erf(v / math.sqrt(2.0)))


def conv(x, w, b, stride, pad):
    """x[n][h][w][c], w[o][kh][kw][c] -> y[n][ho][wo][o]."""
    N, H, W, C = len(x), len(x[0]), len(x[0][0]), len(x[0][0][0])
    O, KH, KW = len(w), len(w[0]), len(w[0][0])
    Ho, Wo = (H + 2 * pad - KH) // stride + 1, (W + 2 * pad - KW) // stride + 1
    y = [[[[0.0] * O for _ in range(Wo)] for _ in range(Ho)] for _ in range(N)]
    for n in range(N):
        for i in range(Ho):
            for j in range(Wo):
                for o in range(O):
                    terms = []
                    for p in range(KH):
                        for q in range(KW):
                            hh, ww = i * stride - pad + p, j * stride - pad + q
                            if 0 <= hh < H and 0 <= ww < W:
                                for c in range(C):
                                    terms.append(x[n][hh][ww][c] * w[o][p][q][c])
                    y[n][i][j][o] = math.fsum(terms) + b[o]
    return y


def maxpool(x, k, stride, pad):
    N, H, W, C = len(x), len(x[0]), len(x[0][0]), len(x[0][0][0])
    Ho, Wo = (H + 2 * pad - k) // stride + 1, (W + 2 * pad - k) // stride + 1
    y = [[[[None] * C for _ in range(Wo)] for _ in range(Ho)] for _ in range(N)]
    for n in range(N):
        for i in range(Ho):
            for j in range(Wo):
                for c in range(C):
                    best = -math.inf
                    for p in range(k):
                        for q in range(k):
                            hh, ww = i * stride - pad + p, j * stride - pad + q
                            if 0 <= hh < H and 0 <= ww < W:
                                best = max(best, x[n][hh][ww][c])
                    y[n][i][j][c] = best
    return y


def avgpool(x):
    N, H, W, C = len(x), len(x[0]), len(x[0][0]), len(x[0][0][0])
    return [[math.fsum([x[n][i][j][c] for i in range(H) for j in range(W)]) / (H * W) for c in range(C)]
            for n in range(N)]


def layernorm_row(r, g, b, eps):
    n = len(r)
    mu = math.fsum(r) / n
    var = math.fsum([(v - mu) ** 2 for v in r]) / n
    return [(r[i] - mu) / math.sqrt(var + eps) * g[i] + b[i] for i in range(n)]


def softmax_row(r):
    m = max(r)
    e = [math.exp(v - m) for v in r]
    s = math.fsum(e)
    return [v / s for v in e]


def attention(q, k, v):
    """q[s][d], k[t][d], v[t][e] (one head) -> [s][e]."""
    d = len(q[0])
    out = []
    for i in range(len(q)):
        sc = [math.fsum([q[i][c] * k[j][c] for c in range(d)]) / math.sqrt(d) for j in range(len(k))]
        p = softmax_row(sc)
        out.append([math.fsum([p[j] * v[j][e] for j in range(len(k))]) for e in range(len(v[0]))])
    return out


def add(a, b):
    if isinstance(a, list):
        return [add(x, y) for x, y in zip(a, b)]
    return a + b


def amap(f, a):
    if isinstance(a, list):
        return [amap(f, x) for x in a]
    return f(a)
