"""Seeded synthetic weights, layouts and inputs for the swap-in + execute workloads.

Workloads (the paper names its models, ResNet via torchvision and BERT, but ships
no weights; the synthetic stand-ins below keep the shapes and distributions):

* MLP: ``layers`` x [width x width] linear layers (weights ``[out][in]``) with biases.
* ResNet-50-shaped CNN (v1.5: stride on the 3x3), BN folded into conv biases,
  conv weights OHWI, FC ``[classes][2048]``.
* BERT-base-shaped post-LN encoder: token/position/type embeddings + LN, then
  ``L`` x {fused QKV [3d][d], O [d][d], LN1, FFN1 [f][d], FFN2 [d][f], LN2}.

Draw rule: one ``numpy.random.Generator(PCG64(seed))`` per model; tensors are drawn
in layout order, each as ``standard_normal(n, float32) * float32(std)``; constant
tensors (zero biases, LN gamma=1 / beta=0) draw nothing. bf16 tensors are rounded
from those float32 draws with round-to-nearest-even.

Layout rule: tensors are packed in first-use order, each starting at a multiple of
``ALIGN`` bytes inside one host buffer. Every tensor carries ``layer`` (its first-use
unit) and a ``role`` name.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

ALIGN = 256

# weight seeds and request-input seed bases of the five benchmark workloads
CONFIG_SEEDS = {1: (1, 10101), 2: (2, 10200), 3: (3, 10300), 4: (4, 10400)}


def bf16_round(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round to nearest, ties to even."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_to_f32(u: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> float32, exact."""
    return (np.asarray(u, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclass
class Tensor:
    name: str
    layer: int
    role: str
    shape: tuple
    dtype: str            # "f32" | "bf16"
    init: tuple           # ("normal", std) | ("const", value)
    offset: int = 0

    @property
    def numel(self) -> int:
        return int(np.prod(self.shape))

    @property
    def nbytes(self) -> int:
        return self.numel * (4 if self.dtype == "f32" else 2)


@dataclass
class Model:
    arch: str                      # "mlp" | "resnet50" | "bert"
    dtype: str                     # "f32" | "bf16"
    dims: dict
    tensors: list = field(default_factory=list)
    total_bytes: int = 0
    seed: int = 0
    _blob: np.ndarray | None = None

    def _pack(self) -> None:
        off = 0
        for t in self.tensors:
            off = (off + ALIGN - 1) // ALIGN * ALIGN
            t.offset = off
            off += t.nbytes
        self.total_bytes = (off + ALIGN - 1) // ALIGN * ALIGN

    @property
    def param_bytes(self) -> int:
        """Bytes of parameters, without alignment padding."""
        return sum(t.nbytes for t in self.tensors)

    def blob(self) -> np.ndarray:
        """The host weight buffer (uint8), drawn on first use and then cached."""
        if self._blob is None:
            self._blob = self._draw()
        return self._blob

    def drop_blob(self) -> None:
        self._blob = None

    def _draw(self) -> np.ndarray:
        rng = np.random.Generator(np.random.PCG64(self.seed))
        buf = np.zeros(self.total_bytes, dtype=np.uint8)
        for t in self.tensors:
            kind, val = t.init
            if kind == "normal":
                x = rng.standard_normal(t.numel, dtype=np.float32)
                x *= np.float32(val)
            else:
                x = np.full(t.numel, val, dtype=np.float32)
            raw = bf16_round(x).view(np.uint8) if t.dtype == "bf16" else x.view(np.uint8)
            buf[t.offset:t.offset + t.nbytes] = raw
            del x, raw
        return buf

    def tensor(self, name: str) -> Tensor:
        for t in self.tensors:
            if t.name == name:
                return t
        raise KeyError(name)

    def tensor_bytes(self, name: str) -> np.ndarray:
        t = self.tensor(name)
        return self.blob()[t.offset:t.offset + t.nbytes]

    @property
    def n_layers(self) -> int:
        return max(t.layer for t in self.tensors) + 1


def mlp(layers: int, width: int, dtype: str, act: str, seed: int,
        bias_std: float | None = None) -> Model:
    """``layers`` square linear layers; W ~ N(0, 1/width); bias 0 (fp32) or N(0, bias_std^2)."""
    m = Model("mlp", dtype, {"layers": layers, "width": width, "act": act}, seed=seed)
    if bias_std is None:
        bias_std = 0.0 if dtype == "f32" else 0.02
    for l in range(layers):
        m.tensors.append(Tensor(f"l{l}.w", l, "w", (width, width), dtype,
                                ("normal", 1.0 / math.sqrt(width))))
        binit = ("normal", bias_std) if bias_std > 0 else ("const", 0.0)
        m.tensors.append(Tensor(f"l{l}.b", l, "b", (width,), dtype, binit))
    m._pack()
    return m


RESNET50_STAGES = ((3, 64, 256, 1), (4, 128, 512, 2), (6, 256, 1024, 2), (3, 512, 2048, 2))


def resnet50_convs(stages=RESNET50_STAGES, stem: int = 64):
    """The convolutions in first-use order (53 for ResNet-50): (name, cout, kh, kw, cin, stride, pad)."""
    convs = [("conv1", stem, 7, 7, 3, 2, 3)]
    cin = stem
    for si, (nblk, mid, out, s) in enumerate(stages):
        for bi in range(nblk):
            st = s if bi == 0 else 1
            p = f"s{si + 1}.b{bi}"
            convs.append((f"{p}.c1", mid, 1, 1, cin, 1, 0))
            convs.append((f"{p}.c2", mid, 3, 3, mid, st, 1))
            convs.append((f"{p}.c3", out, 1, 1, mid, 1, 0))
            if bi == 0:
                convs.append((f"{p}.ds", out, 1, 1, cin, st, 0))
            cin = out
    return convs


def resnet50(seed: int, classes: int = 1000, image: int = 224, bias_std: float = 0.02,
             stages=RESNET50_STAGES, stem: int = 64) -> Model:
    """ResNet-50 shape; conv and FC weights He-initialised N(0, 2/fan_in), biases N(0, bias_std^2).

    ``stages``/``stem`` exist only to build narrow variants for brute-force checks."""
    m = Model("resnet50", "bf16", {"classes": classes, "image": image}, seed=seed)
    if stages != RESNET50_STAGES or stem != 64:
        m.dims.update({"stages": tuple(stages), "stem": stem})
    convs = resnet50_convs(stages, stem)
    for li, (name, co, kh, kw, ci, _s, _p) in enumerate(convs):
        fan_in = ci * kh * kw
        m.tensors.append(Tensor(f"{name}.w", li, "w", (co, kh, kw, ci), "bf16",
                                ("normal", math.sqrt(2.0 / fan_in))))
        m.tensors.append(Tensor(f"{name}.b", li, "b", (co,), "bf16", ("normal", bias_std)))
    li = len(convs)
    feat = stages[-1][2]
    m.tensors.append(Tensor("fc.w", li, "w", (classes, feat), "bf16", ("normal", math.sqrt(2.0 / feat))))
    m.tensors.append(Tensor("fc.b", li, "b", (classes,), "bf16", ("normal", bias_std)))
    m._pack()
    return m


def bert(seed: int, layers: int = 12, d: int = 768, heads: int = 12, ffn: int = 3072,
         seq: int = 128, vocab: int = 30522, maxpos: int = 512, std: float = 0.02) -> Model:
    """BERT-base shape; matrices, embeddings and biases N(0, std^2); LN gamma=1, beta=0."""
    m = Model("bert", "bf16", {"layers": layers, "d": d, "heads": heads, "ffn": ffn,
                               "seq": seq, "vocab": vocab, "maxpos": maxpos}, seed=seed)
    n = ("normal", std)
    T = m.tensors.append
    T(Tensor("emb.tok", 0, "tok_emb", (vocab, d), "bf16", n))
    T(Tensor("emb.pos", 0, "pos_emb", (maxpos, d), "bf16", n))
    T(Tensor("emb.type", 0, "type_emb", (2, d), "bf16", n))
    T(Tensor("emb.ln.g", 0, "emb_ln_g", (d,), "bf16", ("const", 1.0)))
    T(Tensor("emb.ln.b", 0, "emb_ln_b", (d,), "bf16", ("const", 0.0)))
    for l in range(1, layers + 1):
        p = f"l{l}"
        T(Tensor(f"{p}.qkv.w", l, "qkv_w", (3 * d, d), "bf16", n))
        T(Tensor(f"{p}.qkv.b", l, "qkv_b", (3 * d,), "bf16", n))
        T(Tensor(f"{p}.o.w", l, "o_w", (d, d), "bf16", n))
        T(Tensor(f"{p}.o.b", l, "o_b", (d,), "bf16", n))
        T(Tensor(f"{p}.ln1.g", l, "ln1_g", (d,), "bf16", ("const", 1.0)))
        T(Tensor(f"{p}.ln1.b", l, "ln1_b", (d,), "bf16", ("const", 0.0)))
        T(Tensor(f"{p}.ffn1.w", l, "ffn1_w", (ffn, d), "bf16", n))
        T(Tensor(f"{p}.ffn1.b", l, "ffn1_b", (ffn,), "bf16", n))
        T(Tensor(f"{p}.ffn2.w", l, "ffn2_w", (d, ffn), "bf16", n))
        T(Tensor(f"{p}.ffn2.b", l, "ffn2_b", (d,), "bf16", n))
        T(Tensor(f"{p}.ln2.g", l, "ln2_g", (d,), "bf16", ("const", 1.0)))
        T(Tensor(f"{p}.ln2.b", l, "ln2_b", (d,), "bf16", ("const", 0.0)))
    m._pack()
    return m


def config_model(cfg: int, seed: int | None = None) -> Model:
    """Benchmark workloads 1-4 at full size (weight seed from the workload table unless given)."""
    s = CONFIG_SEEDS[cfg][0] if seed is None else seed
    if cfg == 1:
        return mlp(4, 256, "f32", "relu", s)
    if cfg == 2:
        return mlp(24, 4096, "bf16", "gelu", s)
    if cfg == 3:
        return resnet50(s)
    if cfg == 4:
        return bert(s)
    raise ValueError(cfg)


def _normal(seed: int, shape) -> np.ndarray:
    rng = np.random.Generator(np.random.PCG64(seed))
    return rng.standard_normal(int(np.prod(shape)), dtype=np.float32).reshape(shape)


def mlp_input(batch: int, width: int, dtype: str, seed: int) -> np.ndarray:
    """[batch, width] N(0,1): float32, or bf16 bit patterns (uint16) for bf16 models."""
    x = _normal(seed, (batch, width))
    return x if dtype == "f32" else bf16_round(x).reshape(batch, width)


def resnet_input(batch: int, seed: int, image: int = 224) -> np.ndarray:
    """NHWC [batch, image, image, 3] N(0,1) as bf16 bit patterns."""
    return bf16_round(_normal(seed, (batch, image, image, 3))).reshape(batch, image, image, 3)


def bert_input(batch: int, seed: int, seq: int = 128, vocab: int = 30522) -> np.ndarray:
    """int32 token ids [batch, seq] uniform in [0, vocab)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return rng.integers(0, vocab, size=(batch, seq), dtype=np.int32)


def config_input(model: Model, batch: int, seed: int) -> np.ndarray:
    if model.arch == "mlp":
        return mlp_input(batch, model.dims["width"], model.dtype, seed)
    if model.arch == "resnet50":
        return resnet_input(batch, seed, model.dims["image"])
    if model.arch == "bert":
        return bert_input(batch, seed, model.dims["seq"], model.dims["vocab"])
    raise ValueError(model.arch)
