"""Seeded network definitions (layer graphs plus random weights).

A network is a list of layers in topological order.  Each layer is one
convolution (PyTorch ``conv2d`` geometry: weight ``[Cout, Cin/groups, kh,
kw]``, stride, zero padding, dilation 1) with an optional residual input
added to its pre-activation, an optional activation and an optional
max-pool after the activation.  ``src`` names the producer of the layer's
input (-1 is the network input); ``residual_src`` names the producer whose
output is added before the activation (-2 = none, -1 = network input).
The last layer is the network output.

Weights are drawn in float32 from numpy's PCG64 generator and rounded to
the storage dtype with PyTorch's conversion, so both the oracle and the
GPU path read identical values.
"""

from dataclasses import dataclass, field
from typing import List, Optional, Tuple

import numpy as np
import torch

ACT_NONE, ACT_RELU, ACT_SILU = 0, 1, 2

_TORCH_DTYPES = {"f32": torch.float32, "f16": torch.float16,
                 "bf16": torch.bfloat16}


def torch_dtype(dtype: str) -> torch.dtype:
    return _TORCH_DTYPES[dtype]


def to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round float values to ``dtype`` (PyTorch's round-to-nearest-even
    conversion) and return them as float32."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(_TORCH_DTYPES[dtype]).to(torch.float32).numpy()


@dataclass
class LayerSpec:
    src: int
    c_in: int
    c_out: int
    k: Tuple[int, int] = (3, 3)
    s: Tuple[int, int] = (1, 1)
    p: Tuple[int, int] = (1, 1)
    groups: int = 1
    act: int = ACT_RELU
    residual_src: int = -2
    pool_k: Tuple[int, int] = (0, 0)
    pool_s: Tuple[int, int] = (0, 0)
    pool_p: Tuple[int, int] = (0, 0)
    se_mid: int = 0
    weight: Optional[np.ndarray] = None   # [Cout, Cin/groups, kh, kw] f32
    bias: Optional[np.ndarray] = None     # [Cout] f32
    # squeeze-excitation after the activation (se_mid > 0):
    # s = sigmoid(se_w2 @ silu(se_w1 @ mean_hw(a) + se_b1) + se_b2)
    se_w1: Optional[np.ndarray] = None    # [se_mid, Cout]
    se_b1: Optional[np.ndarray] = None    # [se_mid]
    se_w2: Optional[np.ndarray] = None    # [Cout, se_mid]
    se_b2: Optional[np.ndarray] = None    # [Cout]
    name: str = ""


@dataclass
class NetSpec:
    name: str
    layers: List[LayerSpec]
    batch: int
    H: int
    W: int
    C: int
    dtype: str = "f32"
    meta: dict = field(default_factory=dict)


def _finish(layers: List[LayerSpec], dtype: str) -> None:
    for L in layers:
        L.weight = to_storage(L.weight, dtype)
        L.bias = to_storage(L.bias, dtype)
        if L.se_mid:
            L.se_w1 = to_storage(L.se_w1, dtype)
            L.se_b1 = to_storage(L.se_b1, dtype)
            L.se_w2 = to_storage(L.se_w2, dtype)
            L.se_b2 = to_storage(L.se_b2, dtype)


def toy_net(seed: int = 1000, dtype: str = "f32", H: int = 64, W: int = 64,
            batch: int = 1) -> NetSpec:
    """One 3x3 conv (stride 1, pad 1, 16->16) + ReLU, then a 1x1 conv
    16->32 (the toy encoder of a single conv layer followed by a per-pixel
    linear layer).  Weights and biases ~ N(0, 0.1) (standard deviation)."""
    rng = np.random.default_rng(seed)
    l0 = LayerSpec(src=-1, c_in=16, c_out=16, k=(3, 3), s=(1, 1), p=(1, 1),
                   act=ACT_RELU, name="conv3x3")
    l0.weight = rng.normal(0.0, 0.1, (16, 16, 3, 3)).astype(np.float32)
    l0.bias = rng.normal(0.0, 0.1, (16,)).astype(np.float32)
    l1 = LayerSpec(src=0, c_in=16, c_out=32, k=(1, 1), s=(1, 1), p=(0, 0),
                   act=ACT_NONE, name="conv1x1")
    l1.weight = rng.normal(0.0, 0.1, (32, 16, 1, 1)).astype(np.float32)
    l1.bias = rng.normal(0.0, 0.1, (32,)).astype(np.float32)
    layers = [l0, l1]
    _finish(layers, dtype)
    return NetSpec("toy", layers, batch, H, W, 16, dtype)


def _he(rng, cout, cin_g, kh, kw, scale=1.0):
    std = np.sqrt(2.0 / (cin_g * kh * kw)) * scale
    return rng.normal(0.0, std, (cout, cin_g, kh, kw)).astype(np.float32)


def crnn_vgg_net(seed: int = 1001, dtype: str = "f32", H: int = 32,
                 W: int = 128, batch: int = 1) -> NetSpec:
    """CRNN-style VGG text-line encoder: seven 3x3 convs (64, 128, 256,
    256, 512, 512, 512 channels, pad 1, ReLU) with 2x2/2 max-pools after
    convs 1 and 2 and (2,1)/(2,1) max-pools after convs 4 and 6, on a
    single-channel line image.  He-normal weights, biases ~ N(0, 0.01)."""
    rng = np.random.default_rng(seed)
    chans = [64, 128, 256, 256, 512, 512, 512]
    pools = {0: ((2, 2), (2, 2)), 1: ((2, 2), (2, 2)),
             3: ((2, 1), (2, 1)), 5: ((2, 1), (2, 1))}
    layers, cin = [], 1
    for i, c in enumerate(chans):
        L = LayerSpec(src=i - 1, c_in=cin, c_out=c, k=(3, 3), s=(1, 1),
                      p=(1, 1), act=ACT_RELU, name=f"conv{i + 1}")
        if i in pools:
            L.pool_k, L.pool_s = pools[i]
            L.pool_p = (0, 0)
        L.weight = _he(rng, c, cin, 3, 3)
        L.bias = rng.normal(0.0, 0.01, (c,)).astype(np.float32)
        layers.append(L)
        cin = c
    _finish(layers, dtype)
    return NetSpec("crnn_vgg", layers, batch, H, W, 1, dtype)


def resnet_net(seed: int, dtype: str, H: int, W: int, batch: int,
               blocks=(3, 4, 6, 3), widths=(64, 128, 256, 512),
               stem: int = 64, expansion: int = 4,
               name: str = "resnet") -> NetSpec:
    """ResNet v1.5 bottleneck encoder (stride on the 3x3 conv of the first
    block of stages 2-4), batch norm folded into conv biases.  Stem: 7x7/2
    conv + ReLU + 3x3/2 max-pool (pad 1).  He-normal weights, the last conv
    of every residual branch scaled by 0.2, biases ~ N(0, 0.02).  The
    classifier head is not part of the encoder."""
    rng = np.random.default_rng(seed)
    layers: List[LayerSpec] = []

    def add(L: LayerSpec) -> int:
        layers.append(L)
        return len(layers) - 1

    st = LayerSpec(src=-1, c_in=3, c_out=stem, k=(7, 7), s=(2, 2), p=(3, 3),
                   act=ACT_RELU, pool_k=(3, 3), pool_s=(2, 2), pool_p=(1, 1),
                   name="stem")
    st.weight = _he(rng, stem, 3, 7, 7)
    st.bias = rng.normal(0.0, 0.02, (stem,)).astype(np.float32)
    prev, cin = add(st), stem
    for si, (nb, w) in enumerate(zip(blocks, widths)):
        cout = w * expansion
        for b in range(nb):
            stride = 2 if (si > 0 and b == 0) else 1
            block_in = prev
            c1 = LayerSpec(src=block_in, c_in=cin, c_out=w, k=(1, 1),
                           s=(1, 1), p=(0, 0), act=ACT_RELU,
                           name=f"s{si + 1}b{b}c1")
            c1.weight = _he(rng, w, cin, 1, 1)
            c1.bias = rng.normal(0.0, 0.02, (w,)).astype(np.float32)
            i1 = add(c1)
            c2 = LayerSpec(src=i1, c_in=w, c_out=w, k=(3, 3),
                           s=(stride, stride), p=(1, 1), act=ACT_RELU,
                           name=f"s{si + 1}b{b}c2")
            c2.weight = _he(rng, w, w, 3, 3)
            c2.bias = rng.normal(0.0, 0.02, (w,)).astype(np.float32)
            i2 = add(c2)
            res = block_in
            if b == 0:
                ds = LayerSpec(src=block_in, c_in=cin, c_out=cout, k=(1, 1),
                               s=(stride, stride), p=(0, 0), act=ACT_NONE,
                               name=f"s{si + 1}b{b}ds")
                ds.weight = _he(rng, cout, cin, 1, 1)
                ds.bias = rng.normal(0.0, 0.02, (cout,)).astype(np.float32)
                res = add(ds)
            c3 = LayerSpec(src=i2, c_in=w, c_out=cout, k=(1, 1), s=(1, 1),
                           p=(0, 0), act=ACT_RELU, residual_src=res,
                           name=f"s{si + 1}b{b}c3")
            c3.weight = _he(rng, cout, w, 1, 1, scale=0.2)
            c3.bias = rng.normal(0.0, 0.02, (cout,)).astype(np.float32)
            prev = add(c3)
            cin = cout
    _finish(layers, dtype)
    return NetSpec(name, layers, batch, H, W, 3, dtype)


def resnet50_net(seed: int = 1003, dtype: str = "bf16", H: int = 1024,
                 W: int = 2048, batch: int = 1) -> NetSpec:
    """ResNet-50 encoder (bottleneck blocks 3-4-6-3, widths 64-512, output
    2048 channels at stride 32)."""
    return resnet_net(seed, dtype, H, W, batch, name="resnet50")


def resnet_mini_net(seed: int = 1013, dtype: str = "f32", H: int = 32,
                    W: int = 48, batch: int = 1) -> NetSpec:
    """A two-stage ResNet with the same layer kinds as ResNet-50 (7x7/2
    stem, overlapping 3x3/2 pool, bottlenecks, strided 3x3, downsample
    shortcut and identity shortcut) at small widths, for fast tests."""
    return resnet_net(seed, dtype, H, W, batch, blocks=(2, 1),
                      widths=(8, 16), stem=8, expansion=4,
                      name="resnet_mini")


def depthwise_test_net(seed: int = 1021, dtype: str = "f32", H: int = 24,
                       W: int = 40, batch: int = 1, C: int = 16) -> NetSpec:
    """Pointwise expand + depthwise 3x3 (SiLU) + depthwise 5x5 stride 2
    (SiLU) + linear pointwise project: the depthwise layer kinds of an
    inverted-residual stack, without squeeze-excitation."""
    rng = np.random.default_rng(seed)
    E = 4 * C
    l0 = LayerSpec(src=-1, c_in=C, c_out=E, k=(1, 1), s=(1, 1), p=(0, 0),
                   act=ACT_SILU, name="expand")
    l0.weight = _he(rng, E, C, 1, 1)
    l1 = LayerSpec(src=0, c_in=E, c_out=E, k=(3, 3), s=(1, 1), p=(1, 1),
                   groups=E, act=ACT_SILU, name="dw3")
    l1.weight = _he(rng, E, 1, 3, 3)
    l2 = LayerSpec(src=1, c_in=E, c_out=E, k=(5, 5), s=(2, 2), p=(2, 2),
                   groups=E, act=ACT_SILU, name="dw5s2")
    l2.weight = _he(rng, E, 1, 5, 5)
    l3 = LayerSpec(src=2, c_in=E, c_out=C, k=(1, 1), s=(1, 1), p=(0, 0),
                   act=ACT_NONE, name="project")
    l3.weight = _he(rng, C, E, 1, 1, scale=0.5)
    layers = [l0, l1, l2, l3]
    for L in layers:
        L.bias = rng.normal(0.0, 0.02, (L.c_out,)).astype(np.float32)
    _finish(layers, dtype)
    return NetSpec("dw_test", layers, batch, H, W, C, dtype)


# EfficientNet-B0 stage table: expansion t, kernel k, stride s, channels c,
# repeats n.
B0_STAGES = [(1, 3, 1, 16, 1), (6, 3, 2, 24, 2), (6, 5, 2, 40, 2),
             (6, 3, 2, 80, 3), (6, 5, 1, 112, 3), (6, 5, 2, 192, 4),
             (6, 3, 1, 320, 1)]


def efficientnet_net(seed: int = 1005, dtype: str = "f16", H: int = 512,
                     W: int = 512, batch: int = 1, stages=None,
                     stem: int = 32, name: str = "efficientnet_b0") -> NetSpec:
    """EfficientNet-B0 backbone (no head): 3x3/2 stem conv + SiLU, then
    inverted-residual blocks (MBConv): 1x1 expand + SiLU (t > 1), depthwise
    kxk/s + SiLU + squeeze-excitation (reduction to 1/4 of the block's
    input channels, SiLU, sigmoid gate), linear 1x1 project, identity skip
    when stride 1 and channels match.  Batch norm folded; He-normal
    weights (projection scaled by 0.5), biases ~ N(0, 0.02)."""
    rng = np.random.default_rng(seed)
    stages = B0_STAGES if stages is None else stages
    layers: List[LayerSpec] = []

    def add(L):
        layers.append(L)
        return len(layers) - 1

    st = LayerSpec(src=-1, c_in=3, c_out=stem, k=(3, 3), s=(2, 2), p=(1, 1),
                   act=ACT_SILU, name="stem")
    st.weight = _he(rng, stem, 3, 3, 3)
    st.bias = rng.normal(0.0, 0.02, (stem,)).astype(np.float32)
    prev, cin = add(st), stem
    for si, (t, k, s_, c, n) in enumerate(stages):
        for b in range(n):
            stride = s_ if b == 0 else 1
            block_in, mid = prev, cin * t
            src = block_in
            if t != 1:
                ex = LayerSpec(src=block_in, c_in=cin, c_out=mid, k=(1, 1),
                               s=(1, 1), p=(0, 0), act=ACT_SILU,
                               name=f"b{si}{b}_expand")
                ex.weight = _he(rng, mid, cin, 1, 1)
                ex.bias = rng.normal(0.0, 0.02, (mid,)).astype(np.float32)
                src = add(ex)
            se = max(1, int(cin * 0.25))
            dw = LayerSpec(src=src, c_in=mid, c_out=mid, k=(k, k),
                           s=(stride, stride), p=(k // 2, k // 2), groups=mid,
                           act=ACT_SILU, se_mid=se, name=f"b{si}{b}_dw")
            dw.weight = _he(rng, mid, 1, k, k)
            dw.bias = rng.normal(0.0, 0.02, (mid,)).astype(np.float32)
            dw.se_w1 = rng.normal(0.0, np.sqrt(2.0 / mid),
                                  (se, mid)).astype(np.float32)
            dw.se_b1 = rng.normal(0.0, 0.02, (se,)).astype(np.float32)
            dw.se_w2 = rng.normal(0.0, np.sqrt(1.0 / se),
                                  (mid, se)).astype(np.float32)
            dw.se_b2 = rng.normal(1.0, 0.2, (mid,)).astype(np.float32)
            d_i = add(dw)
            pr = LayerSpec(src=d_i, c_in=mid, c_out=c, k=(1, 1), s=(1, 1),
                           p=(0, 0), act=ACT_NONE,
                           residual_src=(block_in if (stride == 1 and
                                                      cin == c) else -2),
                           name=f"b{si}{b}_project")
            pr.weight = _he(rng, c, mid, 1, 1, scale=0.5)
            pr.bias = rng.normal(0.0, 0.02, (c,)).astype(np.float32)
            prev = add(pr)
            cin = c
    _finish(layers, dtype)
    return NetSpec(name, layers, batch, H, W, 3, dtype)


def efficientnet_mini_net(seed: int = 1015, dtype: str = "f32", H: int = 32,
                          W: int = 40, batch: int = 1) -> NetSpec:
    """Three MBConv blocks of the B0 kinds (no-expand block, expand + 5x5
    stride-2 block, block with identity skip) at small widths."""
    return efficientnet_net(seed, dtype, H, W, batch,
                            stages=[(1, 3, 1, 8, 1), (4, 5, 2, 12, 2)],
                            stem=8, name="efficientnet_mini")
