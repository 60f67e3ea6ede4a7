"""Seeded synthetic inputs shared by the tests, the benchmark and the oracle checks.

This module holds no arithmetic of the quadratic neuron: it only draws
random tensors (numpy, counter-seeded) with the shapes and value
distributions of the image-classification workloads the paper evaluates
(CIFAR-style 3x32x32 inputs at batch 128/256, VGG-16 and ResNet stacks,
section 5 and Table 3), and rounds them to bf16 when the workload is bf16.
No dataset is read; every value is synthetic.

Arrays are float32 in the logical PyTorch layouts (N x C x H x W activations,
O x C x KH x KW weights, B x I / O x I for dense layers).  Values for a bf16
workload are already exactly representable in bf16, so the GPU (bf16) and
the oracle (float64) see identical numbers.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

# tensor ids used in the seeds
X_ID, WA_ID, WB_ID, WC_ID, BA_ID, BB_ID, BC_ID, G_ID = range(8)


def round_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even), returned as float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    rounded = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    out = (rounded & 0xFFFFFFFF).astype(np.uint32).view(np.float32)
    nan = np.isnan(a)
    if nan.any():
        out = out.copy()
        out[nan] = np.float32("nan")
    return out.reshape(a.shape)


def _normal(seed, shape, std):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal(size=shape, dtype=np.float32) * np.float32(std)).astype(np.float32)


@dataclass(frozen=True)
class ConvLayer:
    """One quadratic conv layer of a workload: geometry plus init scales."""
    n: int
    c: int
    h: int
    w: int
    o: int
    k: int = 3
    stride: int = 1
    pad: int = 1
    w_var: float | None = None   # weight variance; None = He, 2 / (C*K*K)
    b_var: float = 0.01          # bias variance (biases ~ N(0, b_var))

    @property
    def ho(self):
        return (self.h + 2 * self.pad - self.k) // self.stride + 1

    @property
    def wo(self):
        return (self.w + 2 * self.pad - self.k) // self.stride + 1

    def unit_flops(self) -> int:
        """Flops of ONE first-order convolution of this geometry (every tap counted)."""
        return 2 * self.n * self.ho * self.wo * self.o * self.c * self.k * self.k


@dataclass(frozen=True)
class DenseLayer:
    batch: int
    inp: int
    out: int
    w_var: float | None = None
    b_var: float = 0.0

    def unit_flops(self) -> int:
        return 2 * self.batch * self.inp * self.out


def conv_inputs(cfg_id: int, layer_id: int, L: ConvLayer, bf16: bool, with_grad: bool = True):
    """Draw X, W_a, W_b, W_c, b_a, b_b, b_c (and the upstream gradient G) for one conv layer.

    Seeds are numpy default_rng([cfg_id, layer_id, tensor_id]).  X ~ N(0, 1),
    W_t ~ N(0, w_var) (He: 2 / (C*K*K) when w_var is None), b_t ~ N(0, b_var),
    G ~ N(0, 1).
    """
    wv = L.w_var if L.w_var is not None else 2.0 / (L.c * L.k * L.k)
    out = {
        "x": _normal([cfg_id, layer_id, X_ID], (L.n, L.c, L.h, L.w), 1.0),
        "wa": _normal([cfg_id, layer_id, WA_ID], (L.o, L.c, L.k, L.k), np.sqrt(wv)),
        "wb": _normal([cfg_id, layer_id, WB_ID], (L.o, L.c, L.k, L.k), np.sqrt(wv)),
        "wc": _normal([cfg_id, layer_id, WC_ID], (L.o, L.c, L.k, L.k), np.sqrt(wv)),
        "ba": _normal([cfg_id, layer_id, BA_ID], (L.o,), np.sqrt(L.b_var)),
        "bb": _normal([cfg_id, layer_id, BB_ID], (L.o,), np.sqrt(L.b_var)),
        "bc": _normal([cfg_id, layer_id, BC_ID], (L.o,), np.sqrt(L.b_var)),
    }
    if with_grad:
        out["gy"] = _normal([cfg_id, layer_id, G_ID], (L.n, L.o, L.ho, L.wo), 1.0)
    if bf16:
        for k in ("x", "wa", "wb", "wc", "gy"):
            if k in out:
                out[k] = round_bf16(out[k])
    return out


def dense_inputs(cfg_id: int, layer_id: int, L: DenseLayer, bf16: bool, with_grad: bool = True):
    """Draw the dense-layer tensors: X ~ N(0,1) (B x I), W_t ~ N(0, w_var) (O x I), b_t, G."""
    wv = L.w_var if L.w_var is not None else 1.0 / L.inp
    out = {
        "x": _normal([cfg_id, layer_id, X_ID], (L.batch, L.inp), 1.0),
        "wa": _normal([cfg_id, layer_id, WA_ID], (L.out, L.inp), np.sqrt(wv)),
        "wb": _normal([cfg_id, layer_id, WB_ID], (L.out, L.inp), np.sqrt(wv)),
        "wc": _normal([cfg_id, layer_id, WC_ID], (L.out, L.inp), np.sqrt(wv)),
    }
    for key, tid in (("ba", BA_ID), ("bb", BB_ID), ("bc", BC_ID)):
        out[key] = (_normal([cfg_id, layer_id, tid], (L.out,), np.sqrt(L.b_var)) if L.b_var > 0
                    else np.zeros(L.out, np.float32))
    if with_grad:
        out["gy"] = _normal([cfg_id, layer_id, G_ID], (L.batch, L.out), 1.0)
    if bf16:
        for k in ("x", "wa", "wb", "wc", "gy"):
            if k in out:
                out[k] = round_bf16(out[k])
    return out


# ----------------------------------------------------------------------------
# The five workloads.
# ----------------------------------------------------------------------------

# 1: one small fp32 layer, N=2, C=O=16, 8x8, 3x3, s1 p1, W ~ N(0, 1/(16*9)), b ~ N(0, 0.01).
SMALL_FP32 = ConvLayer(n=2, c=16, h=8, w=8, o=16, k=3, stride=1, pad=1, w_var=1.0 / (16 * 9), b_var=0.01)


def vgg16_layers(batch: int = 128):
    """The 13 3x3 conv layers of a CIFAR VGG-16 (channels 64-64-128-128-256x3-512x6,
    2x2 max-pool between stages, which only sets the spatial sizes here)."""
    cfg = [64, 64, "M", 128, 128, "M", 256, 256, 256, "M", 512, 512, 512, "M", 512, 512, 512]
    layers, c, hw = [], 3, 32
    for v in cfg:
        if v == "M":
            hw //= 2
            continue
        layers.append(ConvLayer(n=batch, c=c, h=hw, w=hw, o=v, k=3, stride=1, pad=1))
        c = v
    return layers


def resnet20_layers(batch: int = 256):
    """The 19 3x3 quadratic convs of a CIFAR ResNet-20: a 3->16 stem, then three
    stages of three basic blocks (two convs each) at 16/32/64 channels; the first
    conv of stages 2 and 3 has stride 2."""
    layers = [ConvLayer(n=batch, c=3, h=32, w=32, o=16)]
    c, hw = 16, 32
    for stage, width in enumerate((16, 32, 64)):
        for blk in range(3):
            s = 2 if (stage > 0 and blk == 0) else 1
            layers.append(ConvLayer(n=batch, c=c, h=hw, w=hw, o=width, stride=s))
            hw = hw // s
            layers.append(ConvLayer(n=batch, c=width, h=hw, w=hw, o=width))
            c = width
    return layers


def resnet20_network(batch: int = 256, bf16: bool = False, cfg_id: int = 3, num_classes: int = 10):
    """Inputs of the whole ResNet-20 training step: per conv layer i the weights
    and biases conv_inputs(cfg_id, i, ...) draws (He-scaled, biases N(0, 0.01)),
    the classifier's (64 -> num_classes: W ~ N(0, 1/64), b ~ N(0, 0.01); seeds
    [cfg_id, 19, *]), the images X ~ N(0, 1) (N, 3, 32, 32) and the gradient of
    the logits G ~ N(0, 1) (N, num_classes) (seeds [cfg_id, 20, *]).
    Returns (params, x, g_logits)."""
    layers = resnet20_layers(batch)
    params = {}
    for i, L in enumerate(layers):
        inp = conv_inputs(cfg_id, i, L, bf16=bf16, with_grad=False)
        params[i] = {k: inp[k] for k in ("wa", "wb", "wc", "ba", "bb", "bc")}
    c_last = layers[-1].o
    head = DenseLayer(batch=batch, inp=c_last, out=num_classes, w_var=1.0 / c_last, b_var=0.01)
    d = dense_inputs(cfg_id, len(layers), head, bf16=bf16, with_grad=False)
    params["head"] = {k: d[k] for k in ("wa", "wb", "wc", "ba", "bb", "bc")}
    x = _normal([cfg_id, len(layers) + 1, X_ID], (batch, 3, 32, 32), 1.0)
    g = _normal([cfg_id, len(layers) + 1, G_ID], (batch, num_classes), 1.0)
    if bf16:
        x, g = round_bf16(x), round_bf16(g)
    return params, x, g


def mobilenet_v1_pairs(batch: int = 128):
    """The 13 depthwise / pointwise pairs of a CIFAR MobileNet-V1 (a 3->32 stem at
    32x32, then blocks of a 3x3 depthwise layer, stride 1 or 2, and a 1x1
    pointwise layer to 64, 128, 128, 256, 256, 512 x 6, 1024, 1024 channels;
    stride 2 in the blocks to 128, 256, 512 and the first 1024).  Returns
    (depthwise, pointwise) ConvLayer pairs; a depthwise layer has o == c."""
    cfg = [64, (128, 2), 128, (256, 2), 256, (512, 2), 512, 512, 512, 512, 512, (1024, 2), 1024]
    pairs, c, hw = [], 32, 32
    for v in cfg:
        o, s = (v, 1) if isinstance(v, int) else v
        dw = ConvLayer(n=batch, c=c, h=hw, w=hw, o=c, k=3, stride=s, pad=1)
        hw = dw.ho
        pairs.append((dw, ConvLayer(n=batch, c=c, h=hw, w=hw, o=o, k=1, stride=1, pad=0)))
        c = o
    return pairs


# 4: one large bf16 layer, N=64, C=O=256, 56x56, 3x3, s1 p1.
LARGE_BF16 = ConvLayer(n=64, c=256, h=56, w=56, o=256, k=3, stride=1, pad=1)

# 5: dense bf16 layer, batch 8192, 4096 -> 4096, W ~ N(0, 1/4096), zero biases.
DENSE_BF16 = DenseLayer(batch=8192, inp=4096, out=4096, w_var=1.0 / 4096, b_var=0.0)


def random_conv_case(seed, N, C, H, W, O, KH, KW, stride=1, pad=0, bf16=False, w_var=None, b_var=0.01):
    """Seeded inputs of an arbitrary conv geometry (ragged/odd shapes for parity tests).

    X ~ N(0,1), W_t ~ N(0, w_var) (default 1/(C*KH*KW)), b_t ~ N(0, b_var), G ~ N(0,1).
    """
    wv = w_var if w_var is not None else 1.0 / (C * KH * KW)
    Ho = (H + 2 * pad - KH) // stride + 1
    Wo = (W + 2 * pad - KW) // stride + 1
    s = list(seed) if isinstance(seed, (list, tuple)) else [seed]
    out = {
        "x": _normal(s + [X_ID], (N, C, H, W), 1.0),
        "wa": _normal(s + [WA_ID], (O, C, KH, KW), np.sqrt(wv)),
        "wb": _normal(s + [WB_ID], (O, C, KH, KW), np.sqrt(wv)),
        "wc": _normal(s + [WC_ID], (O, C, KH, KW), np.sqrt(wv)),
        "ba": _normal(s + [BA_ID], (O,), np.sqrt(b_var)),
        "bb": _normal(s + [BB_ID], (O,), np.sqrt(b_var)),
        "bc": _normal(s + [BC_ID], (O,), np.sqrt(b_var)),
        "gy": _normal(s + [G_ID], (N, O, Ho, Wo), 1.0),
    }
    if bf16:
        for k in ("x", "wa", "wb", "wc", "gy"):
            out[k] = round_bf16(out[k])
    return out


def random_dwconv_case(seed, N, C, H, W, KH, KW, stride=1, pad=0, bf16=False, w_var=None, b_var=0.01):
    """Seeded inputs of a depthwise geometry (groups = C, one filter per channel).

    X ~ N(0,1), W_t ~ N(0, w_var) (default 1/(KH*KW)) of shape C x 1 x KH x KW,
    b_t ~ N(0, b_var), G ~ N(0,1).
    """
    wv = w_var if w_var is not None else 1.0 / (KH * KW)
    Ho = (H + 2 * pad - KH) // stride + 1
    Wo = (W + 2 * pad - KW) // stride + 1
    s = list(seed) if isinstance(seed, (list, tuple)) else [seed]
    out = {
        "x": _normal(s + [X_ID], (N, C, H, W), 1.0),
        "wa": _normal(s + [WA_ID], (C, 1, KH, KW), np.sqrt(wv)),
        "wb": _normal(s + [WB_ID], (C, 1, KH, KW), np.sqrt(wv)),
        "wc": _normal(s + [WC_ID], (C, 1, KH, KW), np.sqrt(wv)),
        "ba": _normal(s + [BA_ID], (C,), np.sqrt(b_var)),
        "bb": _normal(s + [BB_ID], (C,), np.sqrt(b_var)),
        "bc": _normal(s + [BC_ID], (C,), np.sqrt(b_var)),
        "gy": _normal(s + [G_ID], (N, C, Ho, Wo), 1.0),
    }
    if bf16:
        for k in ("x", "wa", "wb", "wc", "gy"):
            out[k] = round_bf16(out[k])
    return out


def random_dense_case(seed, B, I, O, bf16=False, w_var=None, b_var=0.01):
    """Seeded inputs of an arbitrary dense geometry: X ~ N(0,1), W_t ~ N(0, 1/I), b_t, G ~ N(0,1)."""
    wv = w_var if w_var is not None else 1.0 / I
    s = list(seed) if isinstance(seed, (list, tuple)) else [seed]
    out = {
        "x": _normal(s + [X_ID], (B, I), 1.0),
        "wa": _normal(s + [WA_ID], (O, I), np.sqrt(wv)),
        "wb": _normal(s + [WB_ID], (O, I), np.sqrt(wv)),
        "wc": _normal(s + [WC_ID], (O, I), np.sqrt(wv)),
        "ba": _normal(s + [BA_ID], (O,), np.sqrt(b_var)) if b_var > 0 else np.zeros(O, np.float32),
        "bb": _normal(s + [BB_ID], (O,), np.sqrt(b_var)) if b_var > 0 else np.zeros(O, np.float32),
        "bc": _normal(s + [BC_ID], (O,), np.sqrt(b_var)) if b_var > 0 else np.zeros(O, np.float32),
        "gy": _normal(s + [G_ID], (B, O), 1.0),
    }
    if bf16:
        for k in ("x", "wa", "wb", "wc", "gy"):
            out[k] = round_bf16(out[k])
    return out
