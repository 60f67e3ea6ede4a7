"""fp64 oracle of the network glue of the CIFAR ResNet training step -- TEST INFRASTRUCTURE ONLY.

Plain numpy in float64 on the logical PyTorch layouts (N x C x H x W), written
from the definitions; the quadratic layers themselves come from the pinned C
oracle (``oracle.conv2d_fwd`` / ``conv2d_bwd`` / ``linear_fwd`` / ``linear_bwd``).

Model construction (arXiv 2204.01701, section 4.2: a batch normalization after
every quadratic layer, a ReLU in deeper networks), read as the standard CIFAR
ResNet basic block:  qconv -> BN -> ReLU -> qconv -> BN -> (+ shortcut) -> ReLU,
the shortcut the identity, or at a stride-2 transition the input subsampled
by 2 with its channels placed at [C/4, C/4 + C_in) of the C output channels
("option A"); a qconv -> BN -> ReLU stem; global average pooling and a
quadratic fully-connected classifier.  Batch normalization in training mode
with gamma = 1, beta = 0, eps = 1e-5 and the biased batch variance.
"""
from __future__ import annotations

import numpy as np

EPS = 1e-5


def shortcut(x, c_out, h_out, w_out):
    """The block's shortcut of input x (N, C_in, H, W) at the output shape."""
    n, c_in, h, w = x.shape
    if (c_in, h, w) == (c_out, h_out, w_out):
        return x
    assert h == 2 * h_out and w == 2 * w_out and 2 * c_in == c_out, "option A: stride 2, channels doubled"
    out = np.zeros((n, c_out, h_out, w_out))
    p = c_out // 4
    out[:, p:p + c_in] = x[:, :, ::2, ::2]
    return out


def shortcut_bwd(dz, x_shape):
    """Gradient at the block input of shortcut(): dz (N, C, Ho, Wo) -> x_shape."""
    n, c_in, h, w = x_shape
    c = dz.shape[1]
    if (c_in, h, w) == dz.shape[1:]:
        return dz.copy()
    out = np.zeros(x_shape)
    p = c // 4
    out[:, :, ::2, ::2] = dz[:, p:p + c_in]
    return out


def bn_act_fwd(y, res=None, relu=True, eps=EPS):
    """out = relu((y - mean) / sqrt(var + eps) + shortcut(res)); returns (out, mean, var)."""
    mean = y.mean(axis=(0, 2, 3))
    var = ((y - mean[None, :, None, None]) ** 2).mean(axis=(0, 2, 3))
    z = (y - mean[None, :, None, None]) / np.sqrt(var + eps)[None, :, None, None]
    if res is not None:
        z = z + shortcut(res, y.shape[1], y.shape[2], y.shape[3])
    out = np.maximum(z, 0.0) if relu else z
    return out, mean, var


def bn_act_bwd(dout, out, y, relu=True, eps=EPS):
    """Gradient at y of bn_act_fwd (the shortcut's share is shortcut_bwd of dz):
    with dz = dout [out > 0] and x^ = (y - mean) rstd over the M = N H W pixels,
    dy = rstd (dz - mean(dz) - x^ mean(dz x^))."""
    mean = y.mean(axis=(0, 2, 3))
    var = ((y - mean[None, :, None, None]) ** 2).mean(axis=(0, 2, 3))
    rstd = 1.0 / np.sqrt(var + eps)
    xh = (y - mean[None, :, None, None]) * rstd[None, :, None, None]
    dz = dout * (out > 0) if relu else dout
    m1 = dz.mean(axis=(0, 2, 3))
    m2 = (dz * xh).mean(axis=(0, 2, 3))
    return rstd[None, :, None, None] * (dz - m1[None, :, None, None] - xh * m2[None, :, None, None]), dz


def gap_fwd(x):
    return x.mean(axis=(2, 3))


def gap_bwd(dy, shape):
    n, c, h, w = shape
    return np.broadcast_to(dy[:, :, None, None] / (h * w), shape).copy()


def resnet20_step(params, x, g_logits, layers, conv_fwd, conv_bwd, linear_fwd, linear_bwd):
    """Forward and backward of the network.  params: per conv layer a dict
    wa, wb, wc, ba, bb, bc, and "head" for the classifier; layers: the conv
    geometries (stem, then two per block); x: the images (N, 3, 32, 32);
    g_logits: dl/dlogits.  The quadratic layers are the callables conv_fwd(x,
    p, stride, pad) -> (y, ta, tb), conv_bwd(x, p, gy, stride, pad) -> dict,
    linear_fwd, linear_bwd (the fp64 oracle's).  Returns logits, the gradient
    of every weight and bias, and the intermediates (for teacher forcing)."""
    acts = {}
    grads = {}
    # forward
    L0 = layers[0]
    y0, _, _ = conv_fwd(x, params[0], L0.stride, L0.pad)
    a, _, _ = bn_act_fwd(y0)
    acts[0] = {"x": x, "y": y0, "out": a}
    cur = a
    i = 1
    blocks = []
    while i < len(layers):
        L1, L2 = layers[i], layers[i + 1]
        xin = cur
        y1, _, _ = conv_fwd(xin, params[i], L1.stride, L1.pad)
        a1, _, _ = bn_act_fwd(y1)
        y2, _, _ = conv_fwd(a1, params[i + 1], L2.stride, L2.pad)
        out, _, _ = bn_act_fwd(y2, res=xin)
        acts[i] = {"x": xin, "y": y1, "out": a1}
        acts[i + 1] = {"x": a1, "y": y2, "out": out}
        blocks.append((i, i + 1))
        cur = out
        i += 2
    z = gap_fwd(cur)
    hp = params["head"]
    logits, _, _ = linear_fwd(z, hp["wa"], hp["wb"], hp["wc"], hp["ba"], hp["bb"], hp["bc"])
    # backward
    dh = linear_bwd(z, hp["wa"], hp["wb"], hp["wc"], hp["ba"], hp["bb"], hp["bc"], g_logits)
    grads["head"] = {k: dh[k] for k in ("dwa", "dwb", "dwc", "dba", "dbb", "dbc")}
    dcur = gap_bwd(dh["dx"], cur.shape)
    for j1, j2 in reversed(blocks):
        A1, A2 = acts[j1], acts[j2]
        L1, L2 = layers[j1], layers[j2]
        g2, dz = bn_act_bwd(dcur, A2["out"], A2["y"])
        d2 = conv_bwd(A2["x"], params[j2], g2, L2.stride, L2.pad)
        grads[j2] = {k: d2[k] for k in ("dwa", "dwb", "dwc", "dba", "dbb", "dbc")}
        acts[j2]["g"] = g2
        g1, _ = bn_act_bwd(d2["dx"], A1["out"], A1["y"])
        d1 = conv_bwd(A1["x"], params[j1], g1, L1.stride, L1.pad)
        grads[j1] = {k: d1[k] for k in ("dwa", "dwb", "dwc", "dba", "dbb", "dbc")}
        acts[j1]["g"] = g1
        dcur = d1["dx"] + shortcut_bwd(dz, A1["x"].shape)
    g0, _ = bn_act_bwd(dcur, acts[0]["out"], acts[0]["y"])
    d0 = conv_bwd(x, params[0], g0, L0.stride, L0.pad)
    grads[0] = {k: d0[k] for k in ("dwa", "dwb", "dwc", "dba", "dbb", "dbc")}
    acts[0]["g"] = g0
    return logits, grads, acts
