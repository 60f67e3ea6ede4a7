"""Pins of the network glue oracle (oracle/network.py) of the CIFAR ResNet
training step: batch normalization in training mode, ReLU, the identity and
option-A shortcuts, global average pooling, and the whole network's forward
and backward, each against torch (CPU, fp64) library functions and autograd.
"""
import dataclasses

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle import network as net


def _rel(a, b):
    nb = np.linalg.norm(b)
    return np.linalg.norm(a - b) / (nb if nb > 0 else 1.0)


def _torch_shortcut(x, c_out):
    """Option A written with library ops: subsample, then zero-pad the channels."""
    c_in = x.shape[1]
    if c_in == c_out:
        return x
    p = c_out // 4
    return F.pad(x[:, :, ::2, ::2], (0, 0, 0, 0, p, c_out - c_in - p))


def _torch_bn_act(y, res=None, relu=True):
    z = F.batch_norm(y, None, None, training=True, eps=net.EPS)
    if res is not None:
        z = z + _torch_shortcut(res, y.shape[1])
    return torch.relu(z) if relu else z


CASES = [("none", None), ("identity", (3, 8, 6, 5)), ("option_a", (3, 4, 12, 10))]


@pytest.mark.parametrize("relu", [True, False], ids=["relu", "linear"])
@pytest.mark.parametrize("name,rshape", CASES, ids=[c[0] for c in CASES])
def test_bn_act_matches_torch_and_autograd(name, rshape, relu):
    rng = np.random.default_rng([30, len(name), int(relu)])
    y = rng.standard_normal((3, 8, 6, 5)) * 2.0 + 0.5
    res = rng.standard_normal(rshape) if rshape else None
    out, mean, var = net.bn_act_fwd(y, res, relu)
    ty = torch.from_numpy(y.copy()).requires_grad_()
    tr = torch.from_numpy(res.copy()).requires_grad_() if res is not None else None
    tout = _torch_bn_act(ty, tr, relu)
    assert _rel(out, tout.detach().numpy()) < 1e-13
    assert _rel(mean, y.mean(axis=(0, 2, 3))) < 1e-15 and _rel(var, y.var(axis=(0, 2, 3))) < 1e-13
    dout = rng.standard_normal(out.shape)
    tout.backward(torch.from_numpy(dout))
    dy, dz = net.bn_act_bwd(dout, out, y, relu)
    assert _rel(dy, ty.grad.numpy()) < 1e-12
    if res is not None:
        assert _rel(net.shortcut_bwd(dz, res.shape), tr.grad.numpy()) < 1e-13


def test_shortcut_option_a_layout():
    x = np.arange(2 * 2 * 4 * 4, dtype=np.float64).reshape(2, 2, 4, 4)
    s = net.shortcut(x, 4, 2, 2)
    assert s.shape == (2, 4, 2, 2)
    assert np.all(s[:, 0] == 0) and np.all(s[:, 3] == 0)
    assert np.array_equal(s[:, 1:3], x[:, :, ::2, ::2])


def test_gap_matches_torch():
    rng = np.random.default_rng(31)
    x = rng.standard_normal((3, 5, 4, 4))
    tx = torch.from_numpy(x.copy()).requires_grad_()
    ty = tx.mean(dim=(2, 3))
    assert _rel(net.gap_fwd(x), ty.detach().numpy()) < 1e-15
    dy = rng.standard_normal((3, 5))
    ty.backward(torch.from_numpy(dy))
    assert _rel(net.gap_bwd(dy, x.shape), tx.grad.numpy()) < 1e-15


def _oracle_conv_fwd(x, p, s, pad):
    return oracle.conv2d_fwd(x, p["wa"], p["wb"], p["wc"], p["ba"], p["bb"], p["bc"], s, pad)


def _oracle_conv_bwd(x, p, gy, s, pad):
    return oracle.conv2d_bwd(x, p["wa"], p["wb"], p["wc"], p["ba"], p["bb"], p["bc"], gy, s, pad)


def _torch_qconv(x, p, s, pad):
    """The quadratic convolution as the paper builds it (three first-order layers)."""
    return (F.conv2d(x, p["wa"], p["ba"], stride=s, padding=pad) * F.conv2d(x, p["wb"], p["bb"], stride=s, padding=pad)
            + F.conv2d(x, p["wc"], p["bc"], stride=s, padding=pad))


@dataclasses.dataclass
class _L:
    c: int
    o: int
    stride: int
    pad: int = 1


def test_small_resnet_step_matches_autograd():
    """A small network of the same construction (stem 3->8, a block at 8, a
    stride-2 block 8->16, GAP, quadratic FC 16->5), batch 2 of 8x8 images:
    logits and every weight and bias gradient against torch autograd."""
    rng = np.random.default_rng(32)
    layers = [_L(3, 8, 1), _L(8, 8, 1), _L(8, 8, 1), _L(8, 16, 2), _L(16, 16, 1)]
    params = {}
    for i, L in enumerate(layers):
        sd = 1.0 / np.sqrt(L.c * 9)
        params[i] = {k: rng.standard_normal((L.o, L.c, 3, 3)) * sd for k in ("wa", "wb", "wc")}
        params[i].update({k: rng.standard_normal(L.o) * 0.1 for k in ("ba", "bb", "bc")})
    params["head"] = {k: rng.standard_normal((5, 16)) * 0.25 for k in ("wa", "wb", "wc")}
    params["head"].update({k: rng.standard_normal(5) * 0.1 for k in ("ba", "bb", "bc")})
    x = rng.standard_normal((2, 3, 8, 8))
    g = rng.standard_normal((2, 5))
    logits, grads, _ = net.resnet20_step(params, x, g, layers, _oracle_conv_fwd, _oracle_conv_bwd,
                                         oracle.linear_fwd, oracle.linear_bwd)
    tp = {k: {n: torch.from_numpy(v.copy()).requires_grad_() for n, v in p.items()} for k, p in params.items()}
    tx = torch.from_numpy(x)
    a = _torch_bn_act(_torch_qconv(tx, tp[0], 1, 1))
    for i in (1, 3):
        h = _torch_bn_act(_torch_qconv(a, tp[i], layers[i].stride, 1))
        a = _torch_bn_act(_torch_qconv(h, tp[i + 1], 1, 1), res=a)
    z = a.mean(dim=(2, 3))
    hp = tp["head"]
    tl = (z @ hp["wa"].T + hp["ba"]) * (z @ hp["wb"].T + hp["bb"]) + z @ hp["wc"].T + hp["bc"]
    assert _rel(logits, tl.detach().numpy()) < 1e-12
    tl.backward(torch.from_numpy(g))
    for k in list(range(len(layers))) + ["head"]:
        for t in ("a", "b", "c"):
            assert _rel(grads[k]["dw" + t], tp[k]["w" + t].grad.numpy()) < 1e-10, (k, t)
            # (db_c ahead of a batch normalization is zero in exact arithmetic: compare absolutely there)
            ref = tp[k]["b" + t].grad.numpy()
            err = np.linalg.norm(grads[k]["db" + t] - ref)
            assert err < 1e-10 * max(np.linalg.norm(ref), 1e-3), (k, t)
