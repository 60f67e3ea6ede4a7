"""Pins of the oracle's depthwise quadratic convolution (groups = C; the
depth-wise setting the paper's layer modules take, section 4.2), for every
neuron type: library compositions (torch CPU fp64, conv2d with groups = C)
and their autograd, finite differences, and the one-channel case, which is
the dense oracle's."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle

TYPES = [0, 1, 2, 3, 4]
NAMES = ["quadra", "T4", "T4I", "T3", "T2"]


def _rel(a, b):
    nb = np.linalg.norm(b)
    return np.linalg.norm(a - b) / (nb if nb > 0 else 1.0)


def _case(rng, N, C, H, W, K):
    x = rng.standard_normal((N, C, H, W))
    ws = [rng.standard_normal((C, 1, K, K)) / K for _ in range(3)]
    bs = [rng.standard_normal(C) * 0.1 for _ in range(3)]
    return x, ws, bs


def _torch_dw(neuron, tx, tw, tb, s, p, C):
    def conv(inp, t):
        return F.conv2d(inp, tw[t], tb[t], stride=s, padding=p, groups=C)
    if neuron == 4:
        return conv(tx * tx, 0)
    ta = conv(tx, 0)
    if neuron == 3:
        return ta * ta
    y = ta * conv(tx, 1)
    if neuron == 0:
        return y + conv(tx, 2)
    return y + tx if neuron == 2 else y


SHAPES = [(2, 6, 7, 6, 3, 1, 1), (1, 5, 8, 8, 3, 2, 1), (2, 4, 5, 5, 5, 1, 2), (2, 3, 6, 6, 1, 1, 0)]
CASES = [(n, sh) for n in TYPES for sh in SHAPES if n != 2 or sh[5] == 1 and 2 * sh[6] == sh[4] - 1]


@pytest.mark.parametrize("neuron,shape", CASES, ids=[f"{NAMES[n]}-{'x'.join(map(str, sh))}" for n, sh in CASES])
def test_depthwise_matches_library_and_autograd(neuron, shape):
    N, C, H, W, K, s, p = shape
    rng = np.random.default_rng([30, neuron] + list(shape))
    x, ws, bs = _case(rng, N, C, H, W, K)
    tx = torch.from_numpy(x.copy()).requires_grad_()
    tw = [torch.from_numpy(w.copy()).requires_grad_() for w in ws]
    tbias = [torch.from_numpy(b.copy()).requires_grad_() for b in bs]
    yt = _torch_dw(neuron, tx, tw, tbias, s, p, C)
    y, _, _ = oracle.dwconv2d_fwd(neuron, x, *ws, *bs, stride=s, pad=p)
    assert _rel(y, yt.detach().numpy()) < 1e-13
    gy = rng.standard_normal(y.shape)
    yt.backward(torch.from_numpy(gy))
    d = oracle.dwconv2d_bwd(neuron, x, *ws, *bs, gy, stride=s, pad=p)
    assert _rel(d["dx"], tx.grad.numpy()) < 1e-12
    nt = oracle.NEURON_TERMS[neuron]
    for t, (kw, kb) in enumerate((("dwa", "dba"), ("dwb", "dbb"), ("dwc", "dbc"))[:nt]):
        assert _rel(d[kw], tw[t].grad.numpy()) < 1e-12, kw
        assert _rel(d[kb], tbias[t].grad.numpy()) < 1e-12, kb


@pytest.mark.parametrize("neuron", TYPES, ids=NAMES)
def test_depthwise_gradients_match_finite_differences(neuron):
    rng = np.random.default_rng([31, neuron])
    N, C, H, W, K, s, p = 2, 3, 4, 4, 3, 1, 1
    x, ws, bs = _case(rng, N, C, H, W, K)
    nt = oracle.NEURON_TERMS[neuron]
    params = {"x": x}
    for t, (kw, kb) in enumerate((("wa", "ba"), ("wb", "bb"), ("wc", "bc"))[:nt]):
        params[kw], params[kb] = ws[t], bs[t]
    y, _, _ = oracle.dwconv2d_fwd(neuron, x, *ws, *bs, stride=s, pad=p)
    gy = rng.standard_normal(y.shape)

    def loss():
        yy, _, _ = oracle.dwconv2d_fwd(neuron, params["x"], params["wa"], params.get("wb"), params.get("wc"),
                                       params["ba"], params.get("bb"), params.get("bc"), stride=s, pad=p)
        return float(np.sum(gy * yy))

    d = oracle.dwconv2d_bwd(neuron, x, *ws, *bs, gy, stride=s, pad=p)
    grads = {"x": d["dx"]}
    for kw, kb in (("wa", "ba"), ("wb", "bb"), ("wc", "bc"))[:nt]:
        grads[kw], grads[kb] = d["d" + kw], d["d" + kb]
    h = 1e-4
    for name, arr in params.items():
        flat = arr.reshape(-1)
        for i in rng.choice(flat.size, size=min(flat.size, 10), replace=False):
            old = flat[i]
            flat[i] = old + h
            lp = loss()
            flat[i] = old - h
            lm = loss()
            flat[i] = old
            fd = (lp - lm) / (2 * h)
            g = grads[name].reshape(-1)[i]
            assert abs(g - fd) <= 1e-6 * max(1.0, abs(fd)), (name, i, g, fd)


@pytest.mark.parametrize("neuron", TYPES, ids=NAMES)
def test_one_channel_equals_dense_oracle(neuron):
    rng = np.random.default_rng([32, neuron])
    x, ws, bs = _case(rng, 2, 1, 6, 5, 3)
    y, ta, tb = oracle.dwconv2d_fwd(neuron, x, *ws, *bs, stride=1, pad=1)
    nt = oracle.NEURON_TERMS[neuron]
    wl = [ws[t] if t < nt else None for t in range(3)]
    bl = [bs[t] if t < nt else None for t in range(3)]
    y2, _, _ = oracle.conv2d_fwd_neuron(neuron, x, *wl, *bl, stride=1, pad=1)
    assert _rel(y, y2) < 1e-15
    gy = rng.standard_normal(y.shape)
    d = oracle.dwconv2d_bwd(neuron, x, *ws, *bs, gy, stride=1, pad=1)
    d2 = oracle.conv2d_bwd_neuron(neuron, x, *wl, *bl, gy, stride=1, pad=1)
    for k in d2:
        assert _rel(d[k], d2[k]) < 1e-14, k
