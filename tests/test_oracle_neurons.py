"""Pins of the oracle's earlier neuron types (arXiv 2204.01701, Table 1 and
the Table 3 baselines): T4 = T_a o T_b, T4 + identity = T_a o T_b + X,
T3 = T_a o T_a, T2 = W_a * (X o X) + b_a, T2&4 = T_a o T_b + W_c * (X o X) + b_c,
with T_t = W_t * X + b_t.

Each check ties them to something other than the oracle's own code:
compositions of library convolutions (torch CPU, fp64) and their autograd,
central finite differences of the loss, scalar closed forms, and exact
relations to the proposed neuron, whose oracle is pinned separately.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle

T4, T4I, T3, T2 = oracle.NEURON_T4, oracle.NEURON_T4_IDENTITY, oracle.NEURON_T3, oracle.NEURON_T2
T24 = oracle.NEURON_T24
TYPES = [T4, T4I, T3, T2, T24]
NAMES = {T4: "T4", T4I: "T4+identity", T3: "T3", T2: "T2", T24: "T2&4"}


def _rel(a, b):
    nb = np.linalg.norm(b)
    return np.linalg.norm(a - b) / (nb if nb > 0 else 1.0)


def _case(rng, N, C, H, W, O, K):
    x = rng.standard_normal((N, C, H, W))
    ws = [rng.standard_normal((O, C, K, K)) / np.sqrt(C * K * K) for _ in range(3)]
    bs = [rng.standard_normal(O) * 0.1 for _ in range(3)]
    return x, ws, bs


def _torch_neuron(neuron, tx, tw, tb, s, p):
    """The neuron written as library convolutions and elementwise ops."""
    if neuron == T2:
        return F.conv2d(tx * tx, tw[0], tb[0], stride=s, padding=p)
    ta = F.conv2d(tx, tw[0], tb[0], stride=s, padding=p)
    if neuron == T3:
        return ta * ta
    y = ta * F.conv2d(tx, tw[1], tb[1], stride=s, padding=p)
    if neuron == T24:
        return y + F.conv2d(tx * tx, tw[2], tb[2], stride=s, padding=p)
    return y + tx if neuron == T4I else y


def _shapes(neuron):
    if neuron == T4I:  # the shortcut needs C == O and an unchanged map
        return [(2, 4, 6, 5, 4, 3, 1, 1), (1, 3, 5, 5, 3, 1, 1, 0)]
    return [(2, 3, 7, 6, 4, 3, 1, 1), (1, 5, 8, 8, 3, 3, 2, 1), (2, 4, 5, 5, 6, 1, 1, 0)]


CASES = [(n, sh) for n in TYPES for sh in _shapes(n)]
IDS = [f"{NAMES[n]}-{'x'.join(map(str, sh))}" for n, sh in CASES]


@pytest.mark.parametrize("neuron,shape", CASES, ids=IDS)
def test_forward_matches_library_convolutions(neuron, shape):
    N, C, H, W, O, K, s, p = shape
    rng = np.random.default_rng([20, neuron] + list(shape))
    x, ws, bs = _case(rng, N, C, H, W, O, K)
    y, ta, tb = oracle.conv2d_fwd_neuron(neuron, x, *ws, *bs, stride=s, pad=p)
    with torch.no_grad():
        ref = _torch_neuron(neuron, torch.from_numpy(x), [torch.from_numpy(w) for w in ws],
                            [torch.from_numpy(b) for b in bs], s, p).numpy()
    assert _rel(y, ref) < 1e-13
    # the saved maps are the first-order terms the backward needs
    xin = x * x if neuron == T2 else x
    ta_ref = F.conv2d(torch.from_numpy(xin), torch.from_numpy(ws[0]), torch.from_numpy(bs[0]), stride=s,
                      padding=p).numpy()
    assert _rel(ta, ta_ref) < 1e-13
    if neuron in (T4, T4I, T24):
        tb_ref = F.conv2d(torch.from_numpy(x), torch.from_numpy(ws[1]), torch.from_numpy(bs[1]), stride=s,
                          padding=p).numpy()
        assert _rel(tb, tb_ref) < 1e-13


@pytest.mark.parametrize("neuron,shape", CASES, ids=IDS)
def test_gradients_match_autograd_of_composition(neuron, shape):
    N, C, H, W, O, K, s, p = shape
    rng = np.random.default_rng([21, neuron] + list(shape))
    x, ws, bs = _case(rng, N, C, H, W, O, K)
    tx = torch.from_numpy(x.copy()).requires_grad_()
    tw = [torch.from_numpy(w.copy()).requires_grad_() for w in ws]
    tbias = [torch.from_numpy(b.copy()).requires_grad_() for b in bs]
    y = _torch_neuron(neuron, tx, tw, tbias, s, p)
    gy = rng.standard_normal(tuple(y.shape))
    y.backward(torch.from_numpy(gy))
    d = oracle.conv2d_bwd_neuron(neuron, x, *ws, *bs, gy, stride=s, pad=p)
    assert _rel(d["dx"], tx.grad.numpy()) < 1e-12
    nt = oracle.NEURON_TERMS[neuron]
    for k, kb, t, tbb in list(zip(("dwa", "dwb", "dwc"), ("dba", "dbb", "dbc"), tw, tbias))[:nt]:
        assert _rel(d[k], t.grad.numpy()) < 1e-12, k
        assert _rel(d[kb], tbb.grad.numpy()) < 1e-12, kb
    assert (nt == 3 or "dwc" not in d) and (nt >= 2 or "dwb" not in d)


@pytest.mark.parametrize("neuron", TYPES, ids=[NAMES[n] for n in TYPES])
def test_gradients_match_finite_differences(neuron):
    rng = np.random.default_rng([22, neuron])
    N, C, H, W, O, K, s, p = (2, 3, 4, 4, 3, 3, 1, 1)
    if neuron == T4I:
        O = C
    x, ws, bs = _case(rng, N, C, H, W, O, K)
    nt = oracle.NEURON_TERMS[neuron]
    params = {"x": x, "wa": ws[0], "ba": bs[0]}
    if nt >= 2:
        params.update(wb=ws[1], bb=bs[1])
    if nt == 3:
        params.update(wc=ws[2], bc=bs[2])
    y, _, _ = oracle.conv2d_fwd_neuron(neuron, x, *ws, *bs, stride=s, pad=p)
    gy = rng.standard_normal(y.shape)

    def loss():
        yy, _, _ = oracle.conv2d_fwd_neuron(neuron, params["x"], params["wa"], params.get("wb"), params.get("wc"),
                                            params["ba"], params.get("bb"), params.get("bc"), stride=s, pad=p)
        return float(np.sum(gy * yy))

    d = oracle.conv2d_bwd_neuron(neuron, x, *ws, *bs, gy, stride=s, pad=p)
    grads = {"x": d["dx"], "wa": d["dwa"], "ba": d["dba"]}
    if nt >= 2:
        grads.update(wb=d["dwb"], bb=d["dbb"])
    if nt == 3:
        grads.update(wc=d["dwc"], bc=d["dbc"])
    h = 1e-4
    for name, arr in params.items():
        flat = arr.reshape(-1)
        idx = rng.choice(flat.size, size=min(flat.size, 12), replace=False)
        for i in idx:
            old = flat[i]
            flat[i] = old + h
            lp = loss()
            flat[i] = old - h
            lm = loss()
            flat[i] = old
            fd = (lp - lm) / (2 * h)
            g = grads[name].reshape(-1)[i]
            # the loss is a polynomial of degree <= 3 in each argument: the central
            # difference is exact up to h^2 times the third derivative, and rounding
            assert abs(g - fd) <= 1e-6 * max(1.0, abs(fd)), (name, i, g, fd)


def test_relations_to_the_proposed_neuron():
    rng = np.random.default_rng(23)
    N, C, H, W, O, K, s, p = 2, 4, 6, 6, 4, 3, 1, 1
    x, (wa, wb, wc), (ba, bb, bc) = _case(rng, N, C, H, W, O, K)
    z = np.zeros_like(wc)
    zb = np.zeros_like(bc)
    gy = rng.standard_normal((N, O, H, W))
    # T4 is the proposed neuron without its linear term
    y4, _, _ = oracle.conv2d_fwd_neuron(T4, x, wa, wb, None, ba, bb, stride=s, pad=p)
    y0, _, _ = oracle.conv2d_fwd(x, wa, wb, z, ba, bb, zb, s, p)
    assert np.array_equal(y4, y0) or _rel(y4, y0) < 1e-15
    d4 = oracle.conv2d_bwd_neuron(T4, x, wa, wb, None, ba, bb, None, gy, stride=s, pad=p)
    d0 = oracle.conv2d_bwd(x, wa, wb, z, ba, bb, zb, gy, s, p)
    for k in ("dx", "dwa", "dwb", "dba", "dbb"):
        assert _rel(d4[k], d0[k]) < 1e-14, k
    # T3 is T4 with tied weights: the shared weight's gradient is the sum of both partials
    y3, _, _ = oracle.conv2d_fwd_neuron(T3, x, wa, None, None, ba, stride=s, pad=p)
    y4t, _, _ = oracle.conv2d_fwd_neuron(T4, x, wa, wa, None, ba, ba, stride=s, pad=p)
    assert _rel(y3, y4t) < 1e-15
    d3 = oracle.conv2d_bwd_neuron(T3, x, wa, None, None, ba, None, None, gy, stride=s, pad=p)
    d4t = oracle.conv2d_bwd_neuron(T4, x, wa, wa, None, ba, ba, None, gy, stride=s, pad=p)
    assert _rel(d3["dwa"], d4t["dwa"] + d4t["dwb"]) < 1e-14
    assert _rel(d3["dba"], d4t["dba"] + d4t["dbb"]) < 1e-14
    assert _rel(d3["dx"], d4t["dx"]) < 1e-14
    # T4 + identity adds X to Y and G to dX
    yi, _, _ = oracle.conv2d_fwd_neuron(T4I, x, wa, wb, None, ba, bb, stride=s, pad=p)
    assert _rel(yi, y4 + x) < 1e-15
    di = oracle.conv2d_bwd_neuron(T4I, x, wa, wb, None, ba, bb, None, gy, stride=s, pad=p)
    assert _rel(di["dx"], d4["dx"] + gy) < 1e-14
    for k in ("dwa", "dwb", "dba", "dbb"):
        assert np.array_equal(di[k], d4[k]), k
    # T2 is the proposed neuron's linear term applied to X o X ...
    y2, _, _ = oracle.conv2d_fwd_neuron(T2, x, wc, None, None, bc, stride=s, pad=p)
    yl, _, _ = oracle.conv2d_fwd(x * x, z, z, wc, zb, zb, bc, s, p)
    assert _rel(y2, yl) < 1e-15
    d2 = oracle.conv2d_bwd_neuron(T2, x, wc, None, None, bc, None, None, gy, stride=s, pad=p)
    dl = oracle.conv2d_bwd(x * x, z, z, wc, zb, zb, bc, gy, s, p)
    assert _rel(d2["dwa"], dl["dwc"]) < 1e-14 and _rel(d2["dba"], dl["dbc"]) < 1e-14
    # ... with the chain rule through the square
    assert _rel(d2["dx"], 2 * x * dl["dx"]) < 1e-14
    # T2&4 is the proposed neuron with X o X in place of X in its third term:
    # T4 (pinned above) plus T2 with (W_c, b_c), outputs and gradients alike
    y24, ta24, tb24 = oracle.conv2d_fwd_neuron(T24, x, wa, wb, wc, ba, bb, bc, stride=s, pad=p)
    y2c, _, _ = oracle.conv2d_fwd_neuron(T2, x, wc, None, None, bc, stride=s, pad=p)
    assert _rel(y24, y4 + y2c) < 1e-15
    _, ta0, tb0 = oracle.conv2d_fwd(x, wa, wb, z, ba, bb, zb, s, p)
    assert np.array_equal(ta24, ta0) and np.array_equal(tb24, tb0)
    d24 = oracle.conv2d_bwd_neuron(T24, x, wa, wb, wc, ba, bb, bc, gy, stride=s, pad=p)
    for k in ("dwa", "dwb", "dba", "dbb"):
        assert _rel(d24[k], d4[k]) < 1e-14, k
    d2c = oracle.conv2d_bwd_neuron(T2, x, wc, None, None, bc, None, None, gy, stride=s, pad=p)
    assert _rel(d24["dwc"], d2c["dwa"]) < 1e-14 and _rel(d24["dbc"], d2c["dba"]) < 1e-14
    assert _rel(d24["dx"], d4["dx"] + d2c["dx"]) < 1e-14
    # ... and with X o X replaced by X it is the proposed neuron itself
    yq, _, _ = oracle.conv2d_fwd(x, wa, wb, wc, ba, bb, bc, s, p)
    yq2, _, _ = oracle.conv2d_fwd(x, wa, wb, z, ba, bb, zb, s, p)
    yqc, _, _ = oracle.conv2d_fwd(x, z, z, wc, zb, zb, bc, s, p)
    assert _rel(yq, yq2 + yqc) < 1e-14 and _rel(y24 - y2c, yq - yqc) < 1e-14


def test_scalar_closed_forms():
    # one pixel, one channel, a 1x1 kernel: every type is a polynomial in x
    x, wa, wb, ba, bb, g = 1.5, -0.75, 2.0, 0.25, -0.5, 0.3
    wc, bc = 1.25, 0.125
    X = np.full((1, 1, 1, 1), x)
    Wa, Wb, Wc = np.full((1, 1, 1, 1), wa), np.full((1, 1, 1, 1), wb), np.full((1, 1, 1, 1), wc)
    Ba, Bb, Bc = np.array([ba]), np.array([bb]), np.array([bc])
    G = np.full((1, 1, 1, 1), g)
    ta, tb = wa * x + ba, wb * x + bb
    expect = {
        T4: (ta * tb, g * (wa * tb + wb * ta), g * tb * x, g * ta * x),
        T4I: (ta * tb + x, g * (wa * tb + wb * ta) + g, g * tb * x, g * ta * x),
        T3: (ta * ta, g * 2 * ta * wa, g * 2 * ta * x, None),
        T2: (wa * x * x + ba, g * wa * 2 * x, g * x * x, None),
        T24: (ta * tb + wc * x * x + bc, g * (wa * tb + wb * ta + 2 * wc * x), g * tb * x, g * ta * x),
    }
    for n, (y, dx, dwa, dwb) in expect.items():
        yy, _, _ = oracle.conv2d_fwd_neuron(n, X, Wa, Wb, Wc, Ba, Bb, Bc)
        assert yy.item() == pytest.approx(y, rel=1e-15), NAMES[n]
        d = oracle.conv2d_bwd_neuron(n, X, Wa, Wb, Wc, Ba, Bb, Bc, G)
        if n == T24:
            assert d["dwc"].item() == pytest.approx(g * x * x, rel=1e-15)
            assert d["dbc"].item() == pytest.approx(g, rel=1e-15)
        assert d["dx"].item() == pytest.approx(dx, rel=1e-15), NAMES[n]
        assert d["dwa"].item() == pytest.approx(dwa, rel=1e-15), NAMES[n]
        if dwb is not None:
            assert d["dwb"].item() == pytest.approx(dwb, rel=1e-15), NAMES[n]


@pytest.mark.parametrize("neuron", TYPES, ids=[NAMES[n] for n in TYPES])
def test_fc_neurons_match_matrix_closed_forms(neuron):
    rng = np.random.default_rng([24, neuron])
    B, I, O = 5, 6, 6
    x = rng.standard_normal((B, I))
    wa, wb, wc = rng.standard_normal((O, I)), rng.standard_normal((O, I)), rng.standard_normal((O, I))
    ba, bb, bc = rng.standard_normal(O), rng.standard_normal(O), rng.standard_normal(O)
    gy = rng.standard_normal((B, O))
    ta, tb = x @ wa.T + ba, x @ wb.T + bb
    tc = (x * x) @ wc.T + bc
    if neuron == T2:
        ta = (x * x) @ wa.T + ba
    y = {T4: ta * tb, T4I: ta * tb + x, T3: ta * ta, T2: ta, T24: ta * tb + tc}[neuron]
    yy, _, _ = oracle.linear_fwd_neuron(neuron, x, wa, wb, wc, ba, bb, bc)
    assert _rel(yy, y) < 1e-14
    d = oracle.linear_bwd_neuron(neuron, x, wa, wb, wc, ba, bb, bc, gy)
    if neuron in (T4, T4I, T24):
        ga, gb = gy * tb, gy * ta
        dx = ga @ wa + gb @ wb + (gy if neuron == T4I else 0)
        if neuron == T24:
            dx = dx + 2 * x * (gy @ wc)
            assert _rel(d["dwc"], gy.T @ (x * x)) < 1e-14 and _rel(d["dbc"], gy.sum(0)) < 1e-14
        assert _rel(d["dwb"], gb.T @ x) < 1e-14 and _rel(d["dbb"], gb.sum(0)) < 1e-14
        assert _rel(d["dwa"], ga.T @ x) < 1e-14 and _rel(d["dba"], ga.sum(0)) < 1e-14
    elif neuron == T3:
        ga = 2 * gy * ta
        dx = ga @ wa
        assert _rel(d["dwa"], ga.T @ x) < 1e-14 and _rel(d["dba"], ga.sum(0)) < 1e-14
    else:
        dx = 2 * x * (gy @ wa)
        assert _rel(d["dwa"], gy.T @ (x * x)) < 1e-14 and _rel(d["dba"], gy.sum(0)) < 1e-14
    assert _rel(d["dx"], dx) < 1e-14
