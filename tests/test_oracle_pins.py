"""Pins of the fp64 oracle to facts fixed by the paper and by mathematics.

Each check ties the oracle to something other than itself: hand-derived
worked examples (tests/golden), textbook/library convolution routines
(torch CPU, fp64), closed forms, exact invariants of the neuron's definition
(arXiv 2204.01701 section 3.1, eq:2ndneuron3) and central finite differences
of the loss (which are exact up to rounding because the loss is a quadratic
polynomial in every argument).
"""
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _read_golden(name):
    vals, geom = {}, {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, *rest = line.split()
            if key == "geometry":
                geom = {kv.split("=")[0]: int(kv.split("=")[1]) for kv in rest}
            else:
                vals[key] = np.array([float(v) for v in rest])
    return geom, vals


def _rand_case(rng, N, C, H, W, O, KH, KW, bias=True):
    x = rng.standard_normal((N, C, H, W))
    ws = [rng.standard_normal((O, C, KH, KW)) / np.sqrt(C * KH * KW) for _ in range(3)]
    bs = [rng.standard_normal(O) * 0.1 if bias else None for _ in range(3)]
    return x, ws, bs


def _torch_terms(x, ws, bs, stride, pad):
    tx = torch.from_numpy(x)
    out = []
    for w, b in zip(ws, bs):
        tb = None if b is None else torch.from_numpy(b)
        out.append(F.conv2d(tx, torch.from_numpy(w), tb, stride=stride, padding=pad).numpy())
    return out


def _rel(a, b):
    nb = np.linalg.norm(b)
    return np.linalg.norm(a - b) / (nb if nb > 0 else 1.0)


SHAPES = [  # N, C, H, W, O, KH, KW, stride, pad
    (2, 3, 7, 6, 4, 3, 3, 1, 1),
    (1, 5, 8, 8, 3, 3, 3, 2, 1),
    (2, 4, 5, 7, 2, 1, 1, 1, 0),
    (1, 2, 9, 5, 3, 3, 3, 2, 0),
    (2, 3, 6, 6, 5, 2, 3, 1, 0),
    (1, 4, 2, 2, 3, 3, 3, 1, 1),
]


# --- worked examples derived by hand ---------------------------------------
def test_golden_conv_worked_example():
    g, v = _read_golden("conv2x2_worked_example.txt")
    shp_x = (g["N"], g["C"], g["H"], g["W"])
    shp_w = (g["O"], g["C"], g["KH"], g["KW"])
    x = v["x"].reshape(shp_x)
    wa, wb, wc = (v[k].reshape(shp_w) for k in ("wa", "wb", "wc"))
    y, ta, tb = oracle.conv2d_fwd(x, wa, wb, wc, v["ba"], v["bb"], v["bc"], g["stride"], g["pad"])
    assert np.array_equal(y.ravel(), v["y"])
    assert np.array_equal(ta.ravel(), v["ta"])
    assert np.array_equal(tb.ravel(), v["tb"])
    gy = v["gy"].reshape(y.shape)
    d = oracle.conv2d_bwd(x, wa, wb, wc, v["ba"], v["bb"], v["bc"], gy, g["stride"], g["pad"])
    for k in ("dx", "dwa", "dwb", "dwc", "dba", "dbb", "dbc"):
        assert np.array_equal(d[k].ravel(), v[k]), k


def test_golden_fc_worked_example():
    g, v = _read_golden("fc_worked_example.txt")
    x = v["x"].reshape(g["B"], g["I"])
    wa, wb, wc = (v[k].reshape(g["O"], g["I"]) for k in ("wa", "wb", "wc"))
    y, ta, tb = oracle.linear_fwd(x, wa, wb, wc, v["ba"], v["bb"], v["bc"])
    assert np.array_equal(y.ravel(), v["y"])
    assert np.array_equal(ta.ravel(), v["ta"]) and np.array_equal(tb.ravel(), v["tb"])
    d = oracle.linear_bwd(x, wa, wb, wc, v["ba"], v["bb"], v["bc"], v["gy"].reshape(y.shape))
    for k in ("dx", "dwa", "dwb", "dwc", "dba", "dbb", "dbc"):
        assert np.array_equal(d[k].ravel(), v[k]), k


# --- P6: the paper's own construction from three library convolutions ------
@pytest.mark.parametrize("shape", SHAPES)
def test_forward_equals_three_library_convolutions(shape):
    N, C, H, W, O, KH, KW, s, p = shape
    rng = np.random.default_rng(list(shape))
    x, ws, bs = _rand_case(rng, N, C, H, W, O, KH, KW)
    y, ta, tb = oracle.conv2d_fwd(x, *ws, *bs, s, p)
    Ta, Tb, Tc = _torch_terms(x, ws, bs, s, p)
    assert _rel(ta, Ta) < 1e-13 and _rel(tb, Tb) < 1e-13
    assert _rel(y, Ta * Tb + Tc) < 1e-13


# --- P1: with W_a = 0 the neuron is an ordinary convolution -----------------
@pytest.mark.parametrize("shape", SHAPES[:4])
def test_zero_product_weight_reduces_to_convolution(shape):
    N, C, H, W, O, KH, KW, s, p = shape
    rng = np.random.default_rng([1] + list(shape))
    x, ws, bs = _rand_case(rng, N, C, H, W, O, KH, KW)
    wa0 = np.zeros_like(ws[0])
    y, _, _ = oracle.conv2d_fwd(x, wa0, ws[1], ws[2], np.zeros(O), bs[1], bs[2], s, p)
    ref = F.conv2d(torch.from_numpy(x), torch.from_numpy(ws[2]), torch.from_numpy(bs[2]),
                   stride=s, padding=p).numpy()
    assert _rel(y, ref) < 1e-13
    # W_a = 0 with a non-zero bias b_a: Y = conv(X, W_c + b_a W_b) + (b_c + b_a b_b)
    y2, _, _ = oracle.conv2d_fwd(x, wa0, ws[1], ws[2], bs[0], bs[1], bs[2], s, p)
    weff = ws[2] + bs[0][:, None, None, None] * ws[1]
    beff = bs[2] + bs[0] * bs[1]
    ref2 = F.conv2d(torch.from_numpy(x), torch.from_numpy(weff), torch.from_numpy(beff),
                    stride=s, padding=p).numpy()
    assert _rel(y2, ref2) < 1e-13


# --- P2 / P3: symmetry and bilinearity of the product term -----------------
@pytest.mark.parametrize("shape", SHAPES[:3])
def test_swap_and_scale_invariance(shape):
    N, C, H, W, O, KH, KW, s, p = shape
    rng = np.random.default_rng([2] + list(shape))
    x, (wa, wb, wc), (ba, bb, bc) = _rand_case(rng, N, C, H, W, O, KH, KW)
    y, _, _ = oracle.conv2d_fwd(x, wa, wb, wc, ba, bb, bc, s, p)
    ys, _, _ = oracle.conv2d_fwd(x, wb, wa, wc, bb, ba, bc, s, p)
    assert np.array_equal(y, ys)
    for sc in (2.0, 0.5):
        y2, _, _ = oracle.conv2d_fwd(x, wa * sc, wb / sc, wc, ba * sc, bb / sc, bc, s, p)
        assert np.array_equal(y, y2)
    y3, _, _ = oracle.conv2d_fwd(x, wa * 3.0, wb / 3.0, wc, ba * 3.0, bb / 3.0, bc, s, p)
    assert _rel(y3, y) < 1e-14


# --- P4: the dense layer is the 1x1 special case ----------------------------
def test_conv_on_single_pixel_equals_fc():
    rng = np.random.default_rng(4)
    B, I, O = 5, 7, 6
    x = rng.standard_normal((B, I))
    ws = [rng.standard_normal((O, I)) for _ in range(3)]
    bs = [rng.standard_normal(O) for _ in range(3)]
    yf, taf, tbf = oracle.linear_fwd(x, *ws, *bs)
    # FC against the library matrix product written out as the neuron's three terms
    T = [x @ w.T + b for w, b in zip(ws, bs)]
    assert _rel(yf, T[0] * T[1] + T[2]) < 1e-13
    # 1x1 kernels on 1x1 maps
    yc, tac, tbc = oracle.conv2d_fwd(x[:, :, None, None], *[w[:, :, None, None] for w in ws], *bs, 1, 0)
    assert _rel(yc[:, :, 0, 0], yf) < 1e-13 and _rel(tac[:, :, 0, 0], taf) < 1e-13
    # 3x3 kernels with padding 1 on 1x1 maps only see their centre tap
    w3 = []
    for w in ws:
        k = rng.standard_normal((O, I, 3, 3))
        k[:, :, 1, 1] = w
        w3.append(k)
    y3, _, _ = oracle.conv2d_fwd(x[:, :, None, None], *w3, *bs, 1, 1)
    assert _rel(y3[:, :, 0, 0], yf) < 1e-13
    # and the backward agrees too
    gy = rng.standard_normal((B, O))
    df = oracle.linear_bwd(x, *ws, *bs, gy)
    dc = oracle.conv2d_bwd(x[:, :, None, None], *[w[:, :, None, None] for w in ws], *bs,
                           gy[:, :, None, None], 1, 0)
    assert _rel(dc["dx"][:, :, 0, 0], df["dx"]) < 1e-13
    for k in ("dwa", "dwb", "dwc"):
        assert _rel(dc[k][:, :, 0, 0], df[k]) < 1e-13
    for k in ("dba", "dbb", "dbc"):
        assert _rel(dc[k], df[k]) < 1e-13


# --- P5: closed form with identity kernels -----------------------------------
def test_identity_kernels_closed_form():
    rng = np.random.default_rng(5)
    N, C, H, W = 2, 3, 5, 4
    x = rng.standard_normal((N, C, H, W))
    ident = np.zeros((C, C, 3, 3))
    for c in range(C):
        ident[c, c, 1, 1] = 1.0
    y, _, _ = oracle.conv2d_fwd(x, ident, ident, ident, None, None, None, 1, 1)
    assert np.array_equal(y, x * x + x)


# --- G1: central finite differences (exact for a quadratic loss) ------------
def _fd_check(loss, params, grads, h=1e-3, tol=1e-8):
    for name, arr in params.items():
        flat = arr.reshape(-1)
        fd = np.empty(flat.size)
        for i in range(flat.size):
            old = flat[i]
            flat[i] = old + h
            lp = loss()
            flat[i] = old - h
            lm = loss()
            flat[i] = old
            fd[i] = (lp - lm) / (2 * h)
        g = grads[name].reshape(-1)
        assert _rel(g, fd) < tol, (name, _rel(g, fd))


@pytest.mark.parametrize("s,p", [(1, 0), (1, 1), (2, 0), (2, 1)])
def test_conv_gradients_match_finite_differences(s, p):
    rng = np.random.default_rng([6, s, p])
    N, C, H, W, O, K = 2, 3, 5, 5, 2, 3
    x, ws, bs = _rand_case(rng, N, C, H, W, O, K, K)
    params = {"x": x, "wa": ws[0], "wb": ws[1], "wc": ws[2], "ba": bs[0], "bb": bs[1], "bc": bs[2]}
    y, _, _ = oracle.conv2d_fwd(x, *ws, *bs, s, p)
    gy = rng.standard_normal(y.shape)

    def loss():
        yy, _, _ = oracle.conv2d_fwd(params["x"], params["wa"], params["wb"], params["wc"],
                                     params["ba"], params["bb"], params["bc"], s, p)
        return float(np.sum(gy * yy))

    d = oracle.conv2d_bwd(x, *ws, *bs, gy, s, p)
    grads = {"x": d["dx"], "wa": d["dwa"], "wb": d["dwb"], "wc": d["dwc"],
             "ba": d["dba"], "bb": d["dbb"], "bc": d["dbc"]}
    _fd_check(loss, params, grads)


def test_fc_gradients_match_finite_differences():
    rng = np.random.default_rng(7)
    B, I, O = 3, 4, 5
    x = rng.standard_normal((B, I))
    ws = [rng.standard_normal((O, I)) for _ in range(3)]
    bs = [rng.standard_normal(O) for _ in range(3)]
    gy = rng.standard_normal((B, O))
    params = {"x": x, "wa": ws[0], "wb": ws[1], "wc": ws[2], "ba": bs[0], "bb": bs[1], "bc": bs[2]}

    def loss():
        yy, _, _ = oracle.linear_fwd(params["x"], params["wa"], params["wb"], params["wc"],
                                     params["ba"], params["bb"], params["bc"])
        return float(np.sum(gy * yy))

    d = oracle.linear_bwd(x, *ws, *bs, gy)
    grads = {"x": d["dx"], "wa": d["dwa"], "wb": d["dwb"], "wc": d["dwc"],
             "ba": d["dba"], "bb": d["dbb"], "bc": d["dbc"]}
    _fd_check(loss, params, grads)


# --- G2: the paper's AD path (eq:AD) via torch autograd in fp64 -------------
@pytest.mark.parametrize("shape", SHAPES)
def test_gradients_match_autograd_of_composition(shape):
    N, C, H, W, O, KH, KW, s, p = shape
    rng = np.random.default_rng([8] + list(shape))
    x, ws, bs = _rand_case(rng, N, C, H, W, O, KH, KW)
    tx = torch.from_numpy(x.copy()).requires_grad_()
    tw = [torch.from_numpy(w.copy()).requires_grad_() for w in ws]
    tbias = [torch.from_numpy(b.copy()).requires_grad_() for b in bs]
    T = [F.conv2d(tx, w, b, stride=s, padding=p) for w, b in zip(tw, tbias)]
    y = T[0] * T[1] + T[2]
    gy = rng.standard_normal(tuple(y.shape))
    y.backward(torch.from_numpy(gy))
    d = oracle.conv2d_bwd(x, *ws, *bs, gy, s, p)
    assert _rel(d["dx"], tx.grad.numpy()) < 1e-12
    for k, t in zip(("dwa", "dwb", "dwc"), tw):
        assert _rel(d[k], t.grad.numpy()) < 1e-12, k
    for k, t in zip(("dba", "dbb", "dbc"), tbias):
        assert _rel(d[k], t.grad.numpy()) < 1e-12, k


# --- G3 / G4: covariance of the gradients under the P2 / P3 maps ------------
def test_gradient_covariance_under_swap_and_scale():
    rng = np.random.default_rng(9)
    N, C, H, W, O, K, s, p = 2, 3, 6, 5, 4, 3, 1, 1
    x, (wa, wb, wc), (ba, bb, bc) = _rand_case(rng, N, C, H, W, O, K, K)
    y, _, _ = oracle.conv2d_fwd(x, wa, wb, wc, ba, bb, bc, s, p)
    gy = rng.standard_normal(y.shape)
    d = oracle.conv2d_bwd(x, wa, wb, wc, ba, bb, bc, gy, s, p)
    sw_ = oracle.conv2d_bwd(x, wb, wa, wc, bb, ba, bc, gy, s, p)
    assert np.array_equal(sw_["dwa"], d["dwb"]) and np.array_equal(sw_["dwb"], d["dwa"])
    assert np.array_equal(sw_["dba"], d["dbb"]) and np.array_equal(sw_["dbb"], d["dba"])
    assert np.array_equal(sw_["dwc"], d["dwc"])
    assert _rel(sw_["dx"], d["dx"]) < 1e-14
    sc = oracle.conv2d_bwd(x, wa * 2, wb / 2, wc, ba * 2, bb / 2, bc, gy, s, p)
    assert np.array_equal(sc["dwa"], d["dwa"] / 2) and np.array_equal(sc["dba"], d["dba"] / 2)
    assert np.array_equal(sc["dwb"], d["dwb"] * 2) and np.array_equal(sc["dbb"], d["dbb"] * 2)
    assert np.array_equal(sc["dwc"], d["dwc"]) and np.array_equal(sc["dx"], d["dx"])


# --- G5: partner-term wiring with W_a = 0 -----------------------------------
def test_gradients_with_zero_product_weight():
    rng = np.random.default_rng(10)
    N, C, H, W, O, K, s, p = 2, 3, 6, 6, 4, 3, 2, 1
    x, (wa, wb, wc), (ba, bb, bc) = _rand_case(rng, N, C, H, W, O, K, K)
    wa[:] = 0
    ba[:] = 0
    y, _, tb = oracle.conv2d_fwd(x, wa, wb, wc, ba, bb, bc, s, p)
    gy = rng.standard_normal(y.shape)
    d = oracle.conv2d_bwd(x, wa, wb, wc, ba, bb, bc, gy, s, p)
    tx = torch.from_numpy(x.copy()).requires_grad_()
    twc = torch.from_numpy(wc.copy()).requires_grad_()
    F.conv2d(tx, twc, None, stride=s, padding=p).backward(torch.from_numpy(gy))
    assert _rel(d["dx"], tx.grad.numpy()) < 1e-13
    assert _rel(d["dwc"], twc.grad.numpy()) < 1e-13
    assert np.all(d["dwb"] == 0) and np.all(d["dbb"] == 0)
    # dW_a is the correlation of G o T_b with X, which is not zero
    txa = torch.from_numpy(x.copy())
    twa = torch.zeros_like(torch.from_numpy(wa), requires_grad=True)
    F.conv2d(txa, twa, None, stride=s, padding=p).backward(torch.from_numpy(gy * tb))
    assert _rel(d["dwa"], twa.grad.numpy()) < 1e-13 and np.linalg.norm(d["dwa"]) > 0


# --- sampled evaluation used by the full-size checks ------------------------
def test_sampled_functions_agree_with_full():
    rng = np.random.default_rng(11)
    N, C, H, W, O, K, s, p = 2, 4, 7, 6, 5, 3, 2, 1
    x, ws, bs = _rand_case(rng, N, C, H, W, O, K, K)
    y, ta, tb = oracle.conv2d_fwd(x, *ws, *bs, s, p)
    gy = rng.standard_normal(y.shape)
    d = oracle.conv2d_bwd(x, *ws, *bs, gy, s, p)
    # every element of every output (the samplers must agree everywhere, not at a few points)
    idx = np.array(list(np.ndindex(*y.shape)))
    ys, tas, tbs = oracle.conv2d_fwd_at(x, *ws, *bs, idx, s, p)
    n, o, i, j = idx.T
    assert np.array_equal(ys, y[n, o, i, j]) and np.array_equal(tas, ta[n, o, i, j])
    assert np.array_equal(tbs, tb[n, o, i, j])
    xi = np.array(list(np.ndindex(*x.shape)))
    dxs = oracle.conv2d_dx_at(x, *ws, *bs, gy, xi, s, p)
    ref = d["dx"][tuple(xi.T)]
    assert np.max(np.abs(dxs - ref)) <= 1e-13 * max(1.0, np.max(np.abs(ref)))
    # every channel at every input pixel: the same terms in the same order as the
    # per-element sampler, so the same bits, and the full oracle's dX
    pix = np.array(list(np.ndindex(N, H, W)))
    dxp = oracle.conv2d_dx_pixels(x, *ws, *bs, gy, pix, s, p)
    pn, ph_, pw_ = pix.T
    assert dxp.shape == (len(pix), C)
    assert np.max(np.abs(dxp - d["dx"][pn, :, ph_, pw_])) <= 1e-13 * max(1.0, np.max(np.abs(ref)))
    per_elem = oracle.conv2d_dx_at(x, *ws, *bs, gy,
                                   np.array([[n_, c_, h_, w_] for (n_, h_, w_) in pix for c_ in range(C)]), s, p)
    assert np.array_equal(dxp.ravel(), per_elem)
    for o in range(O):
        dc = oracle.conv2d_dw_channel(x, *ws, *bs, gy, o, s, p)
        for k in ("dwa", "dwb", "dwc"):
            assert _rel(dc[k], d[k][o]) < 1e-13
        for k in ("dba", "dbb", "dbc"):
            assert abs(dc[k][0] - d[k][o]) <= 1e-13 * max(1.0, abs(d[k][o]))
    # FC sampled versions
    B, I, O2 = 6, 5, 4
    xf = rng.standard_normal((B, I))
    wf = [rng.standard_normal((O2, I)) for _ in range(3)]
    bf = [rng.standard_normal(O2) for _ in range(3)]
    yf, taf, tbf = oracle.linear_fwd(xf, *wf, *bf)
    gf = rng.standard_normal(yf.shape)
    df = oracle.linear_bwd(xf, *wf, *bf, gf)
    # every output of every sampled element, the whole index space
    fidx = np.array([[b, o] for b in range(B) for o in range(O2)])
    ysf, tasf, tbsf = oracle.linear_fwd_at(xf, *wf, *bf, fidx)
    for k, (b, o) in enumerate(fidx):
        assert ysf[k] == yf[b, o] and tasf[k] == taf[b, o] and tbsf[k] == tbf[b, o]
    dxr = oracle.linear_dx_rows(xf, *wf, *bf, gf, [2, 4])
    assert _rel(dxr, df["dx"][[2, 4]]) < 1e-13
    for o in range(O2):
        dr = oracle.linear_dw_row(xf, *wf, *bf, gf, o)
        for k in ("dwa", "dwb", "dwc"):
            assert _rel(dr[k], df[k][o]) < 1e-13, (k, o)
        for k in ("dba", "dbb", "dbc"):
            assert abs(dr[k][0] - df[k][o]) <= 1e-13 * max(1.0, abs(df[k][o])), (k, o)
    # the full dense backward against numpy closed forms (so that the sampled
    # functions are pinned through it, not only to it)
    ga, gb = gf * tbf, gf * taf
    assert _rel(df["dwa"], ga.T @ xf) < 1e-13 and _rel(df["dwb"], gb.T @ xf) < 1e-13
    assert _rel(df["dwc"], gf.T @ xf) < 1e-13
    assert _rel(df["dba"], ga.sum(0)) < 1e-13 and _rel(df["dbb"], gb.sum(0)) < 1e-13
    assert _rel(df["dbc"], gf.sum(0)) < 1e-13
    assert _rel(df["dx"], ga @ wf[0] + gb @ wf[1] + gf @ wf[2]) < 1e-13
    assert _rel(tbf, xf @ wf[1].T + bf[1]) < 1e-13


# --- the 3x parameter relation of Table 1 / Table 3 -------------------------
def test_parameter_count_is_three_first_order_layers():
    # VGG-16 first-order 1.47E+7 vs quadratic 4.41E+7 parameters (Table 3).
    assert abs(3 * 1.47e7 - 4.41e7) / 4.41e7 < 1e-9
    O, C, K = 7, 5, 3
    rng = np.random.default_rng(12)
    x, ws, bs = _rand_case(rng, 1, C, 4, 4, O, K, K)
    n_params = sum(w.size for w in ws) + sum(b.size for b in bs)
    assert n_params == 3 * (O * C * K * K + O)
