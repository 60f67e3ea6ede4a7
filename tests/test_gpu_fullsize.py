"""GPU parity at the full workload sizes, in the launch configuration the
benchmark times (default planner, workspace of the queried size).

The whole outputs are too large for the fp64 oracle, so it recomputes a
sample of them one by one: forward outputs Y, T_a, T_b at random positions
plus the corners of the index space, input-gradient entries likewise (border
pixels included), and the complete weight and bias gradients of a few output
channels (first, last, one random).  The normwise relative error over each
sampled set must meet the same limits as the small cases: fp32 forward 1e-5,
gradients 1e-4; bf16 with fp32 accumulation 2e-2.

Workloads: the 13 layers of a CIFAR VGG-16 at batch 128 (bf16), the distinct
layer shapes of a CIFAR ResNet-20 at batch 256 (fp32 and bf16), one large
256->256 layer on 64 x 56 x 56 (bf16) and a 8192 x 4096 -> 4096 dense layer
(bf16).
"""
import itertools

import numpy as np
import pytest
import torch

import oracle
import synth

pytestmark = pytest.mark.gpu

import qlh  # noqa: E402

N_SAMPLES = 96


def _corners(extents):
    return [list(c) for c in itertools.product(*[(0, e - 1) for e in extents])]


def _sample_idx(rng, extents, k=N_SAMPLES):
    """k index tuples: every corner of the box, the rest uniform."""
    pts = _corners(extents)
    rest = k - len(pts)
    rnd = np.stack([rng.integers(0, e, size=rest) for e in extents], axis=1)
    return np.concatenate([np.array(pts, dtype=np.int64), rnd.astype(np.int64)], axis=0)


def _at(t, *idx):
    """Gather t[idx] on the device and return it as float64 numpy."""
    ti = tuple(torch.from_numpy(np.ascontiguousarray(a)).to(t.device) for a in idx)
    return t[ti].double().cpu().numpy()


def _check(name, got, ref, bf16, grad):
    e = qlh.relerr(got, ref)
    lim = qlh.tol(bf16, grad)
    assert e <= lim, f"{name}: normwise relative error {e:.3e} > {lim:.0e}"
    return e


def _conv_case(cfg_id, layer_id, L, bf16):
    print(f"full-size conv cfg={cfg_id} layer={layer_id} N={L.n} C={L.c} {L.h}x{L.w} O={L.o} "
          f"k={L.k} s={L.stride} p={L.pad} bf16={bf16}", flush=True)
    inp = synth.conv_inputs(cfg_id, layer_id, L, bf16=bf16)
    dev = qlh.run_conv(inp, L.stride, L.pad, bf16)
    f64 = {k: np.ascontiguousarray(v, dtype=np.float64) for k, v in inp.items()}
    args = (f64["x"], f64["wa"], f64["wb"], f64["wc"], f64["ba"], f64["bb"], f64["bc"])
    rng = np.random.default_rng([900, cfg_id, layer_id, int(bf16)])

    # forward: (n, o, i, j)
    idx = _sample_idx(rng, (L.n, L.o, L.ho, L.wo))
    ry, rta, rtb = oracle.conv2d_fwd_at(*args, idx, L.stride, L.pad)
    n, o, i, j = idx.T
    for key, ref in (("y", ry), ("ta", rta), ("tb", rtb)):
        got = _at(dev[key], n, i, j, o)  # NHWC on the device
        _check(key, got, ref, bf16, False)

    # input gradient: (n, c, h, w)
    idx = _sample_idx(rng, (L.n, L.c, L.h, L.w))
    rdx = oracle.conv2d_dx_at(*args, f64["gy"], idx, L.stride, L.pad)
    n, c, h, w = idx.T
    _check("dx", _at(dev["dx"], n, h, w, c), rdx, bf16, True)

    # weight and bias gradients of whole output channels
    chans = sorted({0, L.o - 1, int(rng.integers(0, L.o))})
    got = {k: [] for k in ("dwa", "dwb", "dwc", "dba", "dbb", "dbc")}
    ref = {k: [] for k in got}
    for oc in chans:
        r = oracle.conv2d_dw_channel(*args, f64["gy"], oc, L.stride, L.pad)
        for t in ("a", "b", "c"):
            # device dW_t is O x KH x KW x C; the oracle's channel slice is C x KH x KW
            got["dw" + t].append(dev["dw" + t][oc].permute(2, 0, 1).double().cpu().numpy().ravel())
            ref["dw" + t].append(r["dw" + t].ravel())
            got["db" + t].append(dev["db" + t][oc:oc + 1].double().cpu().numpy())
            ref["db" + t].append(r["db" + t])
    for k in got:
        _check(k, np.concatenate(got[k]), np.concatenate(ref[k]), bf16, True)


VGG = synth.vgg16_layers(128)


@pytest.mark.parametrize("layer_id", range(len(VGG)), ids=lambda i: f"L{i + 1}")
def test_vgg16_layer_full_size(layer_id):
    _conv_case(2, layer_id, VGG[layer_id], bf16=True)


RESNET = synth.resnet20_layers(256)


def _distinct(layers):
    seen, ids = set(), []
    for i, L in enumerate(layers):
        key = (L.c, L.h, L.w, L.o, L.k, L.stride, L.pad)
        if key not in seen:
            seen.add(key)
            ids.append(i)
    return ids


@pytest.mark.parametrize("bf16", [False, True], ids=["fp32", "bf16"])
@pytest.mark.parametrize("layer_id", _distinct(RESNET), ids=lambda i: f"conv{i}")
def test_resnet20_layer_full_size(layer_id, bf16):
    _conv_case(3, layer_id, RESNET[layer_id], bf16=bf16)


def test_large_conv_full_size():
    _conv_case(4, 0, synth.LARGE_BF16, bf16=True)


def test_dense_full_size():
    D = synth.DENSE_BF16
    print(f"full-size dense {D.batch}x{D.inp}->{D.out} bf16", flush=True)
    inp = synth.dense_inputs(5, 0, D, bf16=True)
    dev = qlh.run_linear(inp, True)
    f64 = {k: np.ascontiguousarray(v, dtype=np.float64) for k, v in inp.items()}
    args = (f64["x"], f64["wa"], f64["wb"], f64["wc"], f64["ba"], f64["bb"], f64["bc"])
    rng = np.random.default_rng([901, 5])

    idx = _sample_idx(rng, (D.batch, D.out))
    ry, rta, rtb = oracle.linear_fwd_at(*args, idx)
    b, o = idx.T
    for key, ref in (("y", ry), ("ta", rta), ("tb", rtb)):
        _check(key, _at(dev[key], b, o), ref, True, False)

    rows = np.array([0, D.batch - 1, int(rng.integers(0, D.batch))], dtype=np.int64)
    rdx = oracle.linear_dx_rows(*args, f64["gy"], rows)
    _check("dx", _at(dev["dx"], rows), rdx, True, True)

    chans = sorted({0, D.out - 1, int(rng.integers(0, D.out))})
    got = {k: [] for k in ("dwa", "dwb", "dwc", "dba", "dbb", "dbc")}
    ref = {k: [] for k in got}
    for oc in chans:
        r = oracle.linear_dw_row(*args, f64["gy"], oc)
        for t in ("a", "b", "c"):
            got["dw" + t].append(dev["dw" + t][oc].double().cpu().numpy())
            ref["dw" + t].append(r["dw" + t])
            got["db" + t].append(dev["db" + t][oc:oc + 1].double().cpu().numpy())
            ref["db" + t].append(r["db" + t])
    for k in got:
        # zero biases: db_t is still the column sum of G_t, non-zero
        _check(k, np.concatenate(got[k]), np.concatenate(ref[k]), True, True)


def test_small_fp32_whole_tensors():
    """The small fp32 workload (N=2, 16->16, 8x8) is cheap enough to compare in full."""
    L = synth.SMALL_FP32
    inp = synth.conv_inputs(1, 0, L, bf16=False)
    got = qlh.conv_to_np(qlh.run_conv(inp, L.stride, L.pad, False))
    args = (inp["x"], inp["wa"], inp["wb"], inp["wc"], inp["ba"], inp["bb"], inp["bc"])
    y, ta, tb = oracle.conv2d_fwd(*args, L.stride, L.pad)
    ref = oracle.conv2d_bwd(*args, inp["gy"], L.stride, L.pad)
    ref.update({"y": y, "ta": ta, "tb": tb})
    for k in ("y", "ta", "tb", "dx", "dwa", "dwb", "dwc", "dba", "dbb", "dbc"):
        _check(k, got[k], ref[k], False, k not in ("y", "ta", "tb"))
