"""GPU parity at the full workload sizes, in the launch configuration the
benchmark times (default planner, workspace of the queried size).

Every output is compared in two ways (qlh):
* the normwise relative error over the compared set, against the limits
  fp32 forward 1e-5 / gradients 1e-4, bf16 with fp32 accumulation 2e-2;
* element by element, against a bound derived from the arithmetic (the
  rounding of each output and operand plus the fp32 accumulation error of
  its reduction), with the magnitudes from the oracle on |inputs|.

Whole tensors where the fp64 oracle can afford them: the 13 layers of a
CIFAR VGG-16 at batch 128 (bf16), the distinct layer shapes of a CIFAR
ResNet-20 at batch 256 (fp32 and bf16), the small fp32 layer.  For the
64 x 256 x 56 x 56 layer and the 8192 x 4096 -> 4096 dense layer, complete
blocks of every output in the shape of the largest workgroup tile any kernel
of the pass uses (256 x 256), at the first, the last and one interior tile
position: forward Y, T_a, T_b; input gradient dX (whole rows of channels for
the dense layer); whole output channels of dW_t and db_t (all of (r, q, c),
so every weight-gradient row tile and every split-K part of those channels:
the first 64-channel tile and the last 16 channels for the 56 x 56 layer).
"""
import numpy as np
import pytest
import torch

import oracle
import synth

pytestmark = pytest.mark.gpu

import qlh  # noqa: E402

TILE = 256  # the largest workgroup tile extent along channels and pixels


def _check(name, kind, got, ref, mag, bf16, K):
    e = qlh.relerr(got, ref)
    lim = qlh.tol(bf16, kind not in ("y", "ta", "tb"))
    assert e <= lim, f"{name}: normwise relative error {e:.3e} > {lim:.0e}"
    qlh.check_elementwise(name, kind, got, ref, mag, bf16, K)
    return e


def _abs_args(f64):
    return {k: np.abs(v) for k, v in f64.items()}


def _conv_whole(cfg_id, layer_id, L, bf16):
    print(f"full-size conv (whole tensors) cfg={cfg_id} layer={layer_id} N={L.n} C={L.c} {L.h}x{L.w} O={L.o} "
          f"k={L.k} s={L.stride} p={L.pad} bf16={bf16}", flush=True)
    inp = synth.conv_inputs(cfg_id, layer_id, L, bf16=bf16)
    got = qlh.conv_to_np(qlh.run_conv(inp, L.stride, L.pad, bf16))
    f64 = {k: np.ascontiguousarray(v, dtype=np.float64) for k, v in inp.items()}
    keys = ("x", "wa", "wb", "wc", "ba", "bb", "bc")
    ref = {}
    ref["y"], ref["ta"], ref["tb"] = oracle.conv2d_fwd(*[f64[k] for k in keys], L.stride, L.pad)
    ref.update(oracle.conv2d_bwd(*[f64[k] for k in keys], f64["gy"], L.stride, L.pad))
    a = _abs_args(f64)
    mag = {}
    mag["y"], mag["ta"], mag["tb"] = oracle.conv2d_fwd(*[a[k] for k in keys], L.stride, L.pad)
    mag.update(oracle.conv2d_bwd(*[a[k] for k in keys], a["gy"], L.stride, L.pad))
    ho, wo = ref["y"].shape[2:]
    K = {"fwd": L.c * L.k * L.k + 1, "dx": 3 * L.o * L.k * L.k, "dw": L.n * ho * wo}
    for k in ("y", "ta", "tb", "dx", "dwa", "dwb", "dwc", "dba", "dbb", "dbc"):
        kk = K["fwd"] if k in ("y", "ta", "tb") else (K["dx"] if k == "dx" else K["dw"])
        _check(k, k, got[k], ref[k], mag[k], bf16, kk)


VGG = synth.vgg16_layers(128)


@pytest.mark.parametrize("layer_id", range(len(VGG)), ids=lambda i: f"L{i + 1}")
def test_vgg16_layer_full_size(layer_id):
    _conv_whole(2, layer_id, VGG[layer_id], bf16=True)


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
    _conv_whole(3, layer_id, RESNET[layer_id], bf16=bf16)


def test_small_fp32_whole_tensors():
    """The small fp32 workload (N=2, 16->16, 8x8), whole tensors."""
    _conv_whole(1, 0, synth.SMALL_FP32, bf16=False)


def _blocks(extent, rng):
    """Start of the first, the last and one interior TILE-aligned block of an extent."""
    last = max(0, extent - TILE)
    mid = int(rng.integers(1, max(2, extent // TILE))) * TILE if extent > 2 * TILE else 0
    return sorted({0, min(mid, last), last})


def _at(t, *idx):
    ti = tuple(torch.from_numpy(np.ascontiguousarray(a)).to(t.device) for a in idx)
    return t[ti].double().cpu().numpy()


def test_large_conv_full_size_tiles():
    L = synth.LARGE_BF16
    print("full-size large conv, complete tile blocks", flush=True)
    inp = synth.conv_inputs(4, 0, L, bf16=True)
    dev = qlh.run_conv(inp, L.stride, L.pad, True)
    f64 = {k: np.ascontiguousarray(v, dtype=np.float64) for k, v in inp.items()}
    a = _abs_args(f64)
    keys = ("x", "wa", "wb", "wc", "ba", "bb", "bc")
    args, aargs = [f64[k] for k in keys], [a[k] for k in keys]
    rng = np.random.default_rng([900, 4])
    ho, wo = L.ho, L.wo
    M = L.n * ho * wo

    # forward: blocks of TILE output channels x TILE output pixels (pixel m = (n ho + i) wo + j)
    for o0 in _blocks(L.o, rng):
        for m0 in _blocks(M, rng):
            o = np.arange(o0, min(L.o, o0 + TILE))
            m = np.arange(m0, min(M, m0 + TILE))
            oo, mm = np.meshgrid(o, m, indexing="ij")
            n, rem = np.divmod(mm.ravel(), ho * wo)
            i, j = np.divmod(rem, wo)
            idx = np.stack([n, oo.ravel(), i, j], axis=1)
            ref = oracle.conv2d_fwd_at(*args, idx, L.stride, L.pad)
            mag = oracle.conv2d_fwd_at(*aargs, idx, L.stride, L.pad)
            for key, r, g in zip(("y", "ta", "tb"), ref, mag):
                _check(f"{key} block o{o0} m{m0}", key, _at(dev[key], n, i, j, idx[:, 1]), r, g, True,
                       L.c * 9 + 1)

    # input gradient: blocks of TILE input channels x TILE input pixels (the
    # oracle's dX at every channel of each block's pixels)
    Mi = L.n * L.h * L.w
    for m0 in _blocks(Mi, rng):
        m = np.arange(m0, min(Mi, m0 + TILE))
        n, rem = np.divmod(m, L.h * L.w)
        h, w = np.divmod(rem, L.w)
        pix = np.stack([n, h, w], axis=1)
        ref_all = oracle.conv2d_dx_pixels(*args, f64["gy"], pix, L.stride, L.pad)
        mag_all = oracle.conv2d_dx_pixels(*aargs, a["gy"], pix, L.stride, L.pad)
        for c0 in _blocks(L.c, rng):
            c = np.arange(c0, min(L.c, c0 + TILE))
            mm, cc = np.meshgrid(np.arange(len(m)), c, indexing="ij")
            got = _at(dev["dx"], n[mm.ravel()], h[mm.ravel()], w[mm.ravel()], cc.ravel())
            _check(f"dx block c{c0} m{m0}", "dx", got, ref_all[mm.ravel(), cc.ravel()], mag_all[mm.ravel(), cc.ravel()],
                   True, 3 * L.o * 9)


def test_large_conv_full_size_weight_channels():
    """Whole output channels of dW_t and db_t of the large layer: the first
    64-channel tile complete and the last 16 channels (one wave's slice of the
    last tile)."""
    L = synth.LARGE_BF16
    print("full-size large conv, weight-gradient channels", flush=True)
    inp = synth.conv_inputs(4, 0, L, bf16=True)
    dev = qlh.run_conv(inp, L.stride, L.pad, True)
    f64 = {k: np.ascontiguousarray(v, dtype=np.float64) for k, v in inp.items()}
    a = _abs_args(f64)
    keys = ("x", "wa", "wb", "wc", "ba", "bb", "bc")
    args, aargs = [f64[k] for k in keys], [a[k] for k in keys]
    M = L.n * L.ho * L.wo

    chans = list(range(0, 64)) + list(range(L.o - 16, L.o))
    got = {k: [] for k in ("dwa", "dwb", "dwc", "dba", "dbb", "dbc")}
    ref = {k: [] for k in got}
    mag = {k: [] for k in got}
    for oc in chans:
        r = oracle.conv2d_dw_channel(*args, f64["gy"], oc, L.stride, L.pad)
        g = oracle.conv2d_dw_channel(*aargs, a["gy"], oc, L.stride, L.pad)
        for t in ("a", "b", "c"):
            got["dw" + t].append(dev["dw" + t][oc].permute(2, 0, 1).double().cpu().numpy().ravel())
            got["db" + t].append(dev["db" + t][oc:oc + 1].double().cpu().numpy())
            for dst, src in ((ref, r), (mag, g)):
                dst["dw" + t].append(src["dw" + t].ravel())
                dst["db" + t].append(src["db" + t])
    for k in got:
        _check(k, k, np.concatenate(got[k]), np.concatenate(ref[k]), np.concatenate(mag[k]), True, M)


def test_dense_full_size_tiles():
    D = synth.DENSE_BF16
    print(f"full-size dense {D.batch}x{D.inp}->{D.out} bf16, complete tile blocks", flush=True)
    inp = synth.dense_inputs(5, 0, D, bf16=True)
    dev = qlh.run_linear(inp, True)
    f64 = {k: np.ascontiguousarray(v, dtype=np.float64) for k, v in inp.items()}
    a = _abs_args(f64)
    keys = ("x", "wa", "wb", "wc", "ba", "bb", "bc")
    args, aargs = [f64[k] for k in keys], [a[k] for k in keys]
    rng = np.random.default_rng([901, 5])

    for b0 in _blocks(D.batch, rng):
        for o0 in _blocks(D.out, rng):
            bb, oo = np.meshgrid(np.arange(b0, b0 + TILE), np.arange(o0, o0 + TILE), indexing="ij")
            idx = np.stack([bb.ravel(), oo.ravel()], axis=1)
            ref = oracle.linear_fwd_at(*args, idx)
            mag = oracle.linear_fwd_at(*aargs, idx)
            for key, r, g in zip(("y", "ta", "tb"), ref, mag):
                _check(f"{key} block b{b0} o{o0}", key, _at(dev[key], idx[:, 0], idx[:, 1]), r, g, True, D.inp + 1)

    # input gradient: whole rows (every input channel), TILE rows at each end
    for b0 in (0, D.batch - TILE):
        rows = np.arange(b0, b0 + TILE)
        ref = oracle.linear_dx_rows(*args, f64["gy"], rows)
        mag = oracle.linear_dx_rows(*aargs, a["gy"], rows)
        _check(f"dx rows {b0}", "dx", _at(dev["dx"], rows), ref, mag, True, 3 * D.out)

    # weight and bias gradients: whole rows o, a 64-row tile at each end
    chans = list(range(0, 64)) + list(range(D.out - 64, D.out))
    got = {k: [] for k in ("dwa", "dwb", "dwc", "dba", "dbb", "dbc")}
    ref = {k: [] for k in got}
    mag = {k: [] for k in got}
    for oc in chans:
        r = oracle.linear_dw_row(*args, f64["gy"], oc)
        g = oracle.linear_dw_row(*aargs, a["gy"], oc)
        for t in ("a", "b", "c"):
            got["dw" + t].append(dev["dw" + t][oc].double().cpu().numpy())
            got["db" + t].append(dev["db" + t][oc:oc + 1].double().cpu().numpy())
            for dst, src in ((ref, r), (mag, g)):
                dst["dw" + t].append(src["dw" + t])
                dst["db" + t].append(src["db" + t])
    for k in got:
        _check(k, k, np.concatenate(got[k]), np.concatenate(ref[k]), np.concatenate(mag[k]), True, D.batch)
