"""The earlier neuron types (T4, T4 + identity, T3, T2, T2&4; arXiv 2204.01701
Table 1 and the Table 3 baselines) through the C ABI against the fp64
oracle, element by element (normwise relative error), in fp32 and bf16:
forward Y and saved maps, input gradient, weight and bias gradients, as
convolution and as fully-connected layers."""
import numpy as np
import pytest
import torch

import oracle
import synth

pytestmark = pytest.mark.gpu

import qlh  # noqa: E402
import paper_2204_01701_amd as ql  # noqa: E402

DEV = qlh.DEV
T4, T4I, T3, T2 = ql.QL_NEURON_T4, ql.QL_NEURON_T4_IDENTITY, ql.QL_NEURON_T3, ql.QL_NEURON_T2
T24 = ql.QL_NEURON_T24
TYPES = (T4, T4I, T3, T2, T24)
NAMES = {T4: "T4", T4I: "T4I", T3: "T3", T2: "T2", T24: "T24"}
TERMS = ql.NEURON_TERMS

# N, C, H, W, O, K, stride, pad.  The shortcut of T4 + identity needs C == O
# and an unchanged map, so it takes the shapes marked same=True.
SHAPES = [
    ((2, 24, 10, 9, 48, 3, 1, 1), False),   # ragged channel and pixel tiles
    ((1, 64, 9, 7, 64, 3, 1, 1), True),     # channel-aligned steps, ragged pixels
    ((2, 16, 9, 9, 16, 3, 2, 1), False),    # stride 2
    ((2, 3, 8, 8, 8, 3, 1, 1), False),      # 3-channel input (padded / generic paths)
    ((4, 256, 4, 4, 256, 3, 1, 1), True),   # few pixels, long K: split-K and its reductions
    ((2, 128, 6, 6, 128, 1, 1, 0), True),   # 1x1
    ((1, 12, 7, 5, 12, 3, 1, 1), True),     # channels not a multiple of the bf16 vector
]
CASES = [(n, sh) for n in TYPES for sh, same in SHAPES if n != T4I or same]
IDS = [f"{NAMES[n]}-{'x'.join(map(str, sh))}" for n, sh in CASES]


def _run_conv_neuron(neuron, inp, s, p, bf16):
    N, C, H, W = inp["x"].shape
    O, _, K, _ = inp["wa"].shape
    nt = TERMS[neuron]
    d = ql.conv_desc(N, C, H, W, O, K, K, s, p, qlh.qdtype(bf16), neuron)
    dt = qlh.tdtype(bf16)
    x = qlh.nchw_to_dev(inp["x"], bf16)
    w = [qlh.oihw_to_dev(inp[k], bf16) if i < nt else None for i, k in enumerate(("wa", "wb", "wc"))]
    b = [qlh.vec_to_dev(inp[k]) if i < nt else None for i, k in enumerate(("ba", "bb", "bc"))]
    y = torch.empty((N, d.ho, d.wo, O), device=DEV, dtype=dt)
    ta = torch.empty_like(y) if neuron != T2 else None
    tb = torch.empty_like(y) if nt >= 2 else None
    ql.qlayer_conv2d_fwd(d, x, *w, *b, y, ta, tb)
    gy = qlh.nchw_to_dev(inp["gy"], bf16)
    dx = torch.empty_like(x)
    if neuron == T24:  # its c term's chain rule through X o X needs X
        ql.qlayer_conv2d_bwd_data_ex(d, gy, ta, tb, x, *w, dx)
    else:
        ql.qlayer_conv2d_bwd_data(d, gy, x if neuron == T2 else ta, tb, *w, dx)
    dw = [torch.empty((O, K, K, C), device=DEV, dtype=torch.float32) if i < nt else None for i in range(3)]
    db = [torch.empty(O, device=DEV, dtype=torch.float32) if i < nt else None for i in range(3)]
    ql.qlayer_conv2d_bwd_weight(d, x, gy, ta, tb, *dw, *db)
    torch.cuda.synchronize()
    out = {"y": y, "dx": dx}
    if ta is not None:
        out["ta"] = ta
    if tb is not None:
        out["tb"] = tb
    for i, (kw, kb) in enumerate((("dwa", "dba"), ("dwb", "dbb"), ("dwc", "dbc"))[:nt]):
        out[kw], out[kb] = dw[i], db[i]
    return qlh.conv_to_np(out)


@pytest.mark.parametrize("bf16", [False, True], ids=["fp32", "bf16"])
@pytest.mark.parametrize("neuron,shape", CASES, ids=IDS)
def test_conv_neuron_matches_oracle(neuron, shape, bf16):
    N, C, H, W, O, K, s, p = shape
    print(f"neuron {NAMES[neuron]} shape {shape} bf16={bf16}", flush=True)
    inp = synth.random_conv_case([500, neuron] + list(shape), N, C, H, W, O, K, K, s, p, bf16=bf16)
    nt = TERMS[neuron]
    w = [inp["wa"], inp["wb"] if nt >= 2 else None, inp["wc"] if nt >= 3 else None]
    b = [inp["ba"], inp["bb"] if nt >= 2 else None, inp["bc"] if nt >= 3 else None]
    y, ta, tb = oracle.conv2d_fwd_neuron(neuron, inp["x"], *w, *b, stride=s, pad=p)
    ref = oracle.conv2d_bwd_neuron(neuron, inp["x"], *w, *b, inp["gy"], stride=s, pad=p)
    ref["y"] = y
    if neuron != T2:
        ref["ta"] = ta
    if nt >= 2:
        ref["tb"] = tb
    got = _run_conv_neuron(neuron, inp, s, p, bf16)
    assert sorted(got) == sorted(ref)
    for k in ref:
        e = qlh.relerr(got[k], ref[k])
        assert e <= qlh.tol(bf16, k not in ("y", "ta", "tb")), f"{k}: normwise relative error {e:.3e}"


@pytest.mark.parametrize("bf16", [False, True], ids=["fp32", "bf16"])
@pytest.mark.parametrize("neuron", TYPES, ids=[NAMES[n] for n in TYPES])
def test_linear_neuron_matches_oracle(neuron, bf16):
    B, I, O = 96, 72, 72 if neuron == T4I else 40
    print(f"neuron {NAMES[neuron]} dense {B}x{I}->{O} bf16={bf16}", flush=True)
    inp = synth.random_dense_case([501, neuron, B, I, O], B, I, O, bf16=bf16)
    nt = TERMS[neuron]
    w = [inp["wa"], inp["wb"] if nt >= 2 else None, inp["wc"] if nt >= 3 else None]
    b = [inp["ba"], inp["bb"] if nt >= 2 else None, inp["bc"] if nt >= 3 else None]
    y, ta, tb = oracle.linear_fwd_neuron(neuron, inp["x"], *w, *b)
    ref = oracle.linear_bwd_neuron(neuron, inp["x"], *w, *b, inp["gy"])
    ref["y"] = y
    d = ql.linear_desc(B, I, O, qlh.qdtype(bf16), neuron)
    dt = qlh.tdtype(bf16)
    x = torch.from_numpy(inp["x"]).to(DEV, dt)
    wd = [torch.from_numpy(inp[k]).to(DEV, dt) if i < nt else None for i, k in enumerate(("wa", "wb", "wc"))]
    bd = [qlh.vec_to_dev(inp[k]) if i < nt else None for i, k in enumerate(("ba", "bb", "bc"))]
    yd = torch.empty((B, O), device=DEV, dtype=dt)
    tad = torch.empty_like(yd) if neuron != T2 else None
    tbd = torch.empty_like(yd) if nt >= 2 else None
    ql.qlayer_linear_fwd(d, x, *wd, *bd, yd, tad, tbd)
    gy = torch.from_numpy(inp["gy"]).to(DEV, dt)
    dx = torch.empty_like(x)
    dw = [torch.empty((O, I), device=DEV, dtype=torch.float32) if i < nt else None for i in range(3)]
    db = [torch.empty(O, device=DEV, dtype=torch.float32) if i < nt else None for i in range(3)]
    ql.qlayer_linear_bwd(d, x, gy, tad, tbd, *wd, dx, *dw, *db)
    torch.cuda.synchronize()
    got = {"y": yd, "dx": dx}
    for i, (kw, kb) in enumerate((("dwa", "dba"), ("dwb", "dbb"), ("dwc", "dbc"))[:nt]):
        got[kw], got[kb] = dw[i], db[i]
    for k, v in got.items():
        e = qlh.relerr(v.double().cpu().numpy(), ref[k])
        assert e <= qlh.tol(bf16, k != "y"), f"{k}: normwise relative error {e:.3e}"


def test_recompute_mode_regenerates_the_saved_maps_bitwise():
    """Hybrid back-propagation with the other types: the forward without Y
    writes the same T_a (and T_b) as the saving forward."""
    shape = (2, 32, 8, 8, 32, 3, 1, 1)
    N, C, H, W, O, K, s, p = shape
    for neuron in (T4, T4I, T3, T24):
        nt = TERMS[neuron]
        inp = synth.random_conv_case([502, neuron], N, C, H, W, O, K, K, s, p, bf16=True)
        d = ql.conv_desc(N, C, H, W, O, K, K, s, p, ql.QL_BF16, neuron)
        x = qlh.nchw_to_dev(inp["x"], True)
        w = [qlh.oihw_to_dev(inp[k], True) if i < nt else None for i, k in enumerate(("wa", "wb", "wc"))]
        b = [qlh.vec_to_dev(inp[k]) if i < nt else None for i, k in enumerate(("ba", "bb", "bc"))]
        y = torch.empty((N, H, W, O), device=DEV, dtype=torch.bfloat16)
        maps = [torch.empty_like(y) for _ in range(4)]
        tb0, tb1 = (maps[1], maps[3]) if nt >= 2 else (None, None)
        ql.qlayer_conv2d_fwd(d, x, *w, *b, y, maps[0], tb0)
        ql.qlayer_conv2d_fwd(d, x, *w, *b, None, maps[2], tb1)
        torch.cuda.synchronize()
        assert torch.equal(maps[0], maps[2]), NAMES[neuron]
        if nt >= 2:
            assert torch.equal(maps[1], maps[3]), NAMES[neuron]
