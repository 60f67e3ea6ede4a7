"""The forward for layers with few input channels (the reduction (r, q, c)
and the bias columns fit one 32-column MFMA reduction; e.g. an RGB stem),
against the fp64 oracle with the path on and forced off, in fp32 and bf16:
padding, stride 2, 5 x 5 and 1 x 1 filters, ragged pixel groups, 32 and 64
output channels, the largest reductions of each precision, no biases, the
fused epilogue and the recompute mode of the hybrid back-propagation
(section 4.3: T_a, T_b regenerated bitwise)."""
import numpy as np
import pytest
import torch

import oracle
import synth

pytestmark = pytest.mark.gpu

import qlh  # noqa: E402
import paper_2204_01701_amd as ql  # noqa: E402

DEV = qlh.DEV
KEYS_FWD = ("y", "ta", "tb")
KEYS_GRAD = ("dx", "dwa", "dwb", "dwc", "dba", "dbb", "dbc")

# (N, C, H, W, O, KH, KW, stride, pad)
SHAPES = [
    (4, 3, 32, 32, 64, 3, 3, 1, 1),     # the RGB stem of the CIFAR networks
    (3, 3, 17, 13, 32, 3, 3, 2, 1),     # stride 2, 32 output channels
    (2, 1, 9, 9, 64, 5, 5, 1, 2),       # one channel, 5 x 5 filter (J = 25)
    (5, 2, 7, 7, 64, 3, 3, 1, 0),       # no padding
    (1, 3, 5, 37, 32, 3, 3, 1, 1),      # 185 pixels: a ragged last group
    (2, 29, 6, 6, 64, 1, 1, 1, 0),      # J = 29: the largest bf16 reduction (3 bias columns)
    (2, 30, 5, 5, 32, 1, 1, 1, 0),      # J = 30: small-C path in fp32 only
]


def _oracle_all(inp, s, p):
    y, ta, tb = oracle.conv2d_fwd(inp["x"], inp["wa"], inp["wb"], inp["wc"], inp["ba"], inp["bb"], inp["bc"], s, p)
    d = oracle.conv2d_bwd(inp["x"], inp["wa"], inp["wb"], inp["wc"], inp["ba"], inp["bb"], inp["bc"], inp["gy"], s, p)
    d.update({"y": y, "ta": ta, "tb": tb})
    return d


@pytest.mark.parametrize("path", ["1", "0"], ids=["smallc", "general"])
@pytest.mark.parametrize("bf16", [False, True], ids=["fp32", "bf16"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_smallc_forward_matches_oracle(shape, bf16, path, monkeypatch):
    N, C, H, W, O, KH, KW, s, p = shape
    print(f"small-C forward path={path} shape={shape} bf16={bf16}", flush=True)
    monkeypatch.setenv("QLAYER_FWD_SMALLC", path)
    inp = synth.random_conv_case([800] + list(shape), N, C, H, W, O, KH, KW, s, p, bf16=bf16)
    got = qlh.conv_to_np(qlh.run_conv(inp, s, p, bf16, recompute=True))
    ref = _oracle_all(inp, s, p)
    for k in KEYS_FWD + KEYS_GRAD:
        e = qlh.relerr(got[k], ref[k])
        assert e <= qlh.tol(bf16, k in KEYS_GRAD), f"{k}: normwise relative error {e:.3e}"
    # recompute mode: the forward without Y regenerates the saved maps bit for bit
    assert np.array_equal(got["ta_re"], got["ta"]) and np.array_equal(got["tb_re"], got["tb"])


@pytest.mark.parametrize("bf16", [False, True], ids=["fp32", "bf16"])
def test_smallc_forward_without_bias(bf16):
    shape = (3, 3, 12, 12, 64, 3, 3, 1, 1)
    N, C, H, W, O, KH, KW, s, p = shape
    print(f"small-C forward without bias shape={shape} bf16={bf16}", flush=True)
    inp = synth.random_conv_case([801], N, C, H, W, O, KH, KW, s, p, bf16=bf16)
    got = qlh.conv_to_np(qlh.run_conv(inp, s, p, bf16, with_bias=False))
    zero = np.zeros_like(inp["ba"])
    y, ta, tb = oracle.conv2d_fwd(inp["x"], inp["wa"], inp["wb"], inp["wc"], zero, zero, zero, s, p)
    for k, ref in (("y", y), ("ta", ta), ("tb", tb)):
        e = qlh.relerr(got[k], ref)
        assert e <= qlh.tol(bf16, False), f"{k}: normwise relative error {e:.3e}"


def test_smallc_bias_is_exact():
    """bf16: each fp32 bias enters as three bf16 parts whose sum is exact; with
    zero weights every output is its bias to fp32 rounding, whatever the bias's
    low significand bits (here biases that bf16 cannot hold)."""
    N, C, H, W, O = 2, 3, 6, 6, 64
    d = ql.conv_desc(N, C, H, W, O, 3, 3, 1, 1, ql.QL_BF16)
    x = torch.randn(N, H, W, C, device=DEV).to(torch.bfloat16)
    w = [torch.zeros(O, 3, 3, C, device=DEV, dtype=torch.bfloat16) for _ in range(3)]
    b = [(torch.arange(O, device=DEV, dtype=torch.float32) + 1.0) / 3.0 + k * 1e-3 for k in range(3)]
    y = torch.empty(N, H, W, O, device=DEV, dtype=torch.bfloat16)
    ta, tb = torch.empty_like(y), torch.empty_like(y)
    ql.qlayer_conv2d_fwd(d, x, *w, *b, y, ta, tb)
    torch.cuda.synchronize()
    ref_y = (b[0].double() * b[1].double() + b[2].double())
    for got, ref in ((ta, b[0].double()), (tb, b[1].double()), (y, ref_y)):
        expect = ref.float().to(torch.bfloat16).double()   # one rounding to bf16 of the exact value
        assert torch.equal(got.double()[0, 3, 3], expect), (got.double()[0, 3, 3] - expect).abs().max()


def test_smallc_fused_epilogue():
    """Scale, shift, ReLU and the channel sums on the small-C forward (bf16)."""
    shape = (8, 3, 16, 16, 64, 3, 3, 1, 1)
    N, C, H, W, O, KH, KW, s, p = shape
    print(f"small-C fused epilogue shape {shape}", flush=True)
    inp = synth.random_conv_case([802], N, C, H, W, O, KH, KW, s, p, bf16=True)
    d = ql.conv_desc(N, C, H, W, O, KH, KW, s, p, ql.QL_BF16)
    x = qlh.nchw_to_dev(inp["x"], True)
    w = [qlh.oihw_to_dev(inp[k], True) for k in ("wa", "wb", "wc")]
    b = [qlh.vec_to_dev(inp[k]) for k in ("ba", "bb", "bc")]
    y = torch.empty((N, d.ho, d.wo, O), device=DEV, dtype=torch.bfloat16)
    ta, tb = torch.empty_like(y), torch.empty_like(y)
    sc = torch.linspace(0.5, 1.5, O, device=DEV)
    sh = torch.linspace(-0.2, 0.2, O, device=DEV)
    ssum, ssq = torch.empty(O, device=DEV), torch.empty(O, device=DEV)
    ql.qlayer_conv2d_fwd_ex(d, x, *w, *b, y, ta, tb, epi=ql.epilogue(sc, sh, True, ssum, ssq))
    torch.cuda.synchronize()
    yr, _, _ = oracle.conv2d_fwd(inp["x"], inp["wa"], inp["wb"], inp["wc"], inp["ba"], inp["bb"], inp["bc"], s, p)
    ref_y, ref_sum, _ = oracle.epilogue(yr, sc.double().cpu().numpy(), sh.double().cpu().numpy(), True)
    got_y = qlh.nhwc_to_np(y)
    assert qlh.relerr(got_y, ref_y) <= qlh.tol(True, False)
    yd = got_y.astype("float64")
    assert qlh.relerr(ssum.double().cpu().numpy(), yd.sum(axis=(0, 2, 3))) <= 1e-5
    assert qlh.relerr(ssq.double().cpu().numpy(), (yd * yd).sum(axis=(0, 2, 3))) <= 1e-5
    assert qlh.relerr(ssum.double().cpu().numpy(), ref_sum) <= qlh.tol(True, False)


# Input gradient of the few-channel layers, stride 1: the per-pixel partial
# sums and their gather fused in one kernel over bands of input rows (the
# partial sums of a band's halo rows recomputed), at several band heights.
FUSED_SHAPES = [
    (4, 3, 32, 32, 64, 3, 3, 1, 1),     # the RGB stem
    (2, 1, 9, 9, 64, 5, 5, 1, 2),       # 5 x 5: a halo of 4 rows
    (3, 2, 11, 7, 32, 3, 3, 1, 0),      # no padding: the output map is smaller
    (2, 3, 5, 6, 16, 3, 3, 1, 1),       # 16 output channels, bands past the last row
]


@pytest.mark.parametrize("rb", ["1", "3", "8"])
@pytest.mark.parametrize("bf16", [False, True], ids=["fp32", "bf16"])
@pytest.mark.parametrize("shape", FUSED_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_fused_input_gradient_matches_oracle(shape, bf16, rb, monkeypatch):
    N, C, H, W, O, KH, KW, s, p = shape
    print(f"fused small-C input gradient rows={rb} shape={shape} bf16={bf16}", flush=True)
    monkeypatch.setenv("QLAYER_BWD_DATA_FUSED_RB", rb)
    inp = synth.random_conv_case([803] + list(shape), N, C, H, W, O, KH, KW, s, p, bf16=bf16)
    got = qlh.conv_to_np(qlh.run_conv(inp, s, p, bf16))
    ref = _oracle_all(inp, s, p)
    e = qlh.relerr(got["dx"], ref["dx"])
    assert e <= qlh.tol(bf16, True), f"dx: normwise relative error {e:.3e}"


@pytest.mark.parametrize("bf16", [False, True], ids=["fp32", "bf16"])
def test_smallc_dense_layer(bf16):
    """A fully-connected layer with few inputs (27 -> 64) takes the same kernels (H = W = 1)."""
    print(f"small-C dense layer bf16={bf16}", flush=True)
    inp = synth.random_dense_case([806], 300, 27, 64, bf16=bf16)
    got = {k: v.double().cpu().numpy() for k, v in qlh.run_linear(inp, bf16).items()}
    y, ta, tb = oracle.linear_fwd(inp["x"], inp["wa"], inp["wb"], inp["wc"], inp["ba"], inp["bb"], inp["bc"])
    ref = oracle.linear_bwd(inp["x"], inp["wa"], inp["wb"], inp["wc"], inp["ba"], inp["bb"], inp["bc"], inp["gy"])
    ref.update({"y": y, "ta": ta, "tb": tb})
    for k in KEYS_FWD + KEYS_GRAD:
        e = qlh.relerr(got[k], ref[k])
        assert e <= qlh.tol(bf16, k in KEYS_GRAD), f"{k}: normwise relative error {e:.3e}"
