"""GPU parity: the HIP path against the fp64 oracle, element by element, on
small and ragged shapes that span several tiles, split-K and the non-vector
load paths.  Normwise relative error limits: fp32 forward 1e-5, gradients
1e-4; bf16 (fp32 accumulation) 2e-2.
"""
import numpy as np
import pytest

import oracle
import synth

pytestmark = pytest.mark.gpu

import qlh  # noqa: E402

# (N, C, H, W, O, KH, KW, stride, pad)
CONV_SHAPES = [
    (2, 16, 8, 8, 16, 3, 3, 1, 1),      # the small fp32 workload's geometry
    (2, 3, 9, 7, 8, 3, 3, 1, 1),        # 3 input channels (element-wise loads)
    (1, 5, 6, 6, 7, 3, 3, 2, 1),        # odd channels, stride 2
    (2, 16, 7, 9, 24, 1, 1, 1, 0),      # 1x1 kernel
    (3, 32, 5, 5, 40, 3, 3, 2, 0),      # stride 2, no padding
    (2, 64, 4, 4, 64, 3, 3, 1, 1),      # few pixels, long K: split-K forward
    (4, 16, 16, 16, 32, 3, 3, 1, 1),    # many pixels: split-K weight gradient
    (1, 8, 1, 1, 8, 3, 3, 1, 1),        # 1x1 map, 3x3 kernel, pad 1
    (2, 24, 10, 10, 136, 3, 3, 1, 1),   # ragged output-channel tiles
    (1, 136, 6, 6, 16, 3, 3, 1, 1),     # ragged input-channel tiles
    (2, 8, 33, 17, 8, 3, 3, 1, 1),      # ragged pixel tiles
    (2, 16, 8, 8, 32, 3, 3, 2, 1),      # residual-stage transition
    (1, 8, 7, 9, 16, 3, 1, 1, 1),       # non-square kernel
    (2, 12, 6, 6, 20, 2, 2, 2, 0),      # even kernel, stride 2
    (4, 3, 32, 32, 64, 3, 3, 1, 1),     # 3-channel image stem (channel padding, small-C input gradient)
    (3, 5, 11, 9, 24, 3, 3, 2, 1),      # 5 channels, stride 2
    (2, 4, 10, 10, 32, 3, 3, 2, 1),     # 4 channels, stride 2: two column blocks of (r, q, c)
    (3, 1, 7, 9, 16, 3, 3, 1, 0),       # 1 channel, no padding
    (2, 2, 6, 7, 16, 5, 5, 1, 2),       # 2 channels, 5x5 kernel
]

KEYS_FWD = ("y", "ta", "tb")
KEYS_GRAD = ("dx", "dwa", "dwb", "dwc", "dba", "dbb", "dbc")


def _oracle_all(inp, s, p):
    y, ta, tb = oracle.conv2d_fwd(inp["x"], inp["wa"], inp["wb"], inp["wc"], inp["ba"], inp["bb"], inp["bc"], s, p)
    d = oracle.conv2d_bwd(inp["x"], inp["wa"], inp["wb"], inp["wc"], inp["ba"], inp["bb"], inp["bc"], inp["gy"], s, p)
    d.update({"y": y, "ta": ta, "tb": tb})
    return d


@pytest.mark.parametrize("bf16", [False, True], ids=["fp32", "bf16"])
@pytest.mark.parametrize("shape", CONV_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_conv_matches_oracle(shape, bf16):
    N, C, H, W, O, KH, KW, s, p = shape
    print(f"conv parity shape={shape} bf16={bf16}", flush=True)
    inp = synth.random_conv_case([100] + list(shape), N, C, H, W, O, KH, KW, s, p, bf16=bf16)
    got = qlh.conv_to_np(qlh.run_conv(inp, s, p, bf16))
    ref = _oracle_all(inp, s, p)
    for k in KEYS_FWD + KEYS_GRAD:
        e = qlh.relerr(got[k], ref[k])
        assert e <= qlh.tol(bf16, k in KEYS_GRAD), f"{k}: normwise relative error {e:.3e}"


DENSE_SHAPES = [(64, 32, 48), (7, 19, 13), (300, 136, 200), (128, 256, 64), (1, 8, 8)]


@pytest.mark.parametrize("bf16", [False, True], ids=["fp32", "bf16"])
@pytest.mark.parametrize("shape", DENSE_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_linear_matches_oracle(shape, bf16):
    B, I, O = shape
    print(f"linear parity shape={shape} bf16={bf16}", flush=True)
    inp = synth.random_dense_case([200] + list(shape), B, I, O, bf16=bf16)
    got = {k: v.double().cpu().numpy() for k, v in qlh.run_linear(inp, bf16).items()}
    y, ta, tb = oracle.linear_fwd(inp["x"], inp["wa"], inp["wb"], inp["wc"], inp["ba"], inp["bb"], inp["bc"])
    ref = oracle.linear_bwd(inp["x"], inp["wa"], inp["wb"], inp["wc"], inp["ba"], inp["bb"], inp["bc"], inp["gy"])
    ref.update({"y": y, "ta": ta, "tb": tb})
    for k in KEYS_FWD + KEYS_GRAD:
        e = qlh.relerr(got[k], ref[k])
        assert e <= qlh.tol(bf16, k in KEYS_GRAD), f"{k}: normwise relative error {e:.3e}"


@pytest.mark.parametrize("bf16", [False, True], ids=["fp32", "bf16"])
def test_no_bias_and_zero_product_weight(bf16):
    """Biases omitted (NULL) and W_a = 0: the layer is an ordinary convolution."""
    shape = (2, 16, 6, 6, 16, 3, 3, 1, 1)
    N, C, H, W, O, KH, KW, s, p = shape
    inp = synth.random_conv_case([300], N, C, H, W, O, KH, KW, s, p, bf16=bf16)
    inp["wa"][:] = 0
    got = qlh.conv_to_np(qlh.run_conv(inp, s, p, bf16, with_bias=False))
    zero = np.zeros(O, np.float32)
    y, ta, tb = oracle.conv2d_fwd(inp["x"], inp["wa"], inp["wb"], inp["wc"], zero, zero, zero, s, p)
    assert np.all(got["ta"] == 0)
    assert qlh.relerr(got["y"], y) <= qlh.tol(bf16, False)
    d = oracle.conv2d_bwd(inp["x"], inp["wa"], inp["wb"], inp["wc"], zero, zero, zero, inp["gy"], s, p)
    for k in KEYS_GRAD:
        if k == "dwb" or k == "dbb":
            assert np.all(got[k] == 0), k  # G_b = G o T_a = 0
            continue
        assert qlh.relerr(got[k], d[k]) <= qlh.tol(bf16, True), k


# Every tile configuration of the three convolution passes, forced through the
# planner's override, on shapes with ragged tiles (the default planner picks
# only some of them for the small shapes above).
TILE_CONFIGS = ([("QLAYER_FWD_CFG", c) for c in range(7)] +
                [("QLAYER_BWD_DATA_CFG", c) for c in range(6)] +
                [("QLAYER_BWD_WEIGHT_CFG", c) for c in range(6)] +
                # channel-aligned forward K steps in image-major order (by default fp32 and position-major only)
                [("QLAYER_FWD_CA", 1)])
TILE_SHAPES = [(2, 24, 10, 9, 48, 3, 3, 1, 1), (1, 264, 5, 7, 144, 3, 3, 1, 1), (2, 32, 9, 9, 16, 3, 3, 2, 1)]


@pytest.mark.parametrize("bf16", [False, True], ids=["fp32", "bf16"])
@pytest.mark.parametrize("shape", TILE_SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("env,cfg", TILE_CONFIGS, ids=lambda v: str(v))
def test_conv_tile_configs(env, cfg, shape, bf16, monkeypatch):
    N, C, H, W, O, KH, KW, s, p = shape
    print(f"tile config {env}={cfg} shape={shape} bf16={bf16}", flush=True)
    monkeypatch.setenv(env, str(cfg))
    inp = synth.random_conv_case([300] + list(shape), N, C, H, W, O, KH, KW, s, p, bf16=bf16)
    got = qlh.conv_to_np(qlh.run_conv(inp, s, p, bf16))
    ref = _oracle_all(inp, s, p)
    for k in KEYS_FWD + KEYS_GRAD:
        e = qlh.relerr(got[k], ref[k])
        assert e <= qlh.tol(bf16, k in KEYS_GRAD), f"{k}: normwise relative error {e:.3e}"


# Block orders of the input gradient's split-K grid (split-major, tile-major,
# row-major), forced through the planner's override on layers whose input
# gradient splits K: the same split partials in every order, so the same bits,
# and within the oracle's limit.
ORDER_SHAPES = [(16, 256, 4, 4, 256, 3, 3, 1, 1), (8, 128, 8, 8, 256, 3, 3, 1, 1), (3, 72, 5, 6, 96, 3, 3, 1, 1),
                (32, 512, 2, 2, 512, 3, 3, 1, 1)]


@pytest.mark.parametrize("bf16", [False, True], ids=["fp32", "bf16"])
@pytest.mark.parametrize("shape", ORDER_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_bwd_data_block_orders(shape, bf16, monkeypatch):
    N, C, H, W, O, KH, KW, s, p = shape
    print(f"bwd_data block orders shape={shape} bf16={bf16}", flush=True)
    inp = synth.random_conv_case([301] + list(shape), N, C, H, W, O, KH, KW, s, p, bf16=bf16)
    ref = _oracle_all(inp, s, p)
    dx = []
    for order in (0, 1, 2):
        monkeypatch.setenv("QLAYER_BWD_DATA_ORDER", str(order))
        got = qlh.conv_to_np(qlh.run_conv(inp, s, p, bf16))
        e = qlh.relerr(got["dx"], ref["dx"])
        assert e <= qlh.tol(bf16, True), f"order {order}: normwise relative error {e:.3e}"
        dx.append(got["dx"])
    for order in (1, 2):
        assert np.array_equal(dx[0], dx[order]), f"order {order} differs from order 0"
