"""The small-output forward (tiles of 3 x 16 RB rows by 16 CB pixels whose
four waves split K, the default where the tiled forward would split K over
workgroups: the 4 x 4 and 2 x 2 maps of a CIFAR VGG-16) against the fp64
oracle, fp32 and bf16: forced on for every tile shape, in both pixel orders
(position-major: taps in the padding skipped per tile), ragged rows and
pixels, stride 2, a 1 x 1 and a 5 x 5 filter, and forced off (the tiled
kernels).  Normwise limits as in test_gpu_parity, plus the elementwise bound
of the full-size tests on Y, T_a and T_b."""
import numpy as np
import pytest

import oracle
import synth

pytestmark = pytest.mark.gpu

import qlh  # noqa: E402

# (N, C, H, W, O, KH, KW, stride, pad)
SHAPES = [
    (16, 64, 2, 2, 64, 3, 3, 1, 1),     # a 2 x 2 map (position-major by default)
    (8, 64, 4, 4, 72, 3, 3, 1, 1),      # a 4 x 4 map, ragged row tile
    (3, 64, 5, 3, 20, 3, 3, 2, 1),      # stride 2, ragged pixels and rows
    (2, 32, 4, 4, 36, 1, 1, 1, 0),      # 1 x 1 filter
    (2, 64, 4, 4, 64, 5, 5, 1, 2),      # 5 x 5 filter
    (5, 128, 3, 3, 32, 3, 3, 1, 1),     # odd chunk counts per wave
]

# (tile index: 0 = 2 x 4 blocks, 1 = 1 x 4, 2 = 2 x 2; position-major order)
MODES = [("t0", "0", None), ("t1", "1", None), ("t2", "2", None), ("t0-pm", "0", "1"), ("t1-im", "1", "0")]

KEYS_FWD = ("y", "ta", "tb")
KEYS_GRAD = ("dx", "dwa", "dwb", "dwc", "dba", "dbb", "dbc")


def _check_fwd(inp, got, s, p, bf16):
    f64 = {k: np.ascontiguousarray(v, dtype=np.float64) for k, v in inp.items()}
    keys = ("x", "wa", "wb", "wc", "ba", "bb", "bc")
    ref = dict(zip(KEYS_FWD, oracle.conv2d_fwd(*[f64[k] for k in keys], s, p)))
    mag = dict(zip(KEYS_FWD, oracle.conv2d_fwd(*[np.abs(f64[k]) for k in keys], s, p)))
    C, KH, KW = inp["wa"].shape[1:]
    for k in KEYS_FWD:
        e = qlh.relerr(got[k], ref[k])
        assert e <= qlh.tol(bf16, False), f"{k}: normwise relative error {e:.3e}"
        qlh.check_elementwise(k, k, got[k], ref[k], mag[k], bf16, C * KH * KW + 1)
    return f64


@pytest.mark.parametrize("mode", MODES, ids=[m[0] for m in MODES])
@pytest.mark.parametrize("bf16", [False, True], ids=["fp32", "bf16"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_ksplit_forward_matches_oracle(shape, bf16, mode, monkeypatch):
    N, C, H, W, O, KH, KW, s, p = shape
    name, tile, pm = mode
    print(f"ksplit {name} shape={shape} bf16={bf16}", flush=True)
    monkeypatch.setenv("QLAYER_FWD_KSPLIT", "1")
    monkeypatch.setenv("QLAYER_FWD_KSPLIT_TILE", tile)
    if pm is not None:
        monkeypatch.setenv("QLAYER_FWD_POSMAJ", pm)
    inp = synth.random_conv_case([810] + list(shape), N, C, H, W, O, KH, KW, s, p, bf16=bf16)
    got = qlh.conv_to_np(qlh.run_conv(inp, s, p, bf16))
    _check_fwd(inp, got, s, p, bf16)


@pytest.mark.parametrize("ksplit", [True, False], ids=["ksplit", "tiled"])
@pytest.mark.parametrize("bf16", [False, True], ids=["fp32", "bf16"])
def test_ksplit_and_tiled_whole_layer(bf16, ksplit, monkeypatch):
    """A whole layer (forward, input and weight gradients) with the small-output
    forward forced on and off: a 2 x 2 map of 128 images, 128 -> 64 channels."""
    N, C, H, W, O, K, s, p = 128, 128, 2, 2, 64, 3, 1, 1
    print(f"ksplit={ksplit} whole layer bf16={bf16}", flush=True)
    monkeypatch.setenv("QLAYER_FWD_KSPLIT", "1" if ksplit else "0")
    inp = synth.random_conv_case([811, N, C, H, O], N, C, H, W, O, K, K, s, p, bf16=bf16)
    got = qlh.conv_to_np(qlh.run_conv(inp, s, p, bf16))
    f64 = _check_fwd(inp, got, s, p, bf16)
    keys = ("x", "wa", "wb", "wc", "ba", "bb", "bc")
    ref = oracle.conv2d_bwd(*[f64[k] for k in keys], f64["gy"], s, p)
    for k in KEYS_GRAD:
        e = qlh.relerr(got[k], ref[k])
        assert e <= qlh.tol(bf16, True), f"{k}: normwise relative error {e:.3e}"


def test_ksplit_is_bitwise_repeatable(monkeypatch):
    """The waves' partial sums are added in a fixed order: two calls agree bit for bit."""
    monkeypatch.setenv("QLAYER_FWD_KSPLIT", "1")
    N, C, H, W, O = 32, 256, 4, 4, 64
    inp = synth.random_conv_case([812], N, C, H, W, O, 3, 3, 1, 1, bf16=True)
    a = qlh.conv_to_np(qlh.run_conv(inp, 1, 1, True))
    b = qlh.conv_to_np(qlh.run_conv(inp, 1, 1, True))
    for k in KEYS_FWD:
        assert np.array_equal(a[k], b[k]), k
