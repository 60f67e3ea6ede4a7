"""The narrow-layer kernels (forward, input gradient, weight gradient: at
most 16 output or input channels and a short reduction) against the fp64
oracle, with the paths on (the default for these shapes) and forced off
(the tiled kernels), fp32 and bf16: 16 channels at stride 1 and 2, 8
channels, the zero-padded 3-channel stem, a ragged last pixel block, a 1x1
filter, 16 -> 8 channels, O < 16, and the weight gradient of wider layers
(up to 64 channels) in 16-channel slices.  Normwise limits as in
test_gpu_parity."""
import pytest

import oracle
import synth

pytestmark = pytest.mark.gpu

import qlh  # noqa: E402

# (N, C, H, W, O, KH, KW, stride, pad)
SHAPES = [
    (4, 16, 12, 12, 16, 3, 3, 1, 1),    # a 16-channel CIFAR ResNet stage
    (3, 16, 11, 9, 16, 3, 3, 2, 1),     # stride 2, ragged last pixel block
    (2, 8, 10, 10, 8, 3, 3, 1, 1),      # 8 channels
    (5, 3, 9, 9, 16, 3, 3, 1, 1),       # the 3-channel stem (X zero-padded)
    (2, 16, 7, 7, 16, 1, 1, 1, 0),      # 1x1 filter
    (2, 16, 9, 9, 8, 3, 3, 1, 1),       # 16 -> 8 channels
    (1, 12, 6, 5, 12, 3, 3, 1, 1),      # 12 channels (fp32: narrow; bf16: off the vector width)
    (4, 3, 10, 10, 64, 3, 3, 1, 1),     # a 3 -> 64-channel stem: weight gradient in four 16-channel slices
    (2, 16, 9, 9, 32, 3, 3, 2, 1),      # 16 -> 32 at stride 2: two slices
    (3, 8, 7, 7, 48, 3, 3, 1, 1),       # three slices
]

KEYS_FWD = ("y", "ta", "tb")
KEYS_GRAD = ("dx", "dwa", "dwb", "dwc", "dba", "dbb", "dbc")
OFF = ("QLAYER_FWD_NARROW", "QLAYER_BWD_DATA_NARROW", "QLAYER_BWD_WEIGHT_NARROW")


@pytest.mark.parametrize("narrow", [True, False], ids=["narrow", "tiled"])
@pytest.mark.parametrize("bf16", [False, True], ids=["fp32", "bf16"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_narrow_paths_match_oracle(shape, bf16, narrow, monkeypatch):
    N, C, H, W, O, KH, KW, s, p = shape
    print(f"narrow={narrow} shape={shape} bf16={bf16}", flush=True)
    if not narrow:
        for k in OFF:
            monkeypatch.setenv(k, "0")
    else:
        monkeypatch.setenv("QLAYER_BWD_WEIGHT_NARROW_MAXO", "64")  # (16-channel slices in bf16 too)
    inp = synth.random_conv_case([800] + list(shape), N, C, H, W, O, KH, KW, s, p, bf16=bf16)
    got = qlh.conv_to_np(qlh.run_conv(inp, s, p, bf16))
    y, ta, tb = oracle.conv2d_fwd(inp["x"], inp["wa"], inp["wb"], inp["wc"], inp["ba"], inp["bb"], inp["bc"], s, p)
    ref = oracle.conv2d_bwd(inp["x"], inp["wa"], inp["wb"], inp["wc"], inp["ba"], inp["bb"], inp["bc"], inp["gy"], s, p)
    ref.update({"y": y, "ta": ta, "tb": tb})
    for k in KEYS_FWD + KEYS_GRAD:
        e = qlh.relerr(got[k], ref[k])
        assert e <= qlh.tol(bf16, k in KEYS_GRAD), f"{k}: normwise relative error {e:.3e}"
