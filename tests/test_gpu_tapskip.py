"""The forward's position-major pixel order with padding-only taps skipped
(small maps, where a pixel tile spans few output positions): the HIP path,
forward and backward, against the fp64 oracle with the order forced on and
off, on shapes where tiles hold one position, several positions, ragged
tails, stride 2, 5 x 5 filters and positions with no tap in bounds at all
(their outputs are the bias terms alone; eq:2ndneuron3 with every product
term zero).  Each shape runs in the tiled kernel and in the small-output
kernel whose waves split K (qconv_fwd_ksplit.h); in bf16 at stride 1 the
input gradient's channel-aligned kernel takes the same order (its taps whose
output pixel lies outside the map skipped)."""
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
    (128, 64, 2, 2, 64, 3, 3, 1, 1),    # one output position per pixel tile
    (40, 32, 4, 4, 48, 3, 3, 1, 1),     # tiles spanning several positions, ragged last tile
    (64, 64, 3, 5, 32, 3, 3, 2, 1),     # stride 2, non-square map
    (33, 32, 4, 4, 32, 5, 5, 1, 2),     # 5 x 5 filter, pad 2: most taps in the padding
    (128, 32, 1, 1, 32, 3, 3, 1, 3),    # pad 3: positions with no tap in bounds
    (7, 96, 8, 8, 40, 3, 3, 1, 1),      # 8 x 8 map, few images (position-major only when forced)
    (256, 64, 2, 2, 96, 3, 3, 1, 1),    # two tiles per position
]


def _oracle_all(inp, s, p):
    y, ta, tb = oracle.conv2d_fwd(inp["x"], inp["wa"], inp["wb"], inp["wc"], inp["ba"], inp["bb"], inp["bc"], s, p)
    d = oracle.conv2d_bwd(inp["x"], inp["wa"], inp["wb"], inp["wc"], inp["ba"], inp["bb"], inp["bc"], inp["gy"], s, p)
    d.update({"y": y, "ta": ta, "tb": tb})
    return d


@pytest.mark.parametrize("kernel", ["0", "1"], ids=["tiled", "ksplit"])
@pytest.mark.parametrize("order", ["1", "0"], ids=["posmajor", "imagemajor"])
@pytest.mark.parametrize("bf16", [False, True], ids=["fp32", "bf16"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_tap_skipping_matches_oracle(shape, bf16, order, kernel, monkeypatch):
    N, C, H, W, O, KH, KW, s, p = shape
    print(f"tap skipping order={order} ksplit={kernel} shape={shape} bf16={bf16}", flush=True)
    monkeypatch.setenv("QLAYER_FWD_POSMAJ", order)
    monkeypatch.setenv("QLAYER_BWD_DATA_POSMAJ", order)  # (bf16, stride 1: the input gradient's order too)
    monkeypatch.setenv("QLAYER_FWD_KSPLIT", kernel)  # the tiled kernel, or the small-output one
    if order == "0":  # the channel-aligned K steps without the position-major order
        monkeypatch.setenv("QLAYER_FWD_CA", "1")
    inp = synth.random_conv_case([700] + list(shape), N, C, H, W, O, KH, KW, s, p, bf16=bf16)
    got = qlh.conv_to_np(qlh.run_conv(inp, s, p, bf16))
    ref = _oracle_all(inp, s, p)
    for k in KEYS_FWD + KEYS_GRAD:
        e = qlh.relerr(got[k], ref[k])
        assert e <= qlh.tol(bf16, k in KEYS_GRAD), f"{k}: normwise relative error {e:.3e}"


T4, T4I, T3, T2 = ql.QL_NEURON_T4, ql.QL_NEURON_T4_IDENTITY, ql.QL_NEURON_T3, ql.QL_NEURON_T2
NAMES = {T4: "T4", T4I: "T4I", T3: "T3", T2: "T2"}


@pytest.mark.parametrize("neuron", [T4, T4I, T3, T2], ids=[NAMES[n] for n in (T4, T4I, T3, T2)])
def test_tap_skipping_neuron_types(neuron, monkeypatch):
    """The other neuron types' kernels (bf16) in position-major order; T4 + identity
    adds X at the output pixel, read through the same row mapping."""
    from test_gpu_neurons import _run_conv_neuron, TERMS
    shape = (64, 64, 4, 4, 64, 3, 1, 1)
    N, C, H, W, O, K, s, p = shape
    print(f"tap skipping neuron {NAMES[neuron]} shape {shape}", flush=True)
    monkeypatch.setenv("QLAYER_FWD_POSMAJ", "1")
    inp = synth.random_conv_case([701, neuron] + list(shape), N, C, H, W, O, K, K, s, p, bf16=True)
    nt = TERMS[neuron]
    w = [inp["wa"], inp["wb"] if nt >= 2 else None, None]
    b = [inp["ba"], inp["bb"] if nt >= 2 else None, None]
    y, ta, tb = oracle.conv2d_fwd_neuron(neuron, inp["x"], *w, *b, stride=s, pad=p)
    ref = oracle.conv2d_bwd_neuron(neuron, inp["x"], *w, *b, inp["gy"], stride=s, pad=p)
    ref["y"] = y
    if neuron != T2:
        ref["ta"] = ta
    if nt >= 2:
        ref["tb"] = tb
    got = _run_conv_neuron(neuron, inp, s, p, True)
    assert sorted(got) == sorted(ref)
    for k in ref:
        e = qlh.relerr(got[k], ref[k])
        assert e <= qlh.tol(True, k not in ("y", "ta", "tb")), f"{k}: normwise relative error {e:.3e}"


def test_tap_skipping_epilogue_sums(monkeypatch):
    """The fused forward epilogue (scale, shift, ReLU; channel sums of the
    result) in position-major order: the sums cover every NHWC row once."""
    shape = (128, 64, 4, 4, 64, 3, 3, 1, 1)
    N, C, H, W, O, KH, KW, s, p = shape
    print(f"tap skipping epilogue shape {shape}", flush=True)
    monkeypatch.setenv("QLAYER_FWD_POSMAJ", "1")
    inp = synth.random_conv_case([702], N, C, H, W, O, KH, KW, s, p, bf16=True)
    d = ql.conv_desc(N, C, H, W, O, KH, KW, s, p, ql.QL_BF16)
    x = qlh.nchw_to_dev(inp["x"], True)
    w = [qlh.oihw_to_dev(inp[k], True) for k in ("wa", "wb", "wc")]
    b = [qlh.vec_to_dev(inp[k]) for k in ("ba", "bb", "bc")]
    y = torch.empty((N, d.ho, d.wo, O), device=DEV, dtype=torch.bfloat16)
    ta, tb = torch.empty_like(y), torch.empty_like(y)
    sc = torch.linspace(0.5, 1.5, O, device=DEV)
    sh = torch.linspace(-0.2, 0.2, O, device=DEV)
    ssum, ssq = torch.empty(O, device=DEV), torch.empty(O, device=DEV)
    e = ql.epilogue(sc, sh, True, ssum, ssq)
    ql.qlayer_conv2d_fwd_ex(d, x, *w, *b, y, ta, tb, epi=e)
    torch.cuda.synchronize()
    yr, _, _ = oracle.conv2d_fwd(inp["x"], inp["wa"], inp["wb"], inp["wc"], inp["ba"], inp["bb"], inp["bc"], s, p)
    ref_y, ref_sum, ref_sq = oracle.epilogue(yr, sc.double().cpu().numpy(), sh.double().cpu().numpy(), True)
    got_y = qlh.nhwc_to_np(y)
    assert qlh.relerr(got_y, ref_y) <= qlh.tol(True, False)
    # the sums are of the stored (rounded) values: compare with the sums of the stored output
    yd = got_y.astype("float64")
    assert qlh.relerr(ssum.double().cpu().numpy(), yd.sum(axis=(0, 2, 3))) <= 1e-5
    assert qlh.relerr(ssq.double().cpu().numpy(), (yd * yd).sum(axis=(0, 2, 3))) <= 1e-5
    assert qlh.relerr(ssum.double().cpu().numpy(), ref_sum) <= qlh.tol(True, False)
