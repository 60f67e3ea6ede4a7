"""The forward epilogue (per-channel scale / shift, ReLU and the batch-
normalization sums of the stored output; arXiv 2204.01701 section 4.2, model
construction) through the C ABI, on every forward path: the staged epilogue
that gathers the sums itself, the 8-wave fp32 tile, split-K, the generic
kernel, unvectorised output channels, the depthwise kernels and the dense
layer; every neuron type.  y' is compared with the oracle element by element
(normwise relative error); the sums with an fp64 sum of the stored y' (bound
by the fp32 accumulation: 3e-5 times the sum of magnitudes) and with the
oracle's (the forward tolerance)."""
import os

import numpy as np
import pytest
import torch

import oracle
import synth

pytestmark = pytest.mark.gpu

import qlh  # noqa: E402
import paper_2204_01701_amd as ql  # noqa: E402

DEV = qlh.DEV
TERMS = ql.NEURON_TERMS

# (name, N, C, H, W, O, K, stride, pad, groups, planner overrides)
CONV_CASES = [
    ("staged", 2, 64, 16, 16, 64, 3, 1, 1, 1, {}),
    ("staged-ragged", 3, 32, 9, 7, 48, 3, 1, 1, 1, {}),
    ("eight-wave-tile", 2, 64, 16, 16, 128, 3, 1, 1, 1, {"QLAYER_FWD_CFG": "4"}),
    ("split-k", 4, 256, 4, 4, 256, 3, 1, 1, 1, {"QLAYER_FWD_KSPLIT": "0"}),  # the tiled kernel's combine
    ("ksplit", 4, 256, 4, 4, 256, 3, 1, 1, 1, {}),            # the small-output forward (sums per block)
    ("ksplit-2x2", 16, 64, 2, 2, 68, 3, 1, 1, 1, {}),         # ... position-major, ragged rows
    ("generic", 2, 12, 7, 5, 20, 3, 1, 1, 1, {}),
    ("odd-out-channels", 2, 16, 8, 8, 12, 3, 2, 1, 1, {}),
    ("narrow", 4, 16, 12, 12, 16, 3, 1, 1, 1, {}),          # the narrow forward (sums per wave)
    ("narrow-stem", 3, 3, 10, 10, 16, 3, 1, 1, 1, {}),       # ... on the zero-padded 3-channel stem
    ("depthwise", 2, 32, 9, 7, 32, 3, 1, 1, 32, {}),
    ("depthwise-5x5", 2, 24, 8, 8, 24, 5, 1, 2, 24, {}),
]
MODES = [  # scale, shift, relu, stats
    ("stats", False, False, False, True),
    ("affine-relu", True, True, True, False),
    ("all", True, True, True, True),
]


def _vec(rng, n, lo=None):
    v = rng.standard_normal(n).astype(np.float32)
    return np.abs(v) + 0.5 if lo else v


def _stats_check(got_y, got_sum, got_sumsq, ref_sum, ref_sumsq, bf16, axes):
    stored = got_y.astype(np.float64)
    s = stored.sum(axis=axes)
    a = np.abs(stored).sum(axis=axes)
    s2 = (stored * stored).sum(axis=axes)
    assert np.all(np.abs(got_sum - s) <= 3e-5 * a + 1e-30), "sum against the stored output"
    assert np.all(np.abs(got_sumsq - s2) <= 3e-5 * s2 + 1e-30), "sum of squares against the stored output"
    tol = qlh.tol(bf16, False)
    assert qlh.relerr(got_sum, ref_sum) <= max(tol, 1e-6) * 10, "sum against the oracle"
    assert qlh.relerr(got_sumsq, ref_sumsq) <= max(tol, 1e-6) * 10, "sum of squares against the oracle"


@pytest.fixture
def env():
    saved = {}

    def set_(kv):
        for k, v in kv.items():
            saved[k] = os.environ.get(k)
            os.environ[k] = v
    yield set_
    for k, v in saved.items():
        if v is None:
            os.environ.pop(k, None)
        else:
            os.environ[k] = v


@pytest.mark.parametrize("mode", MODES, ids=[m[0] for m in MODES])
@pytest.mark.parametrize("bf16", [False, True], ids=["fp32", "bf16"])
@pytest.mark.parametrize("case", CONV_CASES, ids=[c[0] for c in CONV_CASES])
def test_conv_epilogue_matches_oracle(case, bf16, mode, env):
    name, N, C, H, W, O, K, s, p, groups, over = case
    _, use_scale, use_shift, relu, stats = mode
    print(f"epilogue {name} bf16={bf16} mode={mode[0]}", flush=True)
    env(over)
    dw = groups > 1
    if dw:
        inp = synth.random_dwconv_case([700, N, C, H], N, C, H, W, K, K, s, p, bf16=bf16)
        y0, ta0, tb0 = oracle.dwconv2d_fwd(0, inp["x"], inp["wa"], inp["wb"], inp["wc"], inp["ba"], inp["bb"],
                                           inp["bc"], stride=s, pad=p)
    else:
        inp = synth.random_conv_case([701, N, C, H, O], N, C, H, W, O, K, K, s, p, bf16=bf16)
        y0, ta0, tb0 = oracle.conv2d_fwd(inp["x"], inp["wa"], inp["wb"], inp["wc"], inp["ba"], inp["bb"],
                                         inp["bc"], stride=s, pad=p)
    rng = np.random.default_rng(702)
    scale = _vec(rng, O, lo=True) * np.where(rng.random(O) < 0.3, -1, 1).astype(np.float32) if use_scale else None
    shift = _vec(rng, O) if use_shift else None
    ref_y, ref_sum, ref_sumsq = oracle.epilogue(y0, scale, shift, relu)
    d = ql.conv_desc(N, C, H, W, O, K, K, s, p, qlh.qdtype(bf16), groups=groups)
    dt = qlh.tdtype(bf16)
    x = qlh.nchw_to_dev(inp["x"], bf16)
    w = [qlh.oihw_to_dev(inp[k], bf16) for k in ("wa", "wb", "wc")]
    b = [qlh.vec_to_dev(inp[k]) for k in ("ba", "bb", "bc")]
    y = torch.empty((N, d.ho, d.wo, O), device=DEV, dtype=dt)
    ta, tb = torch.empty_like(y), torch.empty_like(y)
    sc, sh = qlh.vec_to_dev(scale), qlh.vec_to_dev(shift)
    ssum = torch.full((O,), float("nan"), device=DEV) if stats else None
    ssq = torch.full((O,), float("nan"), device=DEV) if stats else None
    epi = ql.epilogue(sc, sh, relu, ssum, ssq)
    ql.qlayer_conv2d_fwd_ex(d, x, *w, *b, y, ta, tb, epi=epi)
    torch.cuda.synchronize()
    got = qlh.conv_to_np({"y": y, "ta": ta})
    tol = qlh.tol(bf16, False)
    assert qlh.relerr(got["y"], ref_y) <= tol, "y'"
    assert qlh.relerr(got["ta"], ta0) <= tol, "T_a stays untransformed"
    if stats:
        _stats_check(got["y"], ssum.double().cpu().numpy(), ssq.double().cpu().numpy(), ref_sum, ref_sumsq, bf16,
                     (0, 2, 3))


@pytest.mark.parametrize("neuron", [1, 2, 3, 4], ids=["T4", "T4I", "T3", "T2"])
def test_epilogue_every_neuron_type(neuron):
    N, C, H, W, O = 2, 32, 8, 8, 32
    print(f"epilogue neuron {neuron}", flush=True)
    inp = synth.random_conv_case([703, neuron], N, C, H, W, O, 3, 3, 1, 1, bf16=True)
    nt = TERMS[neuron]
    wn = [inp["wa"], inp["wb"] if nt >= 2 else None, None]
    bn = [inp["ba"], inp["bb"] if nt >= 2 else None, None]
    y0, _, _ = oracle.conv2d_fwd_neuron(neuron, inp["x"], *wn, *bn, stride=1, pad=1)
    rng = np.random.default_rng(704)
    scale, shift = _vec(rng, O), _vec(rng, O)
    ref_y, ref_sum, ref_sumsq = oracle.epilogue(y0, scale, shift, True)
    d = ql.conv_desc(N, C, H, W, O, 3, 3, 1, 1, ql.QL_BF16, neuron)
    x = qlh.nchw_to_dev(inp["x"], True)
    w = [qlh.oihw_to_dev(inp[k], True) if i < nt else None for i, k in enumerate(("wa", "wb", "wc"))]
    b = [qlh.vec_to_dev(inp[k]) if i < nt else None for i, k in enumerate(("ba", "bb", "bc"))]
    y = torch.empty((N, H, W, O), device=DEV, dtype=torch.bfloat16)
    ta = torch.empty_like(y) if neuron != 4 else None
    tb = torch.empty_like(y) if nt >= 2 else None
    ssum, ssq = torch.empty(O, device=DEV), torch.empty(O, device=DEV)
    ql.qlayer_conv2d_fwd_ex(d, x, *w, *b, y, ta, tb,
                            epi=ql.epilogue(qlh.vec_to_dev(scale), qlh.vec_to_dev(shift), True, ssum, ssq))
    torch.cuda.synchronize()
    got = qlh.nhwc_to_np(y)
    assert qlh.relerr(got, ref_y) <= qlh.tol(True, False)
    _stats_check(got, ssum.double().cpu().numpy(), ssq.double().cpu().numpy(), ref_sum, ref_sumsq, True,
                 (0, 2, 3))


@pytest.mark.parametrize("bf16", [False, True], ids=["fp32", "bf16"])
def test_linear_epilogue_matches_oracle(bf16):
    B, I, O = 96, 72, 40
    print(f"epilogue dense bf16={bf16}", flush=True)
    inp = synth.random_dense_case([705], B, I, O, bf16=bf16)
    y0 = oracle.linear_fwd(inp["x"], inp["wa"], inp["wb"], inp["wc"], inp["ba"], inp["bb"], inp["bc"])[0]
    rng = np.random.default_rng(706)
    scale, shift = _vec(rng, O), _vec(rng, O)
    ref_y, ref_sum, ref_sumsq = oracle.epilogue(y0, scale, shift, True)
    d = ql.linear_desc(B, I, O, qlh.qdtype(bf16))
    dt = qlh.tdtype(bf16)
    x = torch.from_numpy(inp["x"]).to(DEV, dt)
    w = [torch.from_numpy(inp[k]).to(DEV, dt) for k in ("wa", "wb", "wc")]
    b = [qlh.vec_to_dev(inp[k]) for k in ("ba", "bb", "bc")]
    y = torch.empty((B, O), device=DEV, dtype=dt)
    ssum, ssq = torch.empty(O, device=DEV), torch.empty(O, device=DEV)
    ql.qlayer_linear_fwd_ex(d, x, *w, *b, y, None, None,
                            epi=ql.epilogue(qlh.vec_to_dev(scale), qlh.vec_to_dev(shift), True, ssum, ssq))
    torch.cuda.synchronize()
    got = y.double().cpu().numpy()
    assert qlh.relerr(got, ref_y) <= qlh.tol(bf16, False)
    _stats_check(got, ssum.double().cpu().numpy(), ssq.double().cpu().numpy(), ref_sum, ref_sumsq, bf16, (0,))


def test_epilogue_full_size_layer_and_repeatability():
    """The large layer (N=64, 256 -> 256, 56 x 56, bf16) in the benchmark's launch configuration:
    sums against an fp64 sum of the stored output, bitwise repeatable, and y' sampled against the oracle."""
    L = synth.LARGE_BF16
    print("epilogue large layer", flush=True)
    inp = synth.conv_inputs(4, 0, L, bf16=True, with_grad=False)
    d = ql.conv_desc(L.n, L.c, L.h, L.w, L.o, L.k, L.k, L.stride, L.pad, ql.QL_BF16)
    x = qlh.nchw_to_dev(inp["x"], True)
    w = [qlh.oihw_to_dev(inp[k], True) for k in ("wa", "wb", "wc")]
    b = [qlh.vec_to_dev(inp[k]) for k in ("ba", "bb", "bc")]
    y = torch.empty((L.n, L.ho, L.wo, L.o), device=DEV, dtype=torch.bfloat16)
    sums = []
    for _ in range(2):
        ssum, ssq = torch.empty(L.o, device=DEV), torch.empty(L.o, device=DEV)
        ql.qlayer_conv2d_fwd_ex(d, x, *w, *b, y, None, None, epi=ql.epilogue(None, None, False, ssum, ssq))
        torch.cuda.synchronize()
        sums.append((ssum.cpu().numpy(), ssq.cpu().numpy()))
    assert np.array_equal(sums[0][0], sums[1][0]) and np.array_equal(sums[0][1], sums[1][1])
    yd = y.double()
    s = yd.sum(dim=(0, 1, 2)).cpu().numpy()
    a = yd.abs().sum(dim=(0, 1, 2)).cpu().numpy()
    s2 = (yd * yd).sum(dim=(0, 1, 2)).cpu().numpy()
    assert np.all(np.abs(sums[0][0] - s) <= 3e-5 * a)
    assert np.all(np.abs(sums[0][1] - s2) <= 3e-5 * s2)
    rng = np.random.default_rng(707)
    idx = np.stack([rng.integers(0, n, 64) for n in (L.n, L.o, L.ho, L.wo)], axis=1)
    ref = oracle.conv2d_fwd_at(inp["x"], inp["wa"], inp["wb"], inp["wc"], inp["ba"], inp["bb"], inp["bc"], idx,
                               stride=L.stride, pad=L.pad)[0]
    got = np.array([y[n, i, j, o].float().item() for n, o, i, j in idx])
    assert qlh.relerr(got, ref) <= qlh.tol(True, False)


@pytest.mark.parametrize("case", [CONV_CASES[0], CONV_CASES[3], CONV_CASES[4], CONV_CASES[8]],
                         ids=["staged", "split-k", "ksplit", "depthwise"])
def test_epilogue_invariants(case, env):
    """fwd_ex with no epilogue (or an empty one) writes the plain forward's bits; the sums
    taken with the epilogue equal those of the plain output stored by it; scale = 1, shift = 0
    changes nothing."""
    name, N, C, H, W, O, K, s, p, groups, over = case
    print(f"epilogue invariants {name}", flush=True)
    env(over)
    if groups > 1:
        inp = synth.random_dwconv_case([708], N, C, H, W, K, K, s, p, bf16=True)
    else:
        inp = synth.random_conv_case([708], N, C, H, W, O, K, K, s, p, bf16=True)
    d = ql.conv_desc(N, C, H, W, O, K, K, s, p, ql.QL_BF16, groups=groups)
    x = qlh.nchw_to_dev(inp["x"], True)
    w = [qlh.oihw_to_dev(inp[k], True) for k in ("wa", "wb", "wc")]
    b = [qlh.vec_to_dev(inp[k]) for k in ("ba", "bb", "bc")]
    outs = []
    for epi in (None, ql.epilogue(), "stats", "unit"):
        y = torch.empty((N, d.ho, d.wo, O), device=DEV, dtype=torch.bfloat16)
        ta, tb = torch.empty_like(y), torch.empty_like(y)
        sums = None
        if epi is None:
            ql.qlayer_conv2d_fwd(d, x, *w, *b, y, ta, tb)
        elif epi == "stats":
            sums = (torch.empty(O, device=DEV), torch.empty(O, device=DEV))
            ql.qlayer_conv2d_fwd_ex(d, x, *w, *b, y, ta, tb, epi=ql.epilogue(None, None, False, *sums))
        elif epi == "unit":
            one, zero = torch.ones(O, device=DEV), torch.zeros(O, device=DEV)
            ql.qlayer_conv2d_fwd_ex(d, x, *w, *b, y, ta, tb, epi=ql.epilogue(one, zero, False))
        else:
            ql.qlayer_conv2d_fwd_ex(d, x, *w, *b, y, ta, tb, epi=epi)
        torch.cuda.synchronize()
        outs.append((y, ta, tb, sums))
    for y, ta, tb, _ in outs[1:]:
        assert torch.equal(y, outs[0][0]) and torch.equal(ta, outs[0][1]) and torch.equal(tb, outs[0][2])
    yd = outs[0][0].double()
    s1 = yd.sum(dim=(0, 1, 2)).cpu().numpy()
    a1 = yd.abs().sum(dim=(0, 1, 2)).cpu().numpy()
    got = outs[2][3][0].double().cpu().numpy()
    assert np.all(np.abs(got - s1) <= 3e-5 * a1 + 1e-30)
