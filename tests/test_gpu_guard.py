"""Guard bands around every output of every entry point.

Each output (and the workspace) is a slice of a larger buffer whose
elements before and after it hold a NaN sentinel bit pattern.  After the
call the guards must be bit for bit untouched (no kernel writes past its
output or its workspace), the outputs must hold no sentinel (every element
written) and must match the fp64 oracle within the normwise limits.
Geometries with ragged tiles, split-K and a depthwise layer, fp32 and bf16.
"""
import numpy as np
import pytest
import torch

import oracle
import synth

pytestmark = pytest.mark.gpu

import qlh  # noqa: E402
import paper_2204_01701_amd as ql  # noqa: E402

DEV = qlh.DEV
GUARD = 256  # guard elements on each side (keeps 16-byte alignment for every dtype)


class Guarded:
    """Buffers with sentinel guards; `view(shape, dtype)` returns the interior."""

    def __init__(self):
        self.bufs = []

    @staticmethod
    def _sentinel(dtype):
        return {torch.bfloat16: (torch.int16, 0x7FC1), torch.float32: (torch.int32, 0x7FC00A5A),
                torch.uint8: (torch.uint8, 0xA5)}[dtype]

    def view(self, shape, dtype):
        n = int(np.prod(shape))
        itype, pat = self._sentinel(dtype)
        raw = torch.full((GUARD + n + GUARD,), pat, dtype=itype, device=DEV)
        self.bufs.append((raw, n, pat))
        return raw.view(dtype)[GUARD:GUARD + n].view(shape)

    def check(self):
        for raw, n, pat in self.bufs:
            assert torch.all(raw[:GUARD] == pat), "guard before the buffer was written"
            assert torch.all(raw[GUARD + n:] == pat), "guard after the buffer was written"


def _conv_case(shape, bf16, groups=1):
    N, C, H, W, O, K, s, p = shape
    dw = groups == C
    inp = synth.random_conv_case([950] + list(shape) + [groups], N, C, H, W, O, K, K, s, p, bf16=bf16)
    if dw:
        for k in ("wa", "wb", "wc"):
            inp[k] = np.ascontiguousarray(inp[k][:, :1])  # one filter per channel: (C, 1, K, K)
    return inp


CONV = [((3, 20, 9, 7, 36, 3, 1, 1), 1), ((4, 256, 4, 4, 256, 3, 1, 1), 1), ((2, 16, 9, 9, 24, 3, 2, 1), 1),
        ((2, 24, 10, 9, 24, 3, 1, 1), 24)]


@pytest.mark.parametrize("bf16", [False, True], ids=["fp32", "bf16"])
@pytest.mark.parametrize("shape,groups", CONV, ids=lambda v: "x".join(map(str, v)) if isinstance(v, tuple) else f"g{v}")
def test_conv_entry_points_stay_inside_their_outputs(shape, groups, bf16):
    N, C, H, W, O, K, s, p = shape
    print(f"guard bands conv {shape} groups={groups} bf16={bf16}", flush=True)
    inp = _conv_case(shape, bf16, groups)
    d = ql.conv_desc(N, C, H, W, O, K, K, s, p, qlh.qdtype(bf16), groups=groups)
    dt = qlh.tdtype(bf16)
    cw = 1 if groups == C else C
    g = Guarded()
    x = qlh.nchw_to_dev(inp["x"], bf16)
    w = [qlh.oihw_to_dev(inp[k], bf16) for k in ("wa", "wb", "wc")]
    b = [qlh.vec_to_dev(inp[k]) for k in ("ba", "bb", "bc")]
    gy = qlh.nchw_to_dev(inp["gy"], bf16)
    ymap = (N, d.ho, d.wo, O)
    y, ta, tb = g.view(ymap, dt), g.view(ymap, dt), g.view(ymap, dt)
    ws = g.view((max(ql.qlayer_conv2d_fwd_workspace_size(d), 16),), torch.uint8)
    ql.qlayer_conv2d_fwd(d, x, *w, *b, y, ta, tb, workspace=ws)
    # the fused epilogue: affine + ReLU + statistics, on its own outputs
    y2 = g.view(ymap, dt)
    ssum, ssq = g.view((O,), torch.float32), g.view((O,), torch.float32)
    scale = torch.rand(O, device=DEV) + 0.5
    shift = torch.randn(O, device=DEV) * 0.1
    epi = ql.epilogue(scale, shift, True, ssum, ssq)
    ws2 = g.view((max(ql.qlayer_conv2d_fwd_ex_workspace_size(d, epi), 16),), torch.uint8)
    ql.qlayer_conv2d_fwd_ex(d, x, *w, *b, y2, None, None, epi=epi, workspace=ws2)
    dx = g.view(tuple(x.shape), dt)
    ws3 = g.view((max(ql.qlayer_conv2d_bwd_data_workspace_size(d), 16),), torch.uint8)
    ql.qlayer_conv2d_bwd_data(d, gy, ta, tb, *w, dx, workspace=ws3)
    dwt = [g.view((O, K, K, cw), torch.float32) for _ in range(3)]
    dbt = [g.view((O,), torch.float32) for _ in range(3)]
    ws4 = g.view((max(ql.qlayer_conv2d_bwd_weight_workspace_size(d), 16),), torch.uint8)
    ql.qlayer_conv2d_bwd_weight(d, x, gy, ta, tb, *dwt, *dbt, workspace=ws4)
    dwn = [g.view((O, K, K, cw), torch.float32) for _ in range(3)]
    dbn = [g.view((O,), torch.float32) for _ in range(3)]
    ql.qlayer_conv2d_bwd_weight_noalloc(d, x, gy, ta, tb, *dwn, *dbn)
    torch.cuda.synchronize()
    g.check()

    if groups == C:
        ry, rta, rtb = oracle.dwconv2d_fwd(0, inp["x"], inp["wa"], inp["wb"], inp["wc"], inp["ba"], inp["bb"],
                                           inp["bc"], stride=s, pad=p)
        ref = oracle.dwconv2d_bwd(0, inp["x"], inp["wa"], inp["wb"], inp["wc"], inp["ba"], inp["bb"], inp["bc"],
                                  inp["gy"], stride=s, pad=p)
    else:
        ry, rta, rtb = oracle.conv2d_fwd(inp["x"], inp["wa"], inp["wb"], inp["wc"], inp["ba"], inp["bb"], inp["bc"],
                                         s, p)
        ref = oracle.conv2d_bwd(inp["x"], inp["wa"], inp["wb"], inp["wc"], inp["ba"], inp["bb"], inp["bc"],
                                inp["gy"], s, p)
    ye, se, s2e = oracle.epilogue(ry, scale.double().cpu().numpy(), shift.double().cpu().numpy(), True)
    got = {"y": y, "ta": ta, "tb": tb, "dx": dx}
    want = {"y": ry, "ta": rta, "tb": rtb, "dx": ref["dx"]}
    for k, v in got.items():
        assert not torch.isnan(v.float()).any(), f"{k}: an element was not written"
        e = qlh.relerr(qlh.nhwc_to_np(v), want[k])
        assert e <= qlh.tol(bf16, k == "dx"), f"{k}: {e:.3e}"
    e = qlh.relerr(qlh.nhwc_to_np(y2), ye)
    assert e <= qlh.tol(bf16, False), f"epilogue y': {e:.3e}"
    for tag, v, r in (("sum", ssum, se), ("sumsq", ssq, s2e)):
        # sums of the stored (rounded) y'; ten times the forward limit as in the epilogue tests
        assert qlh.relerr(v.double().cpu().numpy(), r) <= 10 * qlh.tol(bf16, False), tag
    for dws, dbs in ((dwt, dbt), (dwn, dbn)):
        for t, (kw, kb) in enumerate((("dwa", "dba"), ("dwb", "dbb"), ("dwc", "dbc"))):
            gw = dws[t].permute(0, 3, 1, 2).double().cpu().numpy()
            assert not np.isnan(gw).any() and not torch.isnan(dbs[t]).any()
            assert qlh.relerr(gw, ref[kw]) <= qlh.tol(bf16, True), kw
            assert qlh.relerr(dbs[t].double().cpu().numpy(), ref[kb]) <= qlh.tol(bf16, True), kb


@pytest.mark.parametrize("bf16", [False, True], ids=["fp32", "bf16"])
def test_dense_entry_points_stay_inside_their_outputs(bf16):
    B, I, O = 70, 40, 52
    print(f"guard bands dense {B}x{I}->{O} bf16={bf16}", flush=True)
    inp = synth.random_dense_case([951, B, I, O], B, I, O, bf16=bf16)
    d = ql.linear_desc(B, I, O, qlh.qdtype(bf16))
    dt = qlh.tdtype(bf16)
    g = Guarded()
    x = torch.from_numpy(inp["x"]).to(DEV, dt)
    w = [torch.from_numpy(inp[k]).to(DEV, dt) for k in ("wa", "wb", "wc")]
    b = [qlh.vec_to_dev(inp[k]) for k in ("ba", "bb", "bc")]
    gy = torch.from_numpy(inp["gy"]).to(DEV, dt)
    y, ta, tb = g.view((B, O), dt), g.view((B, O), dt), g.view((B, O), dt)
    ws = g.view((max(ql.qlayer_linear_fwd_workspace_size(d), 16),), torch.uint8)
    ql.qlayer_linear_fwd(d, x, *w, *b, y, ta, tb, workspace=ws)
    y2 = g.view((B, O), dt)
    ssum, ssq = g.view((O,), torch.float32), g.view((O,), torch.float32)
    epi = ql.epilogue(None, None, False, ssum, ssq)
    ws2 = g.view((max(ql.qlayer_linear_fwd_ex_workspace_size(d, epi), 16),), torch.uint8)
    ql.qlayer_linear_fwd_ex(d, x, *w, *b, y2, None, None, epi=epi, workspace=ws2)
    dx = g.view((B, I), dt)
    dwt = [g.view((O, I), torch.float32) for _ in range(3)]
    dbt = [g.view((O,), torch.float32) for _ in range(3)]
    ws3 = g.view((max(ql.qlayer_linear_bwd_workspace_size(d), 16),), torch.uint8)
    ql.qlayer_linear_bwd(d, x, gy, ta, tb, *w, dx, *dwt, *dbt, workspace=ws3)
    torch.cuda.synchronize()
    g.check()
    ry, rta, rtb = oracle.linear_fwd(inp["x"], inp["wa"], inp["wb"], inp["wc"], inp["ba"], inp["bb"], inp["bc"])
    ref = oracle.linear_bwd(inp["x"], inp["wa"], inp["wb"], inp["wc"], inp["ba"], inp["bb"], inp["bc"], inp["gy"])
    _, se, s2e = oracle.epilogue(ry)
    for k, v, r in (("y", y, ry), ("ta", ta, rta), ("tb", tb, rtb), ("y2", y2, ry), ("dx", dx, ref["dx"])):
        assert not torch.isnan(v.float()).any(), k
        assert qlh.relerr(v.double().cpu().numpy(), r) <= qlh.tol(bf16, k == "dx"), k
    for tag, v, r in (("sum", ssum, se), ("sumsq", ssq, s2e)):
        assert qlh.relerr(v.double().cpu().numpy(), r) <= 10 * qlh.tol(bf16, False), tag
    for t, (kw, kb) in enumerate((("dwa", "dba"), ("dwb", "dbb"), ("dwc", "dbc"))):
        assert qlh.relerr(dwt[t].double().cpu().numpy(), ref[kw]) <= qlh.tol(bf16, True), kw
        assert qlh.relerr(dbt[t].double().cpu().numpy(), ref[kb]) <= qlh.tol(bf16, True), kb


def test_t24_input_gradient_stays_inside_its_output():
    N, C, H, W, O, K, s, p = 2, 24, 10, 9, 40, 3, 1, 1
    print("guard bands T2&4 input gradient", flush=True)
    inp = synth.random_conv_case([952], N, C, H, W, O, K, K, s, p, bf16=True)
    d = ql.conv_desc(N, C, H, W, O, K, K, s, p, ql.QL_BF16, ql.QL_NEURON_T24)
    g = Guarded()
    x = qlh.nchw_to_dev(inp["x"], True)
    w = [qlh.oihw_to_dev(inp[k], True) for k in ("wa", "wb", "wc")]
    b = [qlh.vec_to_dev(inp[k]) for k in ("ba", "bb", "bc")]
    y = torch.empty((N, H, W, O), device=DEV, dtype=torch.bfloat16)
    ta, tb = torch.empty_like(y), torch.empty_like(y)
    ql.qlayer_conv2d_fwd(d, x, *w, *b, y, ta, tb)
    dx = g.view(tuple(x.shape), torch.bfloat16)
    ws = g.view((max(ql.qlayer_conv2d_bwd_data_workspace_size(d), 16),), torch.uint8)
    ql.qlayer_conv2d_bwd_data_ex(d, qlh.nchw_to_dev(inp["gy"], True), ta, tb, x, *w, dx, workspace=ws)
    torch.cuda.synchronize()
    g.check()
    ref = oracle.conv2d_bwd_neuron(ql.QL_NEURON_T24, inp["x"], inp["wa"], inp["wb"], inp["wc"], inp["ba"],
                                   inp["bb"], inp["bc"], inp["gy"], stride=s, pad=p)
    assert qlh.relerr(qlh.nhwc_to_np(dx), ref["dx"]) <= qlh.tol(True, True)
