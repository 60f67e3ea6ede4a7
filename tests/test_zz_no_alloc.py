"""The weight-gradient entry point that allocates nothing
(qlayer_conv2d_bwd_weight_noalloc, for callers that cannot allocate device
memory), through the C ABI, against the regular entry point that takes a
caller workspace and against the fp64 oracle.

Two calls in a row on the library's scratch array, the second with a smaller
layer; where the regular call's workspace fits the scratch array the two
entry points run the same plan and must agree bit for bit, otherwise (a layer
whose regular plan needs more) the no-allocation call splits less and must
meet the oracle tolerance."""
import numpy as np
import pytest
import torch

import oracle
import synth

pytestmark = pytest.mark.gpu

import qlh  # noqa: E402
import paper_2204_01701_amd as ql  # noqa: E402

DEV = qlh.DEV


def _inputs(seed, shape, bf16):
    N, C, H, W, O, K, s, p = shape
    inp = synth.random_conv_case(seed, N, C, H, W, O, K, K, s, p, bf16=bf16)
    d = ql.conv_desc(N, C, H, W, O, K, K, s, p, qlh.qdtype(bf16))
    x = qlh.nchw_to_dev(inp["x"], bf16)
    w = [qlh.oihw_to_dev(inp[k], bf16) for k in ("wa", "wb", "wc")]
    b = [qlh.vec_to_dev(inp[k]) for k in ("ba", "bb", "bc")]
    y = torch.empty((N, d.ho, d.wo, O), device=DEV, dtype=qlh.tdtype(bf16))
    ta, tb = torch.empty_like(y), torch.empty_like(y)
    ql.qlayer_conv2d_fwd(d, x, *w, *b, y, ta, tb)
    gy = qlh.nchw_to_dev(inp["gy"], bf16)
    return inp, d, x, gy, ta, tb


def _grads(d, O, K, C, fill=float("nan")):
    dw = [torch.full((O, K, K, C), fill, device=DEV, dtype=torch.float32) for _ in range(3)]
    db = [torch.full((O,), fill, device=DEV, dtype=torch.float32) for _ in range(3)]
    return dw, db


def _check_oracle(inp, shape, dw, db, bf16):
    N, C, H, W, O, K, s, p = shape
    ref = oracle.conv2d_bwd(inp["x"], inp["wa"], inp["wb"], inp["wc"], inp["ba"], inp["bb"], inp["bc"], inp["gy"],
                            s, p)
    for t, (kw, kb) in enumerate((("dwa", "dba"), ("dwb", "dbb"), ("dwc", "dbc"))):
        got_w = dw[t].permute(0, 3, 1, 2).double().cpu().numpy()
        assert qlh.relerr(got_w, ref[kw]) <= qlh.tol(bf16, True), kw
        assert qlh.relerr(db[t].double().cpu().numpy(), ref[kb]) <= qlh.tol(bf16, True), kb


# (shape N, C, H, W, O, K, s, p; bf16; the regular plan fits the scratch array)
CASES = [
    # first call: split-K partials in the scratch array (64 -> 64 on 16 x 16, bf16)
    ((16, 64, 16, 16, 64, 3, 1, 1), True, True),
    # second call, smaller: ragged tiles, stride 2, fp32 generic kernel
    ((2, 24, 9, 9, 40, 3, 2, 1), False, True),
    # a layer whose regular partials exceed the array (VGG-16 layer 6, 256 -> 256 on 8 x 8): fewer splits
    ((128, 256, 8, 8, 256, 3, 1, 1), True, False),
    # smaller again, few input channels (X padded in the scratch array)
    ((8, 3, 12, 12, 32, 3, 1, 1), True, True),
]


def test_noalloc_matches_the_workspace_entry_point_call_after_call():
    print("no-alloc weight gradient, calls in a row", flush=True)
    for i, (shape, bf16, fits) in enumerate(CASES):
        N, C, H, W, O, K, s, p = shape
        print(f"  call {i}: shape {shape} bf16={bf16}", flush=True)
        inp, d, x, gy, ta, tb = _inputs([700, i], shape, bf16)
        need = ql.qlayer_conv2d_bwd_weight_workspace_size(d)
        assert (need <= ql.NOALLOC_SCRATCH_BYTES) == fits, need
        dw0, db0 = _grads(d, O, K, C)
        ql.qlayer_conv2d_bwd_weight(d, x, gy, ta, tb, *dw0, *db0)
        dw1, db1 = _grads(d, O, K, C)
        ql.qlayer_conv2d_bwd_weight_noalloc(d, x, gy, ta, tb, *dw1, *db1)
        torch.cuda.synchronize()
        for a, b in zip(dw0 + db0, dw1 + db1):
            assert not torch.isnan(b).any()
            if fits:
                assert torch.equal(a, b)
        _check_oracle(inp, shape, dw1, db1, bf16)
