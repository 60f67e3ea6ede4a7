"""Exact (bitwise) properties of the GPU path that follow from the neuron's
definition (arXiv 2204.01701, section 3.1 eq:2ndneuron3 and section 4.3
eq:SD) and from how the kernels order their arithmetic:

* swapping (W_a, b_a) <-> (W_b, b_b) swaps T_a <-> T_b, dW_a <-> dW_b and
  db_a <-> db_b exactly and leaves Y unchanged (the product commutes);
* scaling (W_a, b_a) by 2 and (W_b, b_b) by 1/2 leaves Y unchanged;
* the recompute mode (no Y, terms only) regenerates T_a and T_b exactly;
* two runs on the same inputs agree bit for bit (deterministic split-K).
"""
import numpy as np
import pytest
import torch

import synth
import qlh  # noqa: E402

pytestmark = pytest.mark.gpu

SHAPES = [(2, 16, 8, 8, 32, 3, 3, 1, 1), (2, 64, 4, 4, 64, 3, 3, 1, 1), (1, 5, 6, 6, 7, 3, 3, 2, 1),
          (4, 16, 16, 16, 32, 3, 3, 1, 1),
          (4, 16, 12, 12, 16, 3, 3, 1, 1),  # (the narrow kernels of all three passes)
          (16, 64, 2, 2, 64, 3, 3, 1, 1)]   # (position-major small-output forward and input gradient)


def _eq(a, b):
    return torch.equal(a, b)


@pytest.mark.parametrize("bf16", [False, True], ids=["fp32", "bf16"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_swap_scale_recompute_determinism(shape, bf16):
    N, C, H, W, O, KH, KW, s, p = shape
    print(f"invariants shape={shape} bf16={bf16}", flush=True)
    inp = synth.random_conv_case([400] + list(shape), N, C, H, W, O, KH, KW, s, p, bf16=bf16)
    base = qlh.run_conv(inp, s, p, bf16, recompute=True)
    again = qlh.run_conv(inp, s, p, bf16)
    for k in again:
        assert _eq(base[k], again[k]), f"run-to-run difference in {k}"
    assert _eq(base["ta_re"], base["ta"]) and _eq(base["tb_re"], base["tb"])

    sw = dict(inp)
    sw["wa"], sw["wb"], sw["ba"], sw["bb"] = inp["wb"], inp["wa"], inp["bb"], inp["ba"]
    r = qlh.run_conv(sw, s, p, bf16)
    assert _eq(r["y"], base["y"])
    assert _eq(r["ta"], base["tb"]) and _eq(r["tb"], base["ta"])
    assert _eq(r["dwa"], base["dwb"]) and _eq(r["dwb"], base["dwa"]) and _eq(r["dwc"], base["dwc"])
    assert _eq(r["dba"], base["dbb"]) and _eq(r["dbb"], base["dba"]) and _eq(r["dbc"], base["dbc"])
    assert qlh.relerr(qlh.nhwc_to_np(r["dx"]), qlh.nhwc_to_np(base["dx"])) <= qlh.tol(bf16, True)

    sc = dict(inp)
    sc["wa"], sc["ba"] = inp["wa"] * np.float32(2), inp["ba"] * np.float32(2)
    sc["wb"], sc["bb"] = inp["wb"] * np.float32(0.5), inp["bb"] * np.float32(0.5)
    r2 = qlh.run_conv(sc, s, p, bf16)
    assert _eq(r2["y"], base["y"])
    assert _eq(r2["ta"].float(), base["ta"].float() * 2) and _eq(r2["tb"].float(), base["tb"].float() * 0.5)
