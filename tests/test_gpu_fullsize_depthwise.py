"""GPU parity of the depthwise layer at the benchmark's full sizes, in its
launch configuration (default planner, workspace of the queried size): the
13 depthwise layers of a CIFAR MobileNet-V1 at batch 128 and the N=64,
C=256, 56 x 56 layer, bf16, the proposed neuron, each on the benchmark's own
seeded inputs.  The depthwise oracle is cheap enough to compare whole
tensors: Y, T_a, T_b, dX, dW_t and db_t, normwise, against the same limits
as the small cases (bf16 with fp32 accumulation: 2e-2)."""
import pytest

import synth

pytestmark = pytest.mark.gpu

from test_gpu_depthwise import check, oracle_dw, run_dw  # noqa: E402

PAIRS = synth.mobilenet_v1_pairs(128)


def _case(cfg_id, layer_id, L):
    print(f"full-size depthwise cfg={cfg_id} layer={layer_id} N={L.n} C={L.c} {L.h}x{L.w} s={L.stride}", flush=True)
    inp = synth.random_dwconv_case([cfg_id, layer_id], L.n, L.c, L.h, L.w, L.k, L.k, L.stride, L.pad, bf16=True)
    check(run_dw(0, inp, L.stride, L.pad, True), oracle_dw(0, inp, L.stride, L.pad), True)


@pytest.mark.parametrize("layer_id", range(len(PAIRS)), ids=lambda i: f"dw{i + 1}")
def test_mobilenet_v1_depthwise_full_size(layer_id):
    _case(7, layer_id, PAIRS[layer_id][0])


def test_large_depthwise_full_size():
    _case(9, 0, synth.ConvLayer(n=64, c=256, h=56, w=56, o=256, k=3, stride=1, pad=1))
