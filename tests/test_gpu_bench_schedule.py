"""The benchmark's two-stream schedule is race-free: the weight gradients on
the second stream, released by device-scope events recorded after every
second forward, see the forward's T_a, T_b.  The saved maps and every output
are first filled with NaN; one overlapped step must then reproduce the
single-stream results bit for bit (all reductions have a fixed order)."""
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu

import qlh  # noqa: E402
import bench  # noqa: E402
import paper_2204_01701_amd as ql  # noqa: E402

DEV = qlh.DEV

GEOMS = [
    synth.ConvLayer(n=8, c=3, h=16, w=16, o=64, k=3, stride=1, pad=1),     # few-channel paths
    synth.ConvLayer(n=8, c=64, h=16, w=16, o=64, k=3, stride=1, pad=1),
    synth.ConvLayer(n=8, c=64, h=8, w=8, o=128, k=3, stride=1, pad=1),     # split-K reductions
    synth.ConvLayer(n=16, c=128, h=4, w=4, o=128, k=3, stride=1, pad=1),
    synth.ConvLayer(n=128, c=128, h=2, w=2, o=128, k=3, stride=1, pad=1),  # skipped padding taps
]


def _outputs(layers):
    return [[t.clone() for t in [ly.y, ly.ta, ly.tb, ly.dx] + ly.dw + ly.db] for ly in layers]


def test_overlapped_step_matches_single_stream():
    print("two-stream schedule vs single stream", flush=True)
    s1 = torch.cuda.current_stream(DEV)
    s2 = torch.cuda.Stream(DEV)
    layers = [bench.Layer(ql, torch, L, 11, i, DEV) for i, L in enumerate(GEOMS)]
    for ly in layers:
        ly.fwd(s1)
        ly.bwd_data(s1)
        ly.bwd_weight(s1)
    torch.cuda.synchronize()
    ref = _outputs(layers)
    for ly in layers:
        for t in [ly.y, ly.ta, ly.tb, ly.dx] + ly.dw + ly.db:
            t.fill_(float("nan"))
    torch.cuda.synchronize()
    bench.time_overlapped(torch, layers, 1, 0, s1, s2)
    got = _outputs(layers)
    for i, (g, r) in enumerate(zip(got, ref)):
        for k, (a, b) in enumerate(zip(g, r)):
            assert torch.equal(a, b), f"layer {i}, tensor {k}"
