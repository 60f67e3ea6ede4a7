"""A CIFAR ResNet-20 training step built from the library's quadratic layers and
its network glue (arXiv 2204.01701, section 4.2, model construction: batch
normalization after every quadratic layer, ReLU in deeper networks; Table 3's
ResNet rows are CIFAR ResNets of this construction).

Every operation runs in libqlayer.so: the 19 quadratic 3x3 convolutions
(forward with the batch-normalization sums gathered by the forward epilogue,
input and weight gradients), batch normalization + shortcut + ReLU and their
backward (include/qnet.h), global average pooling and the quadratic
fully-connected classifier.  torch only allocates the device tensors.

The network: a 3 -> 16 stem (qconv, BN, ReLU), then three stages of three
basic blocks at 16 / 32 / 64 channels (qconv, BN, ReLU, qconv, BN, + shortcut,
ReLU), the first block of stages 2 and 3 with stride 2 and the option-A
shortcut (input subsampled by 2, channels placed at [C/4, C/4 + C_in)), then
global average pooling and a quadratic dense layer 64 -> 10.  Batch
normalization in training mode, gamma 1, beta 0, eps 1e-5.  One step is the
forward to the logits and the backward from a given gradient of the logits to
every weight and bias gradient (no optimizer update: the step of the
measurement).
"""
from __future__ import annotations

import torch

from . import (QL_BF16, QL_F32, conv_desc, epilogue, linear_desc, qlayer_conv2d_bwd_data,
               qlayer_conv2d_bwd_data_workspace_size, qlayer_conv2d_bwd_weight,
               qlayer_conv2d_bwd_weight_workspace_size, qlayer_conv2d_fwd_ex, qlayer_conv2d_fwd_ex_workspace_size,
               qlayer_linear_bwd, qlayer_linear_bwd_workspace_size, qlayer_linear_fwd,
               qlayer_linear_fwd_workspace_size, qnet_bn_act_bwd, qnet_bn_act_bwd_workspace_size, qnet_bn_act_fwd,
               qnet_gap_bwd, qnet_gap_fwd, qnet_residual_bwd)

EPS = 1e-5


def resnet20_geometry(batch=256, width=(16, 32, 64), blocks=3, image=32):
    """(c_in, h_in, w_in, c_out, stride) of the 19 quadratic 3x3 convolutions, in order."""
    geo = [(3, image, image, width[0], 1)]
    c, hw = width[0], image
    for si, wd in enumerate(width):
        for b in range(blocks):
            s = 2 if (si > 0 and b == 0) else 1
            geo.append((c, hw, hw, wd, s))
            hw //= s
            geo.append((wd, hw, hw, wd, 1))
            c = wd
    return geo


class ResNet20Step:
    """Device state and the forward / backward of the training step.

    params: per conv layer i (0..18) a dict of weights wa, wb, wc (O, C, 3, 3)
    and biases ba, bb, bc (O), and "head" with weights (10, 64) and biases (10),
    as torch CPU tensors or numpy arrays (moved to the device here); x the
    images (N, 3, 32, 32); g_logits dl/dlogits (N, 10)."""

    def __init__(self, params, x, g_logits, dtype=torch.bfloat16, device="cuda:0", num_classes=10):
        dev = torch.device(device)
        self.dev, self.dt = dev, dtype
        self.qdt = QL_BF16 if dtype == torch.bfloat16 else QL_F32
        n = int(x.shape[0])
        self.n = n
        self.geo = resnet20_geometry(n)

        def dev_nhwc(a):
            t = torch.as_tensor(a)
            return t.permute(0, 2, 3, 1).contiguous().to(dev, dtype)

        def dev_f32(a):
            return torch.as_tensor(a).to(dev, torch.float32).contiguous()

        self.x = dev_nhwc(x)
        self.layers = []
        ws_need = 0
        for i, (c, h, w, o, s) in enumerate(self.geo):
            d = conv_desc(n, c, h, w, o, 3, 3, s, 1, self.qdt)
            p = params[i]
            L = {"desc": d, "stride": s,
                 "w": [dev_nhwc(p[k]) for k in ("wa", "wb", "wc")],
                 "b": [dev_f32(p[k]) for k in ("ba", "bb", "bc")]}
            shp = (n, d.ho, d.wo, o)
            for k in ("y", "ta", "tb", "out", "g"):
                L[k] = torch.empty(shp, device=dev, dtype=dtype)
            for k in ("sum", "sumsq", "mean", "rstd"):
                L[k] = torch.empty(o, device=dev, dtype=torch.float32)
            L["dw"] = [torch.empty((o, 3, 3, c), device=dev, dtype=torch.float32) for _ in range(3)]
            L["db"] = [torch.empty(o, device=dev, dtype=torch.float32) for _ in range(3)]
            L["epi"] = epilogue(None, None, False, L["sum"], L["sumsq"])
            ws_need = max(ws_need, qlayer_conv2d_fwd_ex_workspace_size(d, L["epi"]),
                          qlayer_conv2d_bwd_data_workspace_size(d), qlayer_conv2d_bwd_weight_workspace_size(d),
                          qnet_bn_act_bwd_workspace_size(shp))
            self.layers.append(L)
        # the block input of every conv layer, and the gradient buffers of the activations
        for i, L in enumerate(self.layers):
            L["x"] = self.x if i == 0 else (self.layers[i - 1]["out"])
            if i > 0:
                L["dx"] = torch.empty_like(L["x"])
        hp = params["head"]
        c_last = self.geo[-1][3]
        self.z = torch.empty((n, c_last), device=dev, dtype=dtype)
        self.hd = linear_desc(n, c_last, num_classes, self.qdt)
        self.hw = [torch.as_tensor(hp[k]).to(dev, dtype).contiguous() for k in ("wa", "wb", "wc")]
        self.hb = [dev_f32(hp[k]) for k in ("ba", "bb", "bc")]
        self.logits = torch.empty((n, num_classes), device=dev, dtype=dtype)
        self.hta, self.htb = torch.empty_like(self.logits), torch.empty_like(self.logits)
        self.g_logits = torch.as_tensor(g_logits).to(dev, dtype).contiguous()
        self.dz = torch.empty_like(self.z)
        self.hdw = [torch.empty((num_classes, c_last), device=dev, dtype=torch.float32) for _ in range(3)]
        self.hdb = [torch.empty(num_classes, device=dev, dtype=torch.float32) for _ in range(3)]
        self.dlast = torch.empty_like(self.layers[-1]["out"])
        ws_need = max(ws_need, qlayer_linear_fwd_workspace_size(self.hd), qlayer_linear_bwd_workspace_size(self.hd))
        self.ws = torch.empty(max(ws_need, 256), device=dev, dtype=torch.uint8)
        self.wsp = (self.ws.data_ptr(), self.ws.numel())

    # ------------------------------------------------------------------
    def _block_starts(self):
        return range(1, len(self.layers), 2)

    def forward(self, stream):
        """Images -> logits (every quadratic layer saves T_a, T_b for the backward)."""
        Ls = self.layers
        for i, L in enumerate(Ls):
            qlayer_conv2d_fwd_ex(L["desc"], L["x"], *L["w"], *L["b"], L["y"], L["ta"], L["tb"], epi=L["epi"],
                                 workspace=self.wsp, stream=stream)
            # the second conv of a block adds the block input (the first conv's input)
            res = Ls[i - 1]["x"] if (i > 0 and i % 2 == 0) else None
            qnet_bn_act_fwd(L["y"], L["sum"], L["sumsq"], L["out"], L["mean"], L["rstd"], EPS, res=res, relu=True,
                            stream=stream)
        qnet_gap_fwd(Ls[-1]["out"], self.z, stream=stream)
        qlayer_linear_fwd(self.hd, self.z, *self.hw, *self.hb, self.logits, self.hta, self.htb,
                          workspace=self.wsp, stream=stream)

    def backward(self, stream):
        """dl/dlogits -> every weight and bias gradient."""
        Ls = self.layers
        qlayer_linear_bwd(self.hd, self.z, self.g_logits, self.hta, self.htb, *self.hw, self.dz, *self.hdw,
                          *self.hdb, workspace=self.wsp, stream=stream)
        qnet_gap_bwd(self.dz, self.dlast, stream=stream)
        dout = self.dlast
        for j in reversed(list(self._block_starts())):
            L1, L2 = Ls[j], Ls[j + 1]
            qnet_bn_act_bwd(dout, L2["out"], L2["y"], L2["mean"], L2["rstd"], L2["g"], relu=True,
                            workspace=self.wsp, stream=stream)
            qlayer_conv2d_bwd_data(L2["desc"], L2["g"], L2["ta"], L2["tb"], *L2["w"], L2["dx"], workspace=self.wsp,
                                   stream=stream)
            qlayer_conv2d_bwd_weight(L2["desc"], L2["x"], L2["g"], L2["ta"], L2["tb"], *L2["dw"], *L2["db"],
                                     workspace=self.wsp, stream=stream)
            qnet_bn_act_bwd(L2["dx"], L1["out"], L1["y"], L1["mean"], L1["rstd"], L1["g"], relu=True,
                            workspace=self.wsp, stream=stream)
            qlayer_conv2d_bwd_data(L1["desc"], L1["g"], L1["ta"], L1["tb"], *L1["w"], L1["dx"], workspace=self.wsp,
                                   stream=stream)
            qlayer_conv2d_bwd_weight(L1["desc"], L1["x"], L1["g"], L1["ta"], L1["tb"], *L1["dw"], *L1["db"],
                                     workspace=self.wsp, stream=stream)
            # the shortcut's share of the block output's gradient
            qnet_residual_bwd(dout, L2["out"], L1["dx"], stream=stream)
            dout = L1["dx"]
        L0 = Ls[0]
        qnet_bn_act_bwd(dout, L0["out"], L0["y"], L0["mean"], L0["rstd"], L0["g"], relu=True,
                        workspace=self.wsp, stream=stream)
        qlayer_conv2d_bwd_weight(L0["desc"], L0["x"], L0["g"], L0["ta"], L0["tb"], *L0["dw"], *L0["db"],
                                 workspace=self.wsp, stream=stream)

    def step(self, stream):
        self.forward(stream)
        self.backward(stream)

    def capture(self):
        """Record one step (about 130 kernel launches) as a HIP graph, so that a
        step is one launch from the host: replay() runs it on the current
        stream.  The library allocates nothing and clears nothing with
        memset, so the recorded launches are the step's kernels only."""
        side = torch.cuda.Stream(self.dev)
        side.wait_stream(torch.cuda.current_stream(self.dev))
        with torch.cuda.stream(side):
            self.step(side)  # an eager step first, outside the capture
        torch.cuda.current_stream(self.dev).wait_stream(side)
        torch.cuda.synchronize(self.dev)
        self.graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(self.graph):
            self.step(torch.cuda.current_stream(self.dev))
        return self.graph

    def replay(self):
        self.graph.replay()

    def qconv_calls(self):
        """(name, fn(stream)) of every quadratic-layer call of the step, for their share of its time."""
        calls = []
        for i, L in enumerate(self.layers):
            calls.append(((i, "fwd"), lambda st, L=L: qlayer_conv2d_fwd_ex(
                L["desc"], L["x"], *L["w"], *L["b"], L["y"], L["ta"], L["tb"], epi=L["epi"], workspace=self.wsp,
                stream=st)))
            if i > 0:
                calls.append(((i, "bwd_data"), lambda st, L=L: qlayer_conv2d_bwd_data(
                    L["desc"], L["g"], L["ta"], L["tb"], *L["w"], L["dx"], workspace=self.wsp, stream=st)))
            calls.append(((i, "bwd_weight"), lambda st, L=L: qlayer_conv2d_bwd_weight(
                L["desc"], L["x"], L["g"], L["ta"], L["tb"], *L["dw"], *L["db"], workspace=self.wsp, stream=st)))
        return calls
