"""Differentiable quadratic layers on top of the C ABI (arXiv 2204.01701).

``quad_conv2d`` and ``quad_linear`` are torch autograd functions whose
forward and backward run entirely in ``libqlayer.so``: the forward computes
Y = (W_a*X + b_a) o (W_b*X + b_b) + (W_c*X + b_c) (section 3.1,
eq:2ndneuron3), the backward the input, weight and bias gradients of
section 4.3 (eq:SD).  They offer the two memory modes of section 4.3:

* ``recompute=False`` (save): the forward keeps T_a = W_a*X + b_a and
  T_b = W_b*X + b_b for the backward;
* ``recompute=True`` (hybrid back-propagation): the forward keeps only X, and
  the backward regenerates T_a and T_b with the forward kernel (Y not
  written) before the gradient kernels.  The gradients are bitwise those of
  save mode, since the same kernel produces T_a and T_b in both.

``neuron`` selects the layer type (``QL_NEURON_*``): the proposed neuron or
one of the earlier designs of Table 1 (T4, T4 + identity, T3, T2, T2&4).  Weights
and biases of the terms a type lacks are passed as None.  T2 saves nothing
but X in either mode (its backward needs only X).

``relu=True`` applies the activation deeper networks put after each
quadratic layer (section 4.2, model construction) in the forward kernel's
epilogue; the backward is one library call that masks the incoming gradient
with y' > 0 and forms the layer's own gradients from it (no elementwise torch
operation).  ``groups`` (convolution): 1, or C for the
depth-wise setting (weights (C, 1, KH, KW)).

Layouts.  Convolution tensors are NCHW-shaped torch tensors; they are used in
channels_last memory format, whose memory is the library's NHWC (OHWI for
weights), so channels_last inputs are not copied and the outputs come back
channels_last.  X, the weights and Y share one dtype (bfloat16 or float32);
biases are float32 or None (all three or none).  Weight gradients are
returned in the weights' dtype, bias gradients in float32.
"""
from __future__ import annotations

import torch

from . import (NEURON_TERMS, QL_BF16, QL_F32, QL_NEURON_QUADRA, QL_NEURON_T2, QL_NEURON_T24, conv_desc, epilogue,
               linear_desc, qlayer_conv2d_bwd_data, qlayer_conv2d_bwd_data_ex, qlayer_conv2d_bwd_relu,
               qlayer_conv2d_bwd_weight, qlayer_conv2d_fwd, qlayer_conv2d_fwd_ex,
               qlayer_linear_bwd, qlayer_linear_bwd_relu, qlayer_linear_fwd, qlayer_linear_fwd_ex)

__all__ = ["quad_conv2d", "quad_linear", "QuadConv2dFunction", "QuadLinearFunction"]


def _qdtype(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return QL_BF16
    if t.dtype == torch.float32:
        return QL_F32
    raise TypeError(f"unsupported dtype {t.dtype}: use bfloat16 or float32")


def _nhwc(t: torch.Tensor) -> torch.Tensor:
    """NCHW-shaped tensor -> contiguous NHWC view of its channels_last memory."""
    return t.contiguous(memory_format=torch.channels_last).permute(0, 2, 3, 1)


def _biases(ba, bb, bc, nt, O):
    bs = (ba, bb, bc)[:nt]
    if all(b is None for b in bs):
        return None
    if any(b is None for b in bs):
        raise ValueError("give the biases of every term of the neuron type or none")
    if any(b.numel() != O for b in bs):
        raise ValueError(f"each bias must have O = {O} elements")
    return [b.contiguous().float() for b in bs] + [None] * (3 - nt)


def _same_device(x, *others):
    """Every tensor on x's CUDA device (the kernels take raw device pointers)."""
    if x.device.type != "cuda":
        raise ValueError(f"the layer runs on a CUDA device; x is on {x.device}")
    for t in others:
        if t is not None and t.device != x.device:
            raise ValueError(f"every tensor must be on {x.device}; one is on {t.device}")


def _terms(ws, nt):
    if any(w is None for w in ws[:nt]):
        raise ValueError(f"the neuron type has {nt} weighted terms")
    return list(ws[:nt]) + [None] * (3 - nt)


class QuadConv2dFunction(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, wa, wb, wc, ba, bb, bc, stride, pad, recompute, neuron=QL_NEURON_QUADRA, relu=False,
                groups=1):
        N, C, H, W = x.shape
        O, C2, KH, KW = wa.shape
        nt = NEURON_TERMS[neuron]
        ws = _terms((wa, wb, wc), nt)
        if C2 * groups != C or any(w.shape != wa.shape for w in ws[:nt]):
            raise ValueError("weight shapes must be (O, C / groups, KH, KW) for every term")
        _same_device(x, *ws, ba, bb, bc)
        d = conv_desc(N, C, H, W, O, KH, KW, stride, pad, _qdtype(x), neuron, groups=groups)
        xn = _nhwc(x)
        wn = [_nhwc(w.to(x.dtype)) if w is not None else None for w in ws]
        b = _biases(ba, bb, bc, nt, O)
        bl = b if b is not None else [None, None, None]
        y = torch.empty((N, d.ho, d.wo, O), device=x.device, dtype=x.dtype)
        recompute = recompute or neuron == QL_NEURON_T2  # (T2 saves nothing but X)
        ta = torch.empty_like(y) if not recompute else None
        tb = torch.empty_like(y) if not recompute and nt >= 2 else None
        if relu:
            qlayer_conv2d_fwd_ex(d, xn, *wn, *bl, y, ta, tb, epi=epilogue(relu=True))
        else:
            qlayer_conv2d_fwd(d, xn, *wn, *bl, y, ta, tb)
        # Everything the backward reads goes through save_for_backward, the
        # output y' (the ReLU mask) included: an in-place change of any of them
        # then fails the version check instead of silently changing the
        # gradients, and no reference cycle through ctx keeps them alive.
        ctx.save_for_backward(xn, *wn, *bl, ta, tb, y if relu else None)
        ctx.desc, ctx.recompute, ctx.has_bias, ctx.nt, ctx.neuron = d, recompute, b is not None, nt, neuron
        ctx.wdtype = wa.dtype
        return y.permute(0, 3, 1, 2)

    @staticmethod
    def backward(ctx, gy):
        d, nt = ctx.desc, ctx.nt
        xn, wa, wb, wc, ba, bb, bc, ta, tb, relu_y = ctx.saved_tensors
        wn, bl = [wa, wb, wc], [ba, bb, bc]
        if ctx.neuron == QL_NEURON_T2:
            ta = xn  # its input gradient takes X in place of a saved map
        elif ctx.recompute:
            ta = torch.empty((d.n, d.ho, d.wo, d.o), device=xn.device, dtype=xn.dtype)
            tb = torch.empty_like(ta) if nt >= 2 else None
            qlayer_conv2d_fwd(d, xn, *wn, *bl, None, ta, tb)
        gyn = _nhwc(gy.to(xn.dtype))
        need_x, need_w = ctx.needs_input_grad[0], any(ctx.needs_input_grad[1:4])
        need_b = ctx.has_bias and any(ctx.needs_input_grad[4:7])
        dx = dw = db = None
        if relu_y is not None and (need_x or need_w or need_b):
            # the ReLU's mask and both gradients in one library call (G = gy o [y' > 0] formed once)
            dxn = torch.empty_like(xn) if need_x else None
            dwn = [torch.empty(wn[0].shape, device=xn.device, dtype=torch.float32) if i < nt else None
                   for i in range(3)] if (need_w or need_b) else [None, None, None]
            db = [torch.empty(d.o, device=xn.device, dtype=torch.float32) if i < nt else None
                  for i in range(3)] if need_b else None
            qlayer_conv2d_bwd_relu(d, xn, gyn, relu_y, None if ctx.neuron == QL_NEURON_T2 else ta, tb, *wn, dxn,
                                   *dwn, *(db or [None, None, None]))
            dx = dxn.permute(0, 3, 1, 2) if need_x else None
            dw = [g.permute(0, 3, 1, 2).to(ctx.wdtype) if g is not None else None for g in dwn]
            db = db or [None, None, None]
            return (dx, *dw, *db, None, None, None, None, None, None)
        if need_x:
            dxn = torch.empty_like(xn)
            if ctx.neuron == QL_NEURON_T24:  # (the chain rule through X o X needs X)
                qlayer_conv2d_bwd_data_ex(d, gyn, ta, tb, xn, *wn, dxn)
            else:
                qlayer_conv2d_bwd_data(d, gyn, ta, tb, *wn, dxn)
            dx = dxn.permute(0, 3, 1, 2)
        if need_w or need_b:
            dwn = [torch.empty(wn[0].shape, device=xn.device, dtype=torch.float32) if i < nt else None
                   for i in range(3)]
            db = [torch.empty(d.o, device=xn.device, dtype=torch.float32) if i < nt else None
                  for i in range(3)] if need_b else None
            qlayer_conv2d_bwd_weight(d, xn, gyn, None if ctx.neuron == QL_NEURON_T2 else ta, tb, *dwn,
                                     *(db or [None, None, None]))
            dw = [g.permute(0, 3, 1, 2).to(ctx.wdtype) if g is not None else None for g in dwn]
        dw = dw or [None, None, None]
        db = db or [None, None, None]
        return (dx, *dw, *db, None, None, None, None, None, None)


class QuadLinearFunction(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, wa, wb, wc, ba, bb, bc, recompute, neuron=QL_NEURON_QUADRA, relu=False):
        if x.dim() != 2 or wa.dim() != 2:
            raise ValueError("x must be (B, I) and the weights (O, I)")
        B, I = x.shape
        O = wa.shape[0]
        nt = NEURON_TERMS[neuron]
        ws = _terms((wa, wb, wc), nt)
        if wa.shape[1] != I or any(w.shape != wa.shape for w in ws[:nt]):
            raise ValueError(f"weight shapes must be (O, {I}) for every term")
        _same_device(x, *ws, ba, bb, bc)
        d = linear_desc(B, I, O, _qdtype(x), neuron)
        xc = x.contiguous()
        wl = [w.to(x.dtype).contiguous() if w is not None else None for w in ws]
        b = _biases(ba, bb, bc, nt, O)
        bl = b if b is not None else [None, None, None]
        y = torch.empty((B, O), device=x.device, dtype=x.dtype)
        recompute = recompute or neuron == QL_NEURON_T2
        ta = torch.empty_like(y) if not recompute else None
        tb = torch.empty_like(y) if not recompute and nt >= 2 else None
        if relu:
            qlayer_linear_fwd_ex(d, xc, *wl, *bl, y, ta, tb, epi=epilogue(relu=True))
        else:
            qlayer_linear_fwd(d, xc, *wl, *bl, y, ta, tb)
        ctx.save_for_backward(xc, *wl, *bl, ta, tb, y if relu else None)
        ctx.desc, ctx.recompute, ctx.has_bias, ctx.nt, ctx.neuron = d, recompute, b is not None, nt, neuron
        ctx.wdtype = wa.dtype
        return y

    @staticmethod
    def backward(ctx, gy):
        d, nt = ctx.desc, ctx.nt
        xc, wa, wb, wc, ba, bb, bc, ta, tb, relu_y = ctx.saved_tensors
        wl, bl = [wa, wb, wc], [ba, bb, bc]
        if ctx.neuron == QL_NEURON_T2:
            pass  # the dense backward takes X itself
        elif ctx.recompute:
            ta = torch.empty((d.batch, d.out), device=xc.device, dtype=xc.dtype)
            tb = torch.empty_like(ta) if nt >= 2 else None
            qlayer_linear_fwd(d, xc, *wl, *bl, None, ta, tb)
        gyc = gy.to(xc.dtype).contiguous()
        need_x, need_w = ctx.needs_input_grad[0], any(ctx.needs_input_grad[1:4])
        need_b = ctx.has_bias and any(ctx.needs_input_grad[4:7])
        if not (need_x or need_w or need_b):
            return (None,) * 10
        dx = torch.empty_like(xc) if need_x else None
        dw = [torch.empty(wl[0].shape, device=xc.device, dtype=torch.float32) if i < nt else None
              for i in range(3)] if (need_w or need_b) else None
        db = [torch.empty(d.out, device=xc.device, dtype=torch.float32) if i < nt else None
              for i in range(3)] if need_b else None
        if relu_y is not None:  # the ReLU's mask and both gradients in one library call
            qlayer_linear_bwd_relu(d, xc, gyc, relu_y, ta, tb, *wl, dx, *(dw or [None] * 3), *(db or [None] * 3))
        else:
            qlayer_linear_bwd(d, xc, gyc, ta, tb, *wl, dx, *(dw or [None] * 3), *(db or [None] * 3))
        dw = [g.to(ctx.wdtype) if g is not None else None for g in dw] if dw is not None else [None, None, None]
        db = db or [None, None, None]
        return (dx, *dw, *db, None, None, None)


def quad_conv2d(x, wa, wb=None, wc=None, ba=None, bb=None, bc=None, stride=1, pad=0, recompute=False,
                neuron=QL_NEURON_QUADRA, relu=False, groups=1):
    """Quadratic 2-D convolution layer (NCHW-shaped tensors, channels_last memory)."""
    return QuadConv2dFunction.apply(x, wa, wb, wc, ba, bb, bc, stride, pad, recompute, neuron, relu, groups)


def quad_linear(x, wa, wb=None, wc=None, ba=None, bb=None, bc=None, recompute=False, neuron=QL_NEURON_QUADRA,
                relu=False):
    """Quadratic fully-connected layer: x (B, I), weights (O, I)."""
    return QuadLinearFunction.apply(x, wa, wb, wc, ba, bb, bc, recompute, neuron, relu)
