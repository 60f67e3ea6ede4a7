"""MI355X (gfx950) quadratic-neuron layers -- Python binding of ``libqlayer.so``.

The layer is the quadratic neuron of QuadraLib (arXiv 2204.01701, section 3.1,
eq:2ndneuron3): Y = (W_a*X + b_a) o (W_b*X + b_b) + (W_c*X + b_c), applied as a
2-D convolution and as a fully-connected layer, with the backward pass of
section 4.3 (eq:SD).  All arithmetic runs in the HIP kernels of the C
library; this module only marshals arguments through ctypes: torch tensors
become device pointers, the current HIP stream becomes the stream argument,
and workspaces are allocated with torch when the caller passes none.

Function names, argument order and layouts match ``include/qlayer.h``:
activations NHWC, conv weights OHWI, dense X B x I and W O x I, biases and
weight/bias gradients float32.  Every function raises ``QLError`` on a
non-zero status.  There is no fallback: if the library is not built, the
import of the first function call fails loudly.
"""
from __future__ import annotations

import ctypes
import os

__all__ = [
    "QL_F32", "QL_BF16", "QL_NEURON_QUADRA", "QL_NEURON_T4", "QL_NEURON_T4_IDENTITY", "QL_NEURON_T3",
    "QL_NEURON_T2", "QL_NEURON_T24", "NEURON_TERMS", "QLError", "ConvDesc", "LinearDesc", "conv_desc", "linear_desc", "lib",
    "qlayer_version", "qlayer_status_string",
    "qlayer_conv2d_fwd_workspace_size", "qlayer_conv2d_fwd",
    "qlayer_conv2d_bwd_data_workspace_size", "qlayer_conv2d_bwd_data", "qlayer_conv2d_bwd_data_ex",
    "qlayer_conv2d_bwd_weight_workspace_size", "qlayer_conv2d_bwd_weight", "qlayer_conv2d_bwd_weight_noalloc",
    "NOALLOC_SCRATCH_BYTES",
    "qlayer_linear_fwd_workspace_size", "qlayer_linear_fwd",
    "qlayer_linear_bwd_workspace_size", "qlayer_linear_bwd",
    "qlayer_conv2d_bwd_relu_workspace_size", "qlayer_conv2d_bwd_relu",
    "qlayer_linear_bwd_relu_workspace_size", "qlayer_linear_bwd_relu",
]

QL_F32 = 0
QL_BF16 = 1
# neuron types (qlayer.h ql_neuron): the proposed one and the earlier designs of Table 1
QL_NEURON_QUADRA, QL_NEURON_T4, QL_NEURON_T4_IDENTITY, QL_NEURON_T3, QL_NEURON_T2 = 0, 1, 2, 3, 4
QL_NEURON_T24 = 5  # T2&4: T_a o T_b + W_c (X o X) + b_c
NEURON_TERMS = {0: 3, 1: 2, 2: 2, 3: 1, 4: 1, 5: 3}  # first-order terms (weights) per type

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libqlayer.so")


class QLError(RuntimeError):
    def __init__(self, func, status):
        self.status = status
        super().__init__(f"{func} failed: status {status} ({qlayer_status_string(status)})")


class ConvDesc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int) for n in
                ("n", "c", "h", "w", "o", "kh", "kw", "stride_h", "stride_w", "pad_h", "pad_w", "dtype", "neuron",
                 "groups")]

    @property
    def ho(self):
        return (self.h + 2 * self.pad_h - self.kh) // self.stride_h + 1

    @property
    def wo(self):
        return (self.w + 2 * self.pad_w - self.kw) // self.stride_w + 1


class LinearDesc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int), ("in_", ctypes.c_int), ("out", ctypes.c_int), ("dtype", ctypes.c_int),
                ("neuron", ctypes.c_int)]


class NetShape(ctypes.Structure):
    """qnet_shape: an NHWC tensor shape."""
    _fields_ = [(n, ctypes.c_int) for n in ("n", "h", "w", "c")]


def net_shape(t_or_dims) -> NetShape:
    """NetShape of an (N, H, W, C) tensor or tuple."""
    n, h, w, c = tuple(t_or_dims.shape) if hasattr(t_or_dims, "shape") else tuple(t_or_dims)
    return NetShape(n, h, w, c)


class Epilogue(ctypes.Structure):
    """ql_epilogue: y' = relu(scale * Y + shift) per output channel, and the
    per-channel sum / sum of squares of the stored y' (every member optional)."""
    _fields_ = [("scale", ctypes.c_void_p), ("shift", ctypes.c_void_p), ("relu", ctypes.c_int),
                ("sum", ctypes.c_void_p), ("sumsq", ctypes.c_void_p)]


def epilogue(scale=None, shift=None, relu=False, stat_sum=None, stat_sumsq=None) -> Epilogue:
    """An Epilogue over float32 device tensors of O values (or None); the tensors must outlive the call."""
    e = Epilogue(_ptr(scale), _ptr(shift), int(bool(relu)), _ptr(stat_sum), _ptr(stat_sumsq))
    e.tensors = [("epi.scale", scale), ("epi.shift", shift), ("epi.sum", stat_sum), ("epi.sumsq", stat_sumsq)]
    return e


def conv_desc(n, c, h, w, o, kh, kw, stride=1, pad=0, dtype=QL_BF16, neuron=QL_NEURON_QUADRA,
              groups=1) -> ConvDesc:
    """groups = c (with o == c) makes the layer depthwise: weights (c, kh, kw, 1)."""
    sh, sw = (stride, stride) if isinstance(stride, int) else stride
    ph, pw = (pad, pad) if isinstance(pad, int) else pad
    return ConvDesc(n, c, h, w, o, kh, kw, sh, sw, ph, pw, dtype, neuron, groups)


def linear_desc(batch, inp, out, dtype=QL_BF16, neuron=QL_NEURON_QUADRA) -> LinearDesc:
    return LinearDesc(batch, inp, out, dtype, neuron)


_lib = None
_vp = ctypes.c_void_p
_sz = ctypes.c_size_t


def lib():
    """The loaded C library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2204_01701_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    cd, ld = ctypes.POINTER(ConvDesc), ctypes.POINTER(LinearDesc)
    L.qlayer_status_string.argtypes = [ctypes.c_int]
    L.qlayer_status_string.restype = ctypes.c_char_p
    L.qlayer_version.restype = ctypes.c_int
    for name, d in (("conv2d_fwd", cd), ("conv2d_bwd_data", cd), ("conv2d_bwd_weight", cd),
                    ("linear_fwd", ld), ("linear_bwd", ld)):
        f = getattr(L, f"qlayer_{name}_workspace_size")
        f.argtypes = [d]
        f.restype = _sz
    L.qlayer_conv2d_fwd.argtypes = [cd] + [_vp] * 10 + [_vp, _sz, _vp]
    L.qlayer_conv2d_bwd_data.argtypes = [cd] + [_vp] * 7 + [_vp, _sz, _vp]
    L.qlayer_conv2d_bwd_data_ex.argtypes = [cd] + [_vp] * 8 + [_vp, _sz, _vp]
    L.qlayer_conv2d_bwd_data_ex.restype = ctypes.c_int
    L.qlayer_conv2d_bwd_weight.argtypes = [cd] + [_vp] * 10 + [_vp, _sz, _vp]
    L.qlayer_conv2d_bwd_weight_noalloc.argtypes = [cd] + [_vp] * 10 + [_vp]
    L.qlayer_conv2d_bwd_weight_noalloc.restype = ctypes.c_int
    L.qlayer_linear_fwd.argtypes = [ld] + [_vp] * 10 + [_vp, _sz, _vp]
    L.qlayer_linear_bwd.argtypes = [ld] + [_vp] * 14 + [_vp, _sz, _vp]
    for name, d in (("conv2d_bwd_relu", cd), ("linear_bwd_relu", ld)):
        f = getattr(L, f"qlayer_{name}_workspace_size")
        f.argtypes = [d]
        f.restype = _sz
        getattr(L, f"qlayer_{name}").argtypes = [d] + [_vp] * 15 + [_vp, _sz, _vp]
        getattr(L, f"qlayer_{name}").restype = ctypes.c_int
    ep = ctypes.POINTER(Epilogue)
    for name, d in (("conv2d_fwd_ex", cd), ("linear_fwd_ex", ld)):
        f = getattr(L, f"qlayer_{name}_workspace_size")
        f.argtypes = [d, ep]
        f.restype = _sz
        getattr(L, f"qlayer_{name}").argtypes = [d] + [_vp] * 10 + [ep, _vp, _sz, _vp]
        getattr(L, f"qlayer_{name}").restype = ctypes.c_int
    for name in ("conv2d_fwd", "conv2d_bwd_data", "conv2d_bwd_weight", "linear_fwd", "linear_bwd"):
        getattr(L, f"qlayer_{name}").restype = ctypes.c_int
    # the network glue (include/qnet.h)
    sp = ctypes.POINTER(NetShape)
    L.qnet_bn_act_fwd.argtypes = [sp, ctypes.c_int, _vp, _vp, _vp, ctypes.c_float, _vp, sp, ctypes.c_int, _vp, _vp,
                                  _vp, _vp]
    L.qnet_bn_act_bwd_workspace_size.argtypes = [sp]
    L.qnet_bn_act_bwd_workspace_size.restype = _sz
    L.qnet_bn_act_bwd.argtypes = [sp, ctypes.c_int, _vp, _vp, ctypes.c_int, _vp, _vp, _vp, _vp, _vp, _sz, _vp]
    L.qnet_residual_bwd.argtypes = [sp, ctypes.c_int, _vp, _vp, sp, _vp, _vp]
    L.qnet_gap_fwd.argtypes = [sp, ctypes.c_int, _vp, _vp, _vp]
    L.qnet_gap_bwd.argtypes = [sp, ctypes.c_int, _vp, _vp, _vp]
    for name in ("bn_act_fwd", "bn_act_bwd", "residual_bwd", "gap_fwd", "gap_bwd"):
        getattr(L, f"qnet_{name}").restype = ctypes.c_int
    _lib = L
    return L


def qlayer_version() -> int:
    return lib().qlayer_version()


def qlayer_status_string(status: int) -> str:
    try:
        return lib().qlayer_status_string(int(status)).decode()
    except ImportError:
        return "unknown"


# --- marshalling -------------------------------------------------------------

def _ptr(t):
    """Device pointer of a tensor (None -> NULL).  Plain ints pass through (tests)."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not t.is_contiguous():
        raise ValueError("tensors passed to qlayer must be contiguous")
    return t.data_ptr()


def _device(*tensors):
    for t in tensors:
        if t is not None and not isinstance(t, int):
            return t.device
    return None


def _stream(stream, device):
    if stream is not None:
        return stream if isinstance(stream, int) else stream.cuda_stream
    if device is None or device.type != "cuda":
        return None
    import torch
    return torch.cuda.current_stream(device).cuda_stream


def _workspace(workspace, need, device, stream=None):
    """(pointer, bytes) of the workspace; allocates one with torch when none is given.

    The allocation is made on the current stream.  When the call runs on
    another stream, the block is recorded on that stream, so that the caching
    allocator does not hand it out again while the kernels there still use it;
    a raw stream handle (an int) cannot be recorded and needs an explicit
    workspace."""
    if workspace is not None:
        if isinstance(workspace, tuple):
            return workspace
        return workspace.data_ptr(), workspace.numel() * workspace.element_size()
    if need == 0:
        return None, 0
    import torch
    if isinstance(stream, int):
        raise ValueError("a raw stream handle needs an explicit workspace (the allocator cannot track its use)")
    ws = torch.empty(need, dtype=torch.uint8, device=device)
    if stream is not None and stream != torch.cuda.current_stream(device):
        ws.record_stream(stream)
    _workspace.keep = ws  # keep alive until the next allocation; the stream orders reuse
    return ws.data_ptr(), need


# --- host-side checks of tensor arguments -------------------------------------
# The C ABI sees bare pointers, so a tensor of the wrong size, dtype or device
# would make the kernels read or write out of bounds.  Every tensor argument is
# checked against the descriptor before the call: a CUDA tensor on the
# device of the others, with the element count and dtype its role requires.

def _act_dtype(code):
    import torch
    if code == QL_BF16:
        return torch.bfloat16
    if code == QL_F32:
        return torch.float32
    return None  # (the library rejects unknown dtypes itself)


def _expect(name, t, numel, dtype, device):
    if t is None or isinstance(t, int):
        return
    if t.device.type != "cuda":
        raise ValueError(f"{name}: a CUDA device tensor is required, got one on {t.device}")
    if device is not None and t.device != device:
        raise ValueError(f"{name}: on {t.device}, the other tensors on {device}")
    if t.numel() != numel:
        raise ValueError(f"{name}: {t.numel()} elements, the descriptor needs {numel}")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name}: dtype {t.dtype}, expected {dtype}")


def _conv_sizes(d):
    """Element counts of X, each W_t, the output-side maps, the biases."""
    dw = d.groups == d.c and d.c > 1
    nw = d.o * d.kh * d.kw * (1 if dw else d.c)
    return d.n * d.h * d.w * d.c, nw, d.n * d.ho * d.wo * d.o, d.o


def _linear_sizes(d):
    return d.batch * d.in_, d.out * d.in_, d.batch * d.out, d.out


def _check_args(sizes, dtype_code, device, act=(), weights=(), maps=(), vec32=(), w32=()):
    """act: (name, tensor) pairs shaped like X; weights like W_t; maps like Y;
    vec32: float32 vectors of O; w32: float32 tensors shaped like W_t."""
    nx, nw, ny, no = sizes
    import torch
    dt = _act_dtype(dtype_code)
    for n, t in act:
        _expect(n, t, nx, dt, device)
    for n, t in weights:
        _expect(n, t, nw, dt, device)
    for n, t in maps:
        _expect(n, t, ny, dt, device)
    for n, t in vec32:
        _expect(n, t, no, torch.float32, device)
    for n, t in w32:
        _expect(n, t, nw, torch.float32, device)


def _check(func, status):
    if status != 0:
        raise QLError(func, status)


# --- the C ABI, one Python function per entry point -------------------------

def qlayer_conv2d_fwd_workspace_size(desc: ConvDesc) -> int:
    return lib().qlayer_conv2d_fwd_workspace_size(ctypes.byref(desc))


def qlayer_conv2d_fwd(desc, x, wa, wb, wc, ba=None, bb=None, bc=None, y=None, ta=None, tb=None,
                      workspace=None, stream=None):
    dev = _device(x, wa)
    _check_args(_conv_sizes(desc), desc.dtype, dev, act=[("x", x)], weights=[("wa", wa), ("wb", wb), ("wc", wc)],
                maps=[("y", y), ("ta", ta), ("tb", tb)], vec32=[("ba", ba), ("bb", bb), ("bc", bc)])
    wp, wn = _workspace(workspace, qlayer_conv2d_fwd_workspace_size(desc), dev, stream)
    _check("qlayer_conv2d_fwd", lib().qlayer_conv2d_fwd(
        ctypes.byref(desc), _ptr(x), _ptr(wa), _ptr(wb), _ptr(wc), _ptr(ba), _ptr(bb), _ptr(bc),
        _ptr(y), _ptr(ta), _ptr(tb), wp, wn, _stream(stream, dev)))


def qlayer_conv2d_bwd_data_workspace_size(desc: ConvDesc) -> int:
    return lib().qlayer_conv2d_bwd_data_workspace_size(ctypes.byref(desc))


def qlayer_conv2d_bwd_data(desc, gy, ta, tb, wa, wb, wc, dx, workspace=None, stream=None):
    dev = _device(gy, wa)
    t2 = desc.neuron == QL_NEURON_T2  # (its `ta` carries X)
    _check_args(_conv_sizes(desc), desc.dtype, dev, act=[("dx", dx)] + ([("ta (X)", ta)] if t2 else []),
                weights=[("wa", wa), ("wb", wb), ("wc", wc)],
                maps=[("gy", gy), ("tb", tb)] + ([] if t2 else [("ta", ta)]))
    wp, wn = _workspace(workspace, qlayer_conv2d_bwd_data_workspace_size(desc), dev, stream)
    _check("qlayer_conv2d_bwd_data", lib().qlayer_conv2d_bwd_data(
        ctypes.byref(desc), _ptr(gy), _ptr(ta), _ptr(tb), _ptr(wa), _ptr(wb), _ptr(wc), _ptr(dx),
        wp, wn, _stream(stream, dev)))


def qlayer_conv2d_bwd_data_ex(desc, gy, ta, tb, x, wa, wb, wc, dx, workspace=None, stream=None):
    """qlayer_conv2d_bwd_data with the layer input X (T2&4 needs it; T2 may take it in place of `ta`)."""
    dev = _device(gy, wa)
    t2 = desc.neuron == QL_NEURON_T2
    _check_args(_conv_sizes(desc), desc.dtype, dev, act=[("dx", dx), ("x", x)] + ([("ta (X)", ta)] if t2 else []),
                weights=[("wa", wa), ("wb", wb), ("wc", wc)],
                maps=[("gy", gy), ("tb", tb)] + ([] if t2 else [("ta", ta)]))
    wp, wn = _workspace(workspace, qlayer_conv2d_bwd_data_workspace_size(desc), dev, stream)
    _check("qlayer_conv2d_bwd_data_ex", lib().qlayer_conv2d_bwd_data_ex(
        ctypes.byref(desc), _ptr(gy), _ptr(ta), _ptr(tb), _ptr(x), _ptr(wa), _ptr(wb), _ptr(wc), _ptr(dx),
        wp, wn, _stream(stream, dev)))


def qlayer_conv2d_bwd_weight_workspace_size(desc: ConvDesc) -> int:
    return lib().qlayer_conv2d_bwd_weight_workspace_size(ctypes.byref(desc))


def qlayer_conv2d_bwd_weight(desc, x, gy, ta, tb, dwa, dwb, dwc, dba=None, dbb=None, dbc=None,
                             workspace=None, stream=None):
    dev = _device(x, gy)
    _check_args(_conv_sizes(desc), desc.dtype, dev, act=[("x", x)], maps=[("gy", gy), ("ta", ta), ("tb", tb)],
                w32=[("dwa", dwa), ("dwb", dwb), ("dwc", dwc)], vec32=[("dba", dba), ("dbb", dbb), ("dbc", dbc)])
    wp, wn = _workspace(workspace, qlayer_conv2d_bwd_weight_workspace_size(desc), dev, stream)
    _check("qlayer_conv2d_bwd_weight", lib().qlayer_conv2d_bwd_weight(
        ctypes.byref(desc), _ptr(x), _ptr(gy), _ptr(ta), _ptr(tb), _ptr(dwa), _ptr(dwb), _ptr(dwc),
        _ptr(dba), _ptr(dbb), _ptr(dbc), wp, wn, _stream(stream, dev)))


NOALLOC_SCRATCH_BYTES = 32 << 20  # QLAYER_NOALLOC_SCRATCH_BYTES of qlayer.h


def qlayer_conv2d_bwd_weight_noalloc(desc, x, gy, ta, tb, dwa, dwb, dwc, dba=None, dbb=None, dbc=None,
                                     stream=None):
    """qlayer_conv2d_bwd_weight with the library's own scratch array in place of a
    workspace: allocates nothing (for graph capture and other callers that cannot)."""
    dev = _device(x, gy)
    _check_args(_conv_sizes(desc), desc.dtype, dev, act=[("x", x)], maps=[("gy", gy), ("ta", ta), ("tb", tb)],
                w32=[("dwa", dwa), ("dwb", dwb), ("dwc", dwc)], vec32=[("dba", dba), ("dbb", dbb), ("dbc", dbc)])
    _check("qlayer_conv2d_bwd_weight_noalloc", lib().qlayer_conv2d_bwd_weight_noalloc(
        ctypes.byref(desc), _ptr(x), _ptr(gy), _ptr(ta), _ptr(tb), _ptr(dwa), _ptr(dwb), _ptr(dwc),
        _ptr(dba), _ptr(dbb), _ptr(dbc), _stream(stream, dev)))


def qlayer_linear_fwd_workspace_size(desc: LinearDesc) -> int:
    return lib().qlayer_linear_fwd_workspace_size(ctypes.byref(desc))


def qlayer_linear_fwd(desc, x, wa, wb, wc, ba=None, bb=None, bc=None, y=None, ta=None, tb=None,
                      workspace=None, stream=None):
    dev = _device(x, wa)
    _check_args(_linear_sizes(desc), desc.dtype, dev, act=[("x", x)], weights=[("wa", wa), ("wb", wb), ("wc", wc)],
                maps=[("y", y), ("ta", ta), ("tb", tb)], vec32=[("ba", ba), ("bb", bb), ("bc", bc)])
    wp, wn = _workspace(workspace, qlayer_linear_fwd_workspace_size(desc), dev, stream)
    _check("qlayer_linear_fwd", lib().qlayer_linear_fwd(
        ctypes.byref(desc), _ptr(x), _ptr(wa), _ptr(wb), _ptr(wc), _ptr(ba), _ptr(bb), _ptr(bc),
        _ptr(y), _ptr(ta), _ptr(tb), wp, wn, _stream(stream, dev)))


def _epi_ref(epi):
    return ctypes.byref(epi) if epi is not None else None


def qlayer_conv2d_fwd_ex_workspace_size(desc: ConvDesc, epi=None) -> int:
    return lib().qlayer_conv2d_fwd_ex_workspace_size(ctypes.byref(desc), _epi_ref(epi))


def qlayer_conv2d_fwd_ex(desc, x, wa, wb, wc, ba=None, bb=None, bc=None, y=None, ta=None, tb=None, epi=None,
                         workspace=None, stream=None):
    """qlayer_conv2d_fwd with a fused epilogue (an Epilogue, see epilogue())."""
    dev = _device(x, wa)
    _check_args(_conv_sizes(desc), desc.dtype, dev, act=[("x", x)], weights=[("wa", wa), ("wb", wb), ("wc", wc)],
                maps=[("y", y), ("ta", ta), ("tb", tb)],
                vec32=[("ba", ba), ("bb", bb), ("bc", bc)] + list(getattr(epi, "tensors", [])))
    wp, wn = _workspace(workspace, qlayer_conv2d_fwd_ex_workspace_size(desc, epi), dev, stream)
    _check("qlayer_conv2d_fwd_ex", lib().qlayer_conv2d_fwd_ex(
        ctypes.byref(desc), _ptr(x), _ptr(wa), _ptr(wb), _ptr(wc), _ptr(ba), _ptr(bb), _ptr(bc),
        _ptr(y), _ptr(ta), _ptr(tb), _epi_ref(epi), wp, wn, _stream(stream, dev)))


def qlayer_linear_fwd_ex_workspace_size(desc: LinearDesc, epi=None) -> int:
    return lib().qlayer_linear_fwd_ex_workspace_size(ctypes.byref(desc), _epi_ref(epi))


def qlayer_linear_fwd_ex(desc, x, wa, wb, wc, ba=None, bb=None, bc=None, y=None, ta=None, tb=None, epi=None,
                         workspace=None, stream=None):
    """qlayer_linear_fwd with a fused epilogue (an Epilogue, see epilogue())."""
    dev = _device(x, wa)
    _check_args(_linear_sizes(desc), desc.dtype, dev, act=[("x", x)], weights=[("wa", wa), ("wb", wb), ("wc", wc)],
                maps=[("y", y), ("ta", ta), ("tb", tb)],
                vec32=[("ba", ba), ("bb", bb), ("bc", bc)] + list(getattr(epi, "tensors", [])))
    wp, wn = _workspace(workspace, qlayer_linear_fwd_ex_workspace_size(desc, epi), dev, stream)
    _check("qlayer_linear_fwd_ex", lib().qlayer_linear_fwd_ex(
        ctypes.byref(desc), _ptr(x), _ptr(wa), _ptr(wb), _ptr(wc), _ptr(ba), _ptr(bb), _ptr(bc),
        _ptr(y), _ptr(ta), _ptr(tb), _epi_ref(epi), wp, wn, _stream(stream, dev)))


def qlayer_linear_bwd_workspace_size(desc: LinearDesc) -> int:
    return lib().qlayer_linear_bwd_workspace_size(ctypes.byref(desc))


def qlayer_linear_bwd(desc, x, gy, ta, tb, wa, wb, wc, dx=None, dwa=None, dwb=None, dwc=None,
                      dba=None, dbb=None, dbc=None, workspace=None, stream=None):
    dev = _device(x, gy)
    _check_args(_linear_sizes(desc), desc.dtype, dev, act=[("x", x), ("dx", dx)],
                weights=[("wa", wa), ("wb", wb), ("wc", wc)], maps=[("gy", gy), ("ta", ta), ("tb", tb)],
                w32=[("dwa", dwa), ("dwb", dwb), ("dwc", dwc)], vec32=[("dba", dba), ("dbb", dbb), ("dbc", dbc)])
    wp, wn = _workspace(workspace, qlayer_linear_bwd_workspace_size(desc), dev, stream)
    _check("qlayer_linear_bwd", lib().qlayer_linear_bwd(
        ctypes.byref(desc), _ptr(x), _ptr(gy), _ptr(ta), _ptr(tb), _ptr(wa), _ptr(wb), _ptr(wc),
        _ptr(dx), _ptr(dwa), _ptr(dwb), _ptr(dwc), _ptr(dba), _ptr(dbb), _ptr(dbc),
        wp, wn, _stream(stream, dev)))


def _bwd_relu(name, sizes, wsize, desc, x, gy, y_out, ta, tb, wa, wb, wc, dx, dwa, dwb, dwc, dba, dbb, dbc,
              workspace, stream):
    dev = _device(x, gy)
    _check_args(sizes, desc.dtype, dev, act=[("x", x), ("dx", dx)], weights=[("wa", wa), ("wb", wb), ("wc", wc)],
                maps=[("gy", gy), ("y_out", y_out), ("ta", ta), ("tb", tb)],
                w32=[("dwa", dwa), ("dwb", dwb), ("dwc", dwc)], vec32=[("dba", dba), ("dbb", dbb), ("dbc", dbc)])
    wp, wn = _workspace(workspace, wsize(desc), dev, stream)
    _check(name, getattr(lib(), name)(
        ctypes.byref(desc), _ptr(x), _ptr(gy), _ptr(y_out), _ptr(ta), _ptr(tb), _ptr(wa), _ptr(wb), _ptr(wc),
        _ptr(dx), _ptr(dwa), _ptr(dwb), _ptr(dwc), _ptr(dba), _ptr(dbb), _ptr(dbc), wp, wn, _stream(stream, dev)))


def qlayer_conv2d_bwd_relu_workspace_size(desc: ConvDesc) -> int:
    return lib().qlayer_conv2d_bwd_relu_workspace_size(ctypes.byref(desc))


def qlayer_conv2d_bwd_relu(desc, x, gy, y_out, ta, tb, wa, wb, wc, dx=None, dwa=None, dwb=None, dwc=None,
                           dba=None, dbb=None, dbc=None, workspace=None, stream=None):
    """The layer's backward behind the fused ReLU: G = gy o [y_out > 0], then dX and/or dW_t, db_t from G."""
    _bwd_relu("qlayer_conv2d_bwd_relu", _conv_sizes(desc), qlayer_conv2d_bwd_relu_workspace_size, desc, x, gy, y_out,
              ta, tb, wa, wb, wc, dx, dwa, dwb, dwc, dba, dbb, dbc, workspace, stream)


def qlayer_linear_bwd_relu_workspace_size(desc: LinearDesc) -> int:
    return lib().qlayer_linear_bwd_relu_workspace_size(ctypes.byref(desc))


def qlayer_linear_bwd_relu(desc, x, gy, y_out, ta, tb, wa, wb, wc, dx=None, dwa=None, dwb=None, dwc=None,
                           dba=None, dbb=None, dbc=None, workspace=None, stream=None):
    """The dense layer's backward behind the fused ReLU (as qlayer_conv2d_bwd_relu)."""
    _bwd_relu("qlayer_linear_bwd_relu", _linear_sizes(desc), qlayer_linear_bwd_relu_workspace_size, desc, x, gy,
              y_out, ta, tb, wa, wb, wc, dx, dwa, dwb, dwc, dba, dbb, dbc, workspace, stream)


# --- the network glue (include/qnet.h) ----------------------------------------

def _net_dtype(t):
    import torch
    return QL_BF16 if t.dtype == torch.bfloat16 else QL_F32


def _net_expect(name, t, shape, dtype, device):
    _expect(name, t, int(shape[0]) * int(shape[1]) * int(shape[2]) * int(shape[3]) if len(shape) == 4
            else int(shape[0]) * int(shape[1]), dtype, device)


def qnet_bn_act_fwd(y, ssum, ssq, out, mean, rstd, eps=1e-5, res=None, relu=True, stream=None):
    """out = relu((y - mean) rstd + shortcut(res)); y, out, res NHWC device tensors."""
    import torch
    dev = y.device
    s = net_shape(y)
    dt = _net_dtype(y)
    _net_expect("out", out, y.shape, y.dtype, dev)
    for n, t in (("sum", ssum), ("sumsq", ssq), ("mean", mean), ("rstd", rstd)):
        _expect(n, t, s.c, torch.float32, dev)
    rs = net_shape(res) if res is not None else None
    if res is not None:
        _expect("res", res, rs.n * rs.h * rs.w * rs.c, y.dtype, dev)
    _check("qnet_bn_act_fwd", lib().qnet_bn_act_fwd(
        ctypes.byref(s), dt, _ptr(y), _ptr(ssum), _ptr(ssq), ctypes.c_float(eps), _ptr(res),
        ctypes.byref(rs) if rs is not None else None, int(bool(relu)), _ptr(out), _ptr(mean), _ptr(rstd),
        _stream(stream, dev)))


def qnet_bn_act_bwd_workspace_size(shape) -> int:
    return lib().qnet_bn_act_bwd_workspace_size(ctypes.byref(net_shape(shape)))


def qnet_bn_act_bwd(dout, out, y, mean, rstd, dy, relu=True, workspace=None, stream=None):
    """dy = the gradient at y of out = relu(bn(y) [+ r]) given dout."""
    import torch
    dev = y.device
    s = net_shape(y)
    for n, t in (("dout", dout), ("out", out), ("dy", dy)):
        _net_expect(n, t, y.shape, y.dtype, dev)
    for n, t in (("mean", mean), ("rstd", rstd)):
        _expect(n, t, s.c, torch.float32, dev)
    wp, wn = _workspace(workspace, qnet_bn_act_bwd_workspace_size(y.shape), dev, stream)
    _check("qnet_bn_act_bwd", lib().qnet_bn_act_bwd(
        ctypes.byref(s), _net_dtype(y), _ptr(dout), _ptr(out), int(bool(relu)), _ptr(y), _ptr(mean), _ptr(rstd),
        _ptr(dy), wp, wn, _stream(stream, dev)))


def qnet_residual_bwd(dout, out, dx, stream=None):
    """dx (the block input's gradient) += the shortcut's share of dout [out > 0]."""
    dev = dx.device
    _net_expect("out", out, dout.shape, dout.dtype, dev)
    _check("qnet_residual_bwd", lib().qnet_residual_bwd(
        ctypes.byref(net_shape(dout)), _net_dtype(dout), _ptr(dout), _ptr(out), ctypes.byref(net_shape(dx)),
        _ptr(dx), _stream(stream, dev)))


def qnet_gap_fwd(x, y, stream=None):
    dev = x.device
    _expect("y", y, x.shape[0] * x.shape[3], x.dtype, dev)
    _check("qnet_gap_fwd", lib().qnet_gap_fwd(ctypes.byref(net_shape(x)), _net_dtype(x), _ptr(x), _ptr(y),
                                              _stream(stream, dev)))


def qnet_gap_bwd(dy, dx, stream=None):
    dev = dx.device
    _expect("dy", dy, dx.shape[0] * dx.shape[3], dx.dtype, dev)
    _check("qnet_gap_bwd", lib().qnet_gap_bwd(ctypes.byref(net_shape(dx)), _net_dtype(dx), _ptr(dy), _ptr(dx),
                                              _stream(stream, dev)))
