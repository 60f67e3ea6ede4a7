"""fp64 CPU oracle of the QuadraLib quadratic neuron -- TEST INFRASTRUCTURE ONLY.

Only the test-suite, the CPU-baseline leg of ``bench.py`` and
``__graft_entry__.smoke()`` may import this package.  The product library
(``paper_2204_01701_amd``) never imports it, and this package imports
nothing from the product.

The arithmetic lives in ``qlayer_oracle.c`` (plain C, fp64, OpenMP over
independent output elements); this module only compiles it and marshals
numpy arrays through ctypes.  Every array is float64, C-contiguous, in the
logical PyTorch layouts: activations N x C x H x W, conv weights
O x C x KH x KW, FC inputs B x I, FC weights O x I.

Definitions followed (arXiv 2204.01701):
  * forward  -- section 3.1, equation eq:2ndneuron3, Y = (W_a X) o (W_b X) + W_c X,
    each term an ordinary first-order neuron with its own bias (section 3.2 P4);
  * backward -- section 4.3, equations eq:AD / eq:SD: G_a = G o T_b, G_b = G o T_a,
    G_c = G, then the ordinary first-order gradients of each term.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "qlayer_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

_D = ctypes.POINTER(ctypes.c_double)
_L = ctypes.POINTER(ctypes.c_longlong)
_I = ctypes.c_int


def build(force: bool = True, out: str | None = None, extra_flags: tuple = ()) -> str:
    """Compile the oracle with gcc (fp64, OpenMP, no FMA contraction).  `out`
    and `extra_flags` build another copy (e.g. with sanitizers) elsewhere."""
    path = out or _LIB_PATH
    if force or not os.path.exists(path):
        tmp = path + ".tmp"
        cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-ffp-contract=off", *extra_flags,
               "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, path)
    return path


def _load():
    global _lib
    if _lib is not None:
        return _lib
    # ORACLE_LIB: a separately built copy of the same source (the sanitizer run of the test-suite)
    other = os.environ.get("ORACLE_LIB")
    if other:
        lib = ctypes.CDLL(other)
    else:
        if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
            build(force=True)
        lib = ctypes.CDLL(_LIB_PATH)
    conv_geom = [_I] * 11
    w6 = [_D] * 6
    lib.oracle_conv2d_fwd.argtypes = conv_geom + [_D] + w6 + [_D, _D, _D]
    lib.oracle_conv2d_bwd.argtypes = conv_geom + [_D] + w6 + [_D] + [_D] * 7
    lib.oracle_conv2d_fwd_at.argtypes = conv_geom + [_D] + w6 + [ctypes.c_longlong, _L, _D, _D, _D]
    lib.oracle_conv2d_dx_at.argtypes = conv_geom + [_D] + w6 + [_D, ctypes.c_longlong, _L, _D]
    lib.oracle_conv2d_dx_pixels.argtypes = conv_geom + [_D] + w6 + [_D, ctypes.c_longlong, _L, _D]
    lib.oracle_conv2d_dw_channel.argtypes = conv_geom + [_D] + w6 + [_D, _I] + [_D] * 6
    lib.oracle_conv2d_fwd_neuron.argtypes = [_I] + conv_geom + [_D] + w6 + [_D, _D, _D]
    lib.oracle_conv2d_bwd_neuron.argtypes = [_I] + conv_geom + [_D] + w6 + [_D] + [_D] * 7
    dw_geom = [_I] * 11  # neuron, N, C, H, W, KH, KW, sh, sw, ph, pw
    lib.oracle_dwconv2d_fwd.argtypes = dw_geom + [_D] + w6 + [_D, _D, _D]
    lib.oracle_dwconv2d_bwd.argtypes = dw_geom + [_D] + w6 + [_D] + [_D] * 7
    lib.oracle_epilogue.argtypes = [_I, _I, ctypes.c_longlong, _D, _D, _D, _I, _D, _D, _D]
    lib.oracle_conv2d_out_size.argtypes = [_I] * 4
    lib.oracle_conv2d_out_size.restype = _I
    fc_geom = [_I] * 3
    lib.oracle_linear_fwd.argtypes = fc_geom + [_D] + w6 + [_D, _D, _D]
    lib.oracle_linear_bwd.argtypes = fc_geom + [_D] + w6 + [_D] + [_D] * 7
    lib.oracle_linear_fwd_at.argtypes = fc_geom + [_D] + w6 + [ctypes.c_longlong, _L, _D, _D, _D]
    lib.oracle_linear_dx_rows.argtypes = fc_geom + [_D] + w6 + [_D, ctypes.c_longlong, _L, _D]
    lib.oracle_linear_dw_row.argtypes = fc_geom + [_D] + w6 + [_D, _I] + [_D] * 6
    for f in ("oracle_dwconv2d_fwd", "oracle_dwconv2d_bwd", "oracle_conv2d_fwd_neuron", "oracle_conv2d_bwd_neuron", "oracle_conv2d_fwd", "oracle_conv2d_bwd", "oracle_conv2d_fwd_at", "oracle_conv2d_dx_at", "oracle_conv2d_dx_pixels",
              "oracle_conv2d_dw_channel", "oracle_linear_fwd", "oracle_linear_bwd",
              "oracle_linear_fwd_at", "oracle_linear_dx_rows", "oracle_linear_dw_row"):
        getattr(lib, f).restype = None
    _lib = lib
    return lib


def _f64(a):
    if a is None:
        return None
    a = np.ascontiguousarray(np.asarray(a, dtype=np.float64))
    return a


def _p(a):
    if a is None:
        return ctypes.cast(None, _D)
    return a.ctypes.data_as(_D)


def _pl(a):
    return a.ctypes.data_as(_L)


def _pair(v):
    return (v, v) if isinstance(v, int) else tuple(v)


def out_size(n: int, k: int, s: int, p: int) -> int:
    """Output extent of a zero-padded cross-correlation with floor rounding."""
    return _load().oracle_conv2d_out_size(n, k, s, p)


def _conv_geom(x, w, stride, pad):
    N, C, H, W = x.shape
    O, C2, KH, KW = w.shape
    assert C == C2, "weight input channels must match X"
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    return (N, C, H, W, O, KH, KW, sh, sw, ph, pw)


def conv2d_fwd(x, wa, wb, wc, ba=None, bb=None, bc=None, stride=1, pad=0):
    """Returns (Y, T_a, T_b), each N x O x Ho x Wo float64."""
    lib = _load()
    x, wa, wb, wc, ba, bb, bc = map(_f64, (x, wa, wb, wc, ba, bb, bc))
    g = _conv_geom(x, wa, stride, pad)
    N, O = g[0], g[4]
    Ho, Wo = out_size(g[2], g[5], g[7], g[9]), out_size(g[3], g[6], g[8], g[10])
    y = np.empty((N, O, Ho, Wo))
    ta = np.empty_like(y)
    tb = np.empty_like(y)
    lib.oracle_conv2d_fwd(*g, _p(x), _p(wa), _p(wb), _p(wc), _p(ba), _p(bb), _p(bc), _p(y), _p(ta), _p(tb))
    return y, ta, tb


def conv2d_bwd(x, wa, wb, wc, ba, bb, bc, gy, stride=1, pad=0):
    """Returns dict dx, dwa, dwb, dwc, dba, dbb, dbc (float64)."""
    lib = _load()
    x, wa, wb, wc, ba, bb, bc, gy = map(_f64, (x, wa, wb, wc, ba, bb, bc, gy))
    g = _conv_geom(x, wa, stride, pad)
    O = g[4]
    out = {"dx": np.empty_like(x), "dwa": np.empty_like(wa), "dwb": np.empty_like(wa),
           "dwc": np.empty_like(wa), "dba": np.empty(O), "dbb": np.empty(O), "dbc": np.empty(O)}
    lib.oracle_conv2d_bwd(*g, _p(x), _p(wa), _p(wb), _p(wc), _p(ba), _p(bb), _p(bc), _p(gy),
                          *[_p(out[k]) for k in ("dx", "dwa", "dwb", "dwc", "dba", "dbb", "dbc")])
    return out


def conv2d_fwd_at(x, wa, wb, wc, ba, bb, bc, idx, stride=1, pad=0):
    """Y, T_a, T_b at positions idx (k x 4 array of (n, o, i, j))."""
    lib = _load()
    x, wa, wb, wc, ba, bb, bc = map(_f64, (x, wa, wb, wc, ba, bb, bc))
    g = _conv_geom(x, wa, stride, pad)
    idx = np.ascontiguousarray(np.asarray(idx, dtype=np.int64).reshape(-1, 4))
    k = idx.shape[0]
    y, ta, tb = np.empty(k), np.empty(k), np.empty(k)
    lib.oracle_conv2d_fwd_at(*g, _p(x), _p(wa), _p(wb), _p(wc), _p(ba), _p(bb), _p(bc), k, _pl(idx),
                             _p(y), _p(ta), _p(tb))
    return y, ta, tb


def conv2d_dx_at(x, wa, wb, wc, ba, bb, bc, gy, idx, stride=1, pad=0):
    """dX at positions idx (k x 4 array of (n, c, h, w))."""
    lib = _load()
    x, wa, wb, wc, ba, bb, bc, gy = map(_f64, (x, wa, wb, wc, ba, bb, bc, gy))
    g = _conv_geom(x, wa, stride, pad)
    idx = np.ascontiguousarray(np.asarray(idx, dtype=np.int64).reshape(-1, 4))
    k = idx.shape[0]
    dx = np.empty(k)
    lib.oracle_conv2d_dx_at(*g, _p(x), _p(wa), _p(wb), _p(wc), _p(ba), _p(bb), _p(bc), _p(gy), k,
                            _pl(idx), _p(dx))
    return dx


def conv2d_dx_pixels(x, wa, wb, wc, ba, bb, bc, gy, pix, stride=1, pad=0):
    """dX at every input channel of the input pixels pix (k x 3 array of (n, h, w)): k x C."""
    lib = _load()
    x, wa, wb, wc, ba, bb, bc, gy = map(_f64, (x, wa, wb, wc, ba, bb, bc, gy))
    g = _conv_geom(x, wa, stride, pad)
    pix = np.ascontiguousarray(np.asarray(pix, dtype=np.int64).reshape(-1, 3))
    k = pix.shape[0]
    dx = np.empty((k, x.shape[1]))
    lib.oracle_conv2d_dx_pixels(*g, _p(x), _p(wa), _p(wb), _p(wc), _p(ba), _p(bb), _p(bc), _p(gy), k,
                                _pl(pix), _p(dx))
    return dx


def conv2d_dw_channel(x, wa, wb, wc, ba, bb, bc, gy, o, stride=1, pad=0):
    """Weight gradients dW_t[o] (C x KH x KW each) and bias gradients db_t[o] of one channel."""
    lib = _load()
    x, wa, wb, wc, ba, bb, bc, gy = map(_f64, (x, wa, wb, wc, ba, bb, bc, gy))
    g = _conv_geom(x, wa, stride, pad)
    shp = wa.shape[1:]
    out = {"dwa": np.empty(shp), "dwb": np.empty(shp), "dwc": np.empty(shp),
           "dba": np.empty(1), "dbb": np.empty(1), "dbc": np.empty(1)}
    lib.oracle_conv2d_dw_channel(*g, _p(x), _p(wa), _p(wb), _p(wc), _p(ba), _p(bb), _p(bc), _p(gy),
                                 int(o), *[_p(out[k]) for k in ("dwa", "dwb", "dwc", "dba", "dbb", "dbc")])
    return out


def linear_fwd(x, wa, wb, wc, ba=None, bb=None, bc=None):
    """Returns (Y, T_a, T_b), each B x O float64."""
    lib = _load()
    x, wa, wb, wc, ba, bb, bc = map(_f64, (x, wa, wb, wc, ba, bb, bc))
    B, I = x.shape
    O = wa.shape[0]
    y, ta, tb = np.empty((B, O)), np.empty((B, O)), np.empty((B, O))
    lib.oracle_linear_fwd(B, I, O, _p(x), _p(wa), _p(wb), _p(wc), _p(ba), _p(bb), _p(bc),
                          _p(y), _p(ta), _p(tb))
    return y, ta, tb


def linear_bwd(x, wa, wb, wc, ba, bb, bc, gy):
    lib = _load()
    x, wa, wb, wc, ba, bb, bc, gy = map(_f64, (x, wa, wb, wc, ba, bb, bc, gy))
    B, I = x.shape
    O = wa.shape[0]
    out = {"dx": np.empty_like(x), "dwa": np.empty_like(wa), "dwb": np.empty_like(wa),
           "dwc": np.empty_like(wa), "dba": np.empty(O), "dbb": np.empty(O), "dbc": np.empty(O)}
    lib.oracle_linear_bwd(B, I, O, _p(x), _p(wa), _p(wb), _p(wc), _p(ba), _p(bb), _p(bc), _p(gy),
                          *[_p(out[k]) for k in ("dx", "dwa", "dwb", "dwc", "dba", "dbb", "dbc")])
    return out


def linear_fwd_at(x, wa, wb, wc, ba, bb, bc, idx):
    lib = _load()
    x, wa, wb, wc, ba, bb, bc = map(_f64, (x, wa, wb, wc, ba, bb, bc))
    B, I = x.shape
    O = wa.shape[0]
    idx = np.ascontiguousarray(np.asarray(idx, dtype=np.int64).reshape(-1, 2))
    k = idx.shape[0]
    y, ta, tb = np.empty(k), np.empty(k), np.empty(k)
    lib.oracle_linear_fwd_at(B, I, O, _p(x), _p(wa), _p(wb), _p(wc), _p(ba), _p(bb), _p(bc), k,
                             _pl(idx), _p(y), _p(ta), _p(tb))
    return y, ta, tb


def linear_dx_rows(x, wa, wb, wc, ba, bb, bc, gy, rows):
    lib = _load()
    x, wa, wb, wc, ba, bb, bc, gy = map(_f64, (x, wa, wb, wc, ba, bb, bc, gy))
    B, I = x.shape
    O = wa.shape[0]
    rows = np.ascontiguousarray(np.asarray(rows, dtype=np.int64).reshape(-1))
    dx = np.empty((rows.shape[0], I))
    lib.oracle_linear_dx_rows(B, I, O, _p(x), _p(wa), _p(wb), _p(wc), _p(ba), _p(bb), _p(bc), _p(gy),
                              rows.shape[0], _pl(rows), _p(dx))
    return dx


def linear_dw_row(x, wa, wb, wc, ba, bb, bc, gy, o):
    lib = _load()
    x, wa, wb, wc, ba, bb, bc, gy = map(_f64, (x, wa, wb, wc, ba, bb, bc, gy))
    B, I = x.shape
    O = wa.shape[0]
    out = {"dwa": np.empty(I), "dwb": np.empty(I), "dwc": np.empty(I),
           "dba": np.empty(1), "dbb": np.empty(1), "dbc": np.empty(1)}
    lib.oracle_linear_dw_row(B, I, O, _p(x), _p(wa), _p(wb), _p(wc), _p(ba), _p(bb), _p(bc), _p(gy),
                             int(o), *[_p(out[k]) for k in ("dwa", "dwb", "dwc", "dba", "dbb", "dbc")])
    return out


# Neuron types (the proposed one and the earlier designs of Table 1 / Table 3).
NEURON_QUADRA, NEURON_T4, NEURON_T4_IDENTITY, NEURON_T3, NEURON_T2, NEURON_T24 = 0, 1, 2, 3, 4, 5
NEURON_TERMS = {0: 3, 1: 2, 2: 2, 3: 1, 4: 1, 5: 3}  # first-order terms (weights) per type


def conv2d_fwd_neuron(neuron, x, wa, wb=None, wc=None, ba=None, bb=None, bc=None, stride=1, pad=0):
    """Forward of neuron type `neuron`: returns (Y, T_a, T_b), N x O x Ho x Wo
    (T_b is zeros for the one-term types, T_a is W_a*(X o X) + b_a for T2;
    T2&4 = T_a o T_b + W_c*(X o X) + b_c)."""
    lib = _load()
    x, wa, wb, wc, ba, bb, bc = map(_f64, (x, wa, wb, wc, ba, bb, bc))
    g = _conv_geom(x, wa, stride, pad)
    N, O = g[0], g[4]
    Ho, Wo = out_size(g[2], g[5], g[7], g[9]), out_size(g[3], g[6], g[8], g[10])
    if neuron == NEURON_T4_IDENTITY:
        assert g[1] == O and Ho == g[2] and Wo == g[3], "the identity shortcut needs C == O and an unchanged map"
    y, ta, tb = np.empty((N, O, Ho, Wo)), np.empty((N, O, Ho, Wo)), np.empty((N, O, Ho, Wo))
    lib.oracle_conv2d_fwd_neuron(int(neuron), *g, _p(x), _p(wa), _p(wb), _p(wc), _p(ba), _p(bb), _p(bc),
                                 _p(y), _p(ta), _p(tb))
    return y, ta, tb


def conv2d_bwd_neuron(neuron, x, wa, wb, wc, ba, bb, bc, gy, stride=1, pad=0):
    """Backward of neuron type `neuron`: dict dx and dw*/db* of the terms it has."""
    lib = _load()
    x, wa, wb, wc, ba, bb, bc, gy = map(_f64, (x, wa, wb, wc, ba, bb, bc, gy))
    g = _conv_geom(x, wa, stride, pad)
    O = g[4]
    nt = NEURON_TERMS[int(neuron)]
    keys = [("dwa", "dba"), ("dwb", "dbb"), ("dwc", "dbc")][:nt]
    out = {"dx": np.empty_like(x)}
    for kw, kb in keys:
        out[kw] = np.empty_like(wa)
        out[kb] = np.empty(O)
    lib.oracle_conv2d_bwd_neuron(int(neuron), *g, _p(x), _p(wa), _p(wb), _p(wc), _p(ba), _p(bb), _p(bc), _p(gy),
                                 *[_p(out.get(k)) for k in ("dx", "dwa", "dwb", "dwc", "dba", "dbb", "dbc")])
    return out


def linear_fwd_neuron(neuron, x, wa, wb=None, wc=None, ba=None, bb=None, bc=None):
    """Fully-connected layer of neuron type `neuron` (the 1x1 convolution of a 1x1 map): (Y, T_a, T_b), B x O."""
    B, I = np.shape(x)
    w4 = [None if w is None else np.asarray(w).reshape(np.shape(w)[0], I, 1, 1) for w in (wa, wb, wc)]
    y, ta, tb = conv2d_fwd_neuron(neuron, np.asarray(x).reshape(B, I, 1, 1), *w4, ba, bb, bc)
    return y.reshape(B, -1), ta.reshape(B, -1), tb.reshape(B, -1)


def linear_bwd_neuron(neuron, x, wa, wb, wc, ba, bb, bc, gy):
    B, I = np.shape(x)
    O = np.shape(wa)[0]
    w4 = [None if w is None else np.asarray(w).reshape(O, I, 1, 1) for w in (wa, wb, wc)]
    out = conv2d_bwd_neuron(neuron, np.asarray(x).reshape(B, I, 1, 1), *w4, ba, bb, bc,
                            np.asarray(gy).reshape(B, O, 1, 1))
    return {k: (v.reshape(B, I) if k == "dx" else (v.reshape(O, I) if k.startswith("dw") else v))
            for k, v in out.items()}


def _dw_geom(neuron, x, w, stride, pad):
    assert int(neuron) in (0, 1, 2, 3, 4), "the depthwise oracle covers the proposed neuron, T4, T4+identity, T3, T2"
    N, C, H, W = x.shape
    C2, one, KH, KW = w.shape
    assert C2 == C and one == 1, "depthwise weights are C x 1 x KH x KW"
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    return (int(neuron), N, C, H, W, KH, KW, sh, sw, ph, pw)


def dwconv2d_fwd(neuron, x, wa, wb=None, wc=None, ba=None, bb=None, bc=None, stride=1, pad=0):
    """Depthwise quadratic convolution (groups = C), weights C x 1 x KH x KW: (Y, T_a, T_b), N x C x Ho x Wo."""
    lib = _load()
    x, wa, wb, wc, ba, bb, bc = map(_f64, (x, wa, wb, wc, ba, bb, bc))
    g = _dw_geom(neuron, x, wa, stride, pad)
    N, C = g[1], g[2]
    Ho, Wo = out_size(g[3], g[5], g[7], g[9]), out_size(g[4], g[6], g[8], g[10])
    y, ta, tb = np.empty((N, C, Ho, Wo)), np.zeros((N, C, Ho, Wo)), np.zeros((N, C, Ho, Wo))
    lib.oracle_dwconv2d_fwd(*g, _p(x), _p(wa), _p(wb), _p(wc), _p(ba), _p(bb), _p(bc), _p(y), _p(ta), _p(tb))
    return y, ta, tb


def dwconv2d_bwd(neuron, x, wa, wb, wc, ba, bb, bc, gy, stride=1, pad=0):
    """Backward of the depthwise layer: dict dx and dw*/db* of the terms the type has."""
    lib = _load()
    x, wa, wb, wc, ba, bb, bc, gy = map(_f64, (x, wa, wb, wc, ba, bb, bc, gy))
    g = _dw_geom(neuron, x, wa, stride, pad)
    nt = NEURON_TERMS[int(neuron)]
    out = {"dx": np.empty_like(x)}
    for kw, kb in [("dwa", "dba"), ("dwb", "dbb"), ("dwc", "dbc")][:nt]:
        out[kw] = np.empty_like(wa)
        out[kb] = np.empty(g[2])
    lib.oracle_dwconv2d_bwd(*g, _p(x), _p(wa), _p(wb), _p(wc), _p(ba), _p(bb), _p(bc), _p(gy),
                            *[_p(out.get(k)) for k in ("dx", "dwa", "dwb", "dwc", "dba", "dbb", "dbc")])
    return out


def epilogue(y, scale=None, shift=None, relu=False):
    """Forward epilogue of a layer output y (N x O x H x W, or B x O for a dense
    layer): y' = relu(scale * y + shift) per channel, and the per-channel sum
    and sum of squares of y' over every other axis.  Returns (y', sum, sumsq)."""
    lib = _load()
    y = _f64(y)
    shp = y.shape
    N, O = shp[0], shp[1]
    P = int(np.prod(shp[2:])) if len(shp) > 2 else 1
    scale, shift = _f64(scale), _f64(shift)
    yo, s, s2 = np.empty_like(y), np.empty(O), np.empty(O)
    lib.oracle_epilogue(N, O, ctypes.c_longlong(P), _p(y), _p(scale), _p(shift), int(bool(relu)), _p(yo), _p(s),
                        _p(s2))
    return yo, s, s2


def num_threads() -> int:
    """Threads OpenMP will use for oracle calls in this process."""
    v = os.environ.get("OMP_NUM_THREADS")
    if v and v.isdigit():
        return int(v)
    return len(os.sched_getaffinity(0))
