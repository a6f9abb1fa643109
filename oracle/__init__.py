"""CPU oracle for the sparse 1x1 convolution -- test infrastructure only.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The GPU library never does, and this
package never imports the GPU library: the two share no code.

``spconv_ref`` evaluates the plain definition

    Y[n, r, p] = act( b[r] + sum_{stored (r, c)} W[r, c] * X[n, c, p] )

(paper Sec. 1 and Sec. 3.2 / Fig. 2: a 1x1 convolution in CHW layout is a
sparse-weight x dense-activation product; Sec. 3.2: 1xk output-channel blocks
share one pattern; Sec. 3.3: block-CSR weights) in double precision with the C
code in ``spconv_ref.c``, then rounds each element once, to nearest-even, to
the storage type.  It also returns the per-element error scale
S = sum |W[r, c] * X[n, c, p]| that the parity tolerance is stated in.

``dw3x3_ref`` and ``fused_ref`` evaluate the fused MobileNet block order
(depthwise 3x3, then the sparse 1x1 on its output; paper Sec. 2 and Sec.
3.3) the same way, in double.  ``conv3x3_hwc_ref`` (the dense first
convolution from an HWC image to CHW, Sec. 3.1), ``gap_ref`` (global average
pooling, Sec. 3.3) and ``mobilenet_v1_ref`` (the whole network, chaining
the double-precision stages and their error scales) complete a network.
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "spconv_ref.c")
_LIB = os.path.join(_HERE, "libspconv_ref.so")
_ACTS = {"none": 0, "relu": 1, "relu6": 2}
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (portable x86-64 code, OpenMP, no FP contraction)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fPIC", "-shared",
                               "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def load_library(path: str):
    """Open an oracle shared library (the default one, or a test's own build)."""
    lib = ctypes.CDLL(path)
    lib.spconv_ref_run.restype = ctypes.c_int
    lib.spconv_ref_run.argtypes = [
        ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
        ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_int64,
        ctypes.c_void_p, ctypes.c_void_p,
    ]
    lib.spconv_ref_run_blocked.restype = ctypes.c_int
    lib.spconv_ref_run_blocked.argtypes = [
        ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
        ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_int64,
        ctypes.c_void_p, ctypes.c_void_p,
    ]
    lib.spconv_ref_run_f64.restype = ctypes.c_int
    lib.spconv_ref_run_f64.argtypes = [
        ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
        ctypes.c_void_p, ctypes.c_void_p,
    ]
    lib.spconv_ref_dw3x3.restype = ctypes.c_int
    lib.spconv_ref_dw3x3.argtypes = [
        ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
    ]
    lib.spconv_ref_dw3x3_f64.restype = ctypes.c_int
    lib.spconv_ref_dw3x3_f64.argtypes = [
        ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
        ctypes.c_void_p, ctypes.c_void_p,
    ]
    lib.spconv_ref_conv3x3_hwc.restype = ctypes.c_int
    lib.spconv_ref_conv3x3_hwc.argtypes = [
        ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
    ]
    lib.spconv_ref_gap.restype = ctypes.c_int
    lib.spconv_ref_gap.argtypes = [
        ctypes.c_int64, ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_void_p,
    ]
    lib.spconv_ref_threads.restype = ctypes.c_int
    lib.spconv_ref_half_to_double.restype = ctypes.c_double
    lib.spconv_ref_half_to_double.argtypes = [ctypes.c_uint16]
    return lib


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        _lib = load_library(_LIB)
    return _lib


def threads() -> int:
    """OpenMP threads the oracle runs with."""
    return int(_load().spconv_ref_threads())


def half_to_double(bits: int) -> float:
    """The oracle's own binary16 decoder (exposed so tests can pin it)."""
    return float(_load().spconv_ref_half_to_double(int(bits) & 0xFFFF))


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def spconv_ref(cout, cin, block_rows, row_ptr, col_idx, values, bias, act, x,
               storage: str = "f32", with_scale: bool = True, lib=None, block_cols: int = 1):
    """Run the oracle.

    ``x`` is [N, Cin, H, W] (or [N, Cin, HW]) float32 for storage "f32" and
    float16 for "f16".  Returns ``(y, y64, scale)``: ``y`` rounded to the
    storage type with the shape [N, Cout, ...] of ``x``, ``y64`` the unrounded
    double values, ``scale`` the error scale (or None).  ``lib`` selects
    another build of the oracle (the tests' planted-mistake builds).
    ``block_cols`` > 1: blocks of block_rows output x block_cols input
    channels, values[(t * block_rows + i) * block_cols + j].
    """
    lib = _load() if lib is None else lib
    row_ptr = np.ascontiguousarray(row_ptr, dtype=np.int32)
    col_idx = np.ascontiguousarray(col_idx, dtype=np.int32)
    values = np.ascontiguousarray(values, dtype=np.float32)
    bias_a = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
    if storage == "f16":
        xa = np.ascontiguousarray(x, dtype=np.float16)
        xbits = xa.view(np.uint16)
        f16 = 1
    else:
        xa = np.ascontiguousarray(x, dtype=np.float32)
        xbits = xa
        f16 = 0
    n = xa.shape[0]
    if xa.shape[1] != cin:
        raise ValueError("x has %d channels, expected %d" % (xa.shape[1], cin))
    spatial = xa.shape[2:]
    hw = int(np.prod(spatial)) if len(spatial) else 1
    y64 = np.empty((n, cout, hw), dtype=np.float64)
    scale = np.empty((n, cout, hw), dtype=np.float64) if with_scale else None
    if block_cols == 1:
        rc = lib.spconv_ref_run(int(cout), int(cin), int(block_rows), _ptr(row_ptr), _ptr(col_idx),
                                _ptr(values), _ptr(bias_a), _ACTS[act], _ptr(xbits), f16,
                                int(n), int(hw), _ptr(y64), _ptr(scale))
    else:
        rc = lib.spconv_ref_run_blocked(int(cout), int(cin), int(block_rows), int(block_cols), _ptr(row_ptr),
                                        _ptr(col_idx), _ptr(values), _ptr(bias_a), _ACTS[act], _ptr(xbits), f16,
                                        int(n), int(hw), _ptr(y64), _ptr(scale))
    if rc != 0:
        raise ValueError("oracle rejected the input (code %d)" % rc)
    y = y64.astype(np.float16 if storage == "f16" else np.float32)
    shape = (n, cout) + tuple(spatial)
    return (y.reshape(shape), y64.reshape(shape),
            None if scale is None else scale.reshape(shape))


def spconv_ref_layer(layer, x=None, with_scale: bool = True):
    """Run the oracle on a ``synth.Layer`` (optionally on another input x)."""
    return spconv_ref(layer.cout, layer.cin, layer.block_rows, layer.row_ptr, layer.col_idx,
                      layer.values, layer.bias, layer.act, layer.x if x is None else x,
                      storage=layer.storage, with_scale=with_scale, block_cols=getattr(layer, "block_cols", 1))


def dw3x3_ref(x, k, bias, act, stride: int, lib=None):
    """Depthwise 3x3, zero padding 1, stride ``stride`` over float32 x [N, C, H, W]
    (k [C, 3, 3]); returns (d, sd) in double, [N, C, Ho, Wo]: the outputs and
    their scale |b| + sum |K * X|."""
    lib = _load() if lib is None else lib
    xa = np.ascontiguousarray(x, dtype=np.float32)
    ka = np.ascontiguousarray(k, dtype=np.float32)
    ba = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
    n, c, h, w = xa.shape
    if ka.shape != (c, 3, 3):
        raise ValueError("k must be [C, 3, 3]")
    ho, wo = (h - 1) // stride + 1, (w - 1) // stride + 1
    d = np.empty((n, c, ho, wo), dtype=np.float64)
    sd = np.empty((n, c, ho, wo), dtype=np.float64)
    rc = lib.spconv_ref_dw3x3(int(n), int(c), int(h), int(w), int(stride), _ptr(xa), _ptr(ka), _ptr(ba),
                              _ACTS[act], _ptr(d), _ptr(sd))
    if rc != 0:
        raise ValueError("oracle rejected the depthwise input (code %d)" % rc)
    return d, sd


def fused_ref(cout, cin, block_rows, row_ptr, col_idx, values, bias, act, x, dw_k, dw_bias, dw_act,
              stride: int, lib=None):
    """The depthwise 3x3 stage, then the sparse 1x1 over its exact (double)
    output.  Returns (y float32, y64, scale) with scale
    S = sum |W * D| + |W| * SD, SD the depthwise stage's own scale."""
    lib = _load() if lib is None else lib
    d, sd = dw3x3_ref(x, dw_k, dw_bias, dw_act, stride, lib=lib)
    n, c, ho, wo = d.shape
    if c != cin:
        raise ValueError("x has %d channels, expected %d" % (c, cin))
    row_ptr = np.ascontiguousarray(row_ptr, dtype=np.int32)
    col_idx = np.ascontiguousarray(col_idx, dtype=np.int32)
    values = np.ascontiguousarray(values, dtype=np.float32)
    bias_a = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
    hw = ho * wo
    y64 = np.empty((n, cout, hw), dtype=np.float64)
    scale = np.empty((n, cout, hw), dtype=np.float64)
    rc = lib.spconv_ref_run_f64(int(cout), int(cin), int(block_rows), _ptr(row_ptr), _ptr(col_idx),
                                _ptr(values), _ptr(bias_a), _ACTS[act], _ptr(d), _ptr(sd),
                                int(n), int(hw), _ptr(y64), _ptr(scale))
    if rc != 0:
        raise ValueError("oracle rejected the input (code %d)" % rc)
    shape = (n, cout, ho, wo)
    return y64.astype(np.float32).reshape(shape), y64.reshape(shape), scale.reshape(shape)


def dw3x3_ref64(x, xs, k, bias, act, stride: int, lib=None):
    """The depthwise 3x3 stage over a double input x [N, C, H, W] with its own
    error scale xs (or None); returns (d, sd) as ``dw3x3_ref``, sd also
    carrying sum |K| * xs."""
    lib = _load() if lib is None else lib
    xa = np.ascontiguousarray(x, dtype=np.float64)
    xsa = None if xs is None else np.ascontiguousarray(xs, dtype=np.float64)
    ka = np.ascontiguousarray(k, dtype=np.float32)
    ba = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
    n, c, h, w = xa.shape
    ho, wo = (h - 1) // stride + 1, (w - 1) // stride + 1
    d = np.empty((n, c, ho, wo), dtype=np.float64)
    sd = np.empty((n, c, ho, wo), dtype=np.float64)
    rc = lib.spconv_ref_dw3x3_f64(int(n), int(c), int(h), int(w), int(stride), _ptr(xa), _ptr(xsa), _ptr(ka),
                                  _ptr(ba), _ACTS[act], _ptr(d), _ptr(sd))
    if rc != 0:
        raise ValueError("oracle rejected the depthwise input (code %d)" % rc)
    return d, sd


def spmm_ref64(cout, cin, block_rows, row_ptr, col_idx, values, bias, act, x, xs, lib=None):
    """The sparse 1x1 over a double input x [N, Cin, H, W] with error scale xs
    (or None); returns (y, scale) in double, scale = sum |W X| + |W| xs."""
    lib = _load() if lib is None else lib
    xa = np.ascontiguousarray(x, dtype=np.float64)
    xsa = None if xs is None else np.ascontiguousarray(xs, dtype=np.float64)
    n, c, h, w = xa.shape
    if c != cin:
        raise ValueError("x has %d channels, expected %d" % (c, cin))
    rp = np.ascontiguousarray(row_ptr, dtype=np.int32)
    ci = np.ascontiguousarray(col_idx, dtype=np.int32)
    va = np.ascontiguousarray(values, dtype=np.float32)
    ba = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
    y = np.empty((n, cout, h * w), dtype=np.float64)
    sc = np.empty((n, cout, h * w), dtype=np.float64)
    rc = lib.spconv_ref_run_f64(int(cout), int(cin), int(block_rows), _ptr(rp), _ptr(ci), _ptr(va), _ptr(ba),
                                _ACTS[act], _ptr(xa), _ptr(xsa), int(n), int(h * w), _ptr(y), _ptr(sc))
    if rc != 0:
        raise ValueError("oracle rejected the input (code %d)" % rc)
    return y.reshape(n, cout, h, w), sc.reshape(n, cout, h, w)


def conv3x3_hwc_ref(x, wt, bias, act, stride: int, lib=None):
    """Dense 3x3 convolution (zero padding 1, stride ``stride``) of float32
    HWC images x [N, H, W, Cin] with wt [Cout, 3, 3, Cin]; returns (y, ys) in
    double, CHW [N, Cout, Ho, Wo], ys = |b| + sum |Wt X|."""
    lib = _load() if lib is None else lib
    xa = np.ascontiguousarray(x, dtype=np.float32)
    wa = np.ascontiguousarray(wt, dtype=np.float32)
    ba = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
    n, h, w, cin = xa.shape
    cout = wa.shape[0]
    if wa.shape != (cout, 3, 3, cin):
        raise ValueError("wt must be [Cout, 3, 3, Cin]")
    ho, wo = (h - 1) // stride + 1, (w - 1) // stride + 1
    y = np.empty((n, cout, ho, wo), dtype=np.float64)
    ys = np.empty((n, cout, ho, wo), dtype=np.float64)
    rc = lib.spconv_ref_conv3x3_hwc(int(n), int(h), int(w), int(cin), int(cout), int(stride), _ptr(xa), _ptr(wa),
                                    _ptr(ba), _ACTS[act], _ptr(y), _ptr(ys))
    if rc != 0:
        raise ValueError("oracle rejected the convolution input (code %d)" % rc)
    return y, ys


def gap_ref(x, xs=None, lib=None):
    """Global average pooling of x [N, C, H, W] (any float type) with error
    scale xs (or None); returns (y, ys) in double, [N, C]."""
    lib = _load() if lib is None else lib
    xa = np.ascontiguousarray(x, dtype=np.float64)
    xsa = None if xs is None else np.ascontiguousarray(xs, dtype=np.float64)
    n, c, h, w = xa.shape
    y = np.empty((n, c), dtype=np.float64)
    ys = np.empty((n, c), dtype=np.float64)
    rc = lib.spconv_ref_gap(int(n), int(c), int(h * w), _ptr(xa), _ptr(xsa), _ptr(y), _ptr(ys))
    if rc != 0:
        raise ValueError("oracle rejected the pooling input (code %d)" % rc)
    return y, ys


def mobilenet_v1_ref(net, x, lib=None):
    """A whole MobileNet v1 forward pass (``synth.MobileNetV1`` weights) on
    HWC images x [N, H, W, 3], in double: the dense stem convolution (stride
    2, ReLU6), 13 blocks of depthwise 3x3 (ReLU6) -> sparse 1x1 (ReLU6),
    global average pooling, the dense classifier (no activation; the
    classifier runs as a 1x1 over 1 x 1 images).  Returns (logits [N,
    classes] double, their error scale S propagated through every layer)."""
    d, s = conv3x3_hwc_ref(x, net.stem_w, net.stem_b, "relu6", 2, lib=lib)
    for blk in net.blocks:
        d, s = dw3x3_ref64(d, s, blk.dw_k, blk.dw_b, "relu6", blk.stride, lib=lib)
        pw = blk.pw
        d, s = spmm_ref64(pw.cout, pw.cin, pw.block_rows, pw.row_ptr, pw.col_idx, pw.values, pw.bias, "relu6",
                          d, s, lib=lib)
    g, gs = gap_ref(d, s, lib=lib)
    n, c = g.shape
    classes = net.fc_w.shape[0]
    rp = np.arange(0, classes * c + 1, c, dtype=np.int32)
    ci = np.tile(np.arange(c, dtype=np.int32), classes)
    y, ys = spmm_ref64(classes, c, 1, rp, ci, net.fc_w.reshape(-1), net.fc_b, "none",
                       g.reshape(n, c, 1, 1), gs.reshape(n, c, 1, 1), lib=lib)
    return y.reshape(n, classes), ys.reshape(n, classes)


def tolerance(y_ref, scale, storage: str):
    """Per-element bound |y_gpu - y_ref| may not exceed.

    fp32: 1e-5 * S + 1e-6.  fp16 storage with fp32 accumulation:
    2e-3 * |y_ref| + 1e-5 * S + 1e-6 (one fp16 ulp of output rounding, the
    fp32 accumulation, and fp16 subnormals).
    """
    tol = 1e-5 * scale + 1e-6
    if storage == "f16":
        tol = tol + 2e-3 * np.abs(y_ref.astype(np.float64))
    return tol
