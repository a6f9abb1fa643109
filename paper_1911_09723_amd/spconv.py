"""Python binding of libspconv's C ABI (include/spconv.h).

Argument marshalling only: every step of the operation runs inside the
library (host planner and HIP kernels).  The functions carry the C names;
``Plan`` is a small convenience wrapper.  PyTorch supplies device memory and
streams when tensors are passed; raw integer device addresses work too.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIBRARY_PATH = os.path.join(_HERE, "libspconv.so")

OK, E_ARG, E_FORMAT, E_SHAPE, E_UNSUPPORTED, E_NOMEM, E_HIP = range(7)
STATUS_NAMES = {0: "SPCONV_OK", 1: "SPCONV_E_ARG", 2: "SPCONV_E_FORMAT", 3: "SPCONV_E_SHAPE",
                4: "SPCONV_E_UNSUPPORTED", 5: "SPCONV_E_NOMEM", 6: "SPCONV_E_HIP"}
F32, F16 = 0, 1
ACT_NONE, ACT_RELU, ACT_RELU6 = 0, 1, 2
_ACTS = {"none": ACT_NONE, "relu": ACT_RELU, "relu6": ACT_RELU6}
_DTYPES = {"f32": F32, "f16": F16}

# Symbols declared in include/spconv.h.
EXPORTED = ("spconv_plan_create", "spconv_run", "spconv_destroy", "spconv_last_error",
            "spconv_options_init", "spconv_plan_create_ex", "spconv_plan_get_info", "spconv_plan_unpack",
            "spconv_plan_unpack_interleaved", "spconv_detect_block_rows", "spconv_dense_to_bcsr",
            "spconv_plan_create_dense", "spconv_plan_create_fused", "spconv_conv3x3_hwc", "spconv_depthwise3x3",
            "spconv_global_avg_pool", "spconv_linear", "spconv_plan_create_blocked", "spconv_detect_blocks",
            "spconv_dense_to_bcsr_blocked", "spconv_plan_create_dense_blocked", "spconv_plan_unpack_indexed",
            "spconv_plan_check", "spconv_plan_set_wait_limit", "spconv_plan_create_static",
            "spconv_plan_unpack_outer")


class SpconvError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__("%s: %s" % (STATUS_NAMES.get(status, status), message))
        self.status = status
        self.message = message


class spconv_options(ctypes.Structure):
    _fields_ = [("struct_size", ctypes.c_int32), ("reorder", ctypes.c_int32), ("host_only", ctypes.c_int32),
                ("kernel", ctypes.c_int32), ("group_lanes", ctypes.c_int32), ("waves", ctypes.c_int32),
                ("pipe_sets", ctypes.c_int32), ("regions", ctypes.c_int32),
                ("lane_cols", ctypes.c_int32)]


class spconv_plan_info(ctypes.Structure):
    _fields_ = [("cout", ctypes.c_int32), ("cin", ctypes.c_int32), ("block_rows", ctypes.c_int32),
                ("storage", ctypes.c_int32), ("act", ctypes.c_int32), ("kernel", ctypes.c_int32),
                ("group_lanes", ctypes.c_int32), ("bundle_rows", ctypes.c_int32), ("cols_per_lane", ctypes.c_int32),
                ("tile_cols", ctypes.c_int32), ("waves", ctypes.c_int32), ("lds_bytes", ctypes.c_int32),
                ("max_parts", ctypes.c_int32), ("pipe_sets", ctypes.c_int32), ("regions", ctypes.c_int32),
                ("nnzb", ctypes.c_int64), ("slots", ctypes.c_int64),
                ("max_wave_cost", ctypes.c_int64), ("sum_wave_cost", ctypes.c_int64),
                ("device_bytes", ctypes.c_int64), ("dw_stride", ctypes.c_int32), ("dw_act", ctypes.c_int32),
                ("block_cols", ctypes.c_int32), ("split_rows", ctypes.c_int32), ("indexed_min_cols", ctypes.c_int64),
                ("outer_min_cols", ctypes.c_int64), ("channel_passes", ctypes.c_int64)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


_lib = None


def load_library(path: Optional[str] = None):
    """Load libspconv.so (built in-tree by paper_1911_09723_amd.build).  Fails loudly if missing."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIBRARY_PATH
    if not os.path.exists(p):
        raise RuntimeError("libspconv.so is not built (%s); run `python -m paper_1911_09723_amd.build`" % p)
    # PyTorch for ROCm carries its own HIP runtime with the same soname
    # (libamdhip64.so.7) as the one this library links.  Loaded after
    # PyTorch, the library binds to PyTorch's runtime and the process has one;
    # loaded first, PyTorch would bring up a second runtime instance and this
    # library's calls would find no device.  So PyTorch, when installed, is
    # imported first.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ctypes.CDLL(p)
    vp, i32 = ctypes.c_void_p, ctypes.c_int32
    lib.spconv_plan_create.restype = i32
    lib.spconv_plan_create.argtypes = [ctypes.POINTER(vp), i32, i32, i32, vp, vp, vp, vp, i32, i32]
    lib.spconv_plan_create_ex.restype = i32
    lib.spconv_plan_create_ex.argtypes = [ctypes.POINTER(vp), i32, i32, i32, vp, vp, vp, vp, i32, i32,
                                          ctypes.POINTER(spconv_options)]
    lib.spconv_run.restype = i32
    lib.spconv_run.argtypes = [vp, vp, vp, i32, i32, i32, vp]
    lib.spconv_destroy.restype = i32
    lib.spconv_destroy.argtypes = [vp]
    lib.spconv_last_error.restype = ctypes.c_char_p
    lib.spconv_last_error.argtypes = []
    lib.spconv_options_init.restype = None
    lib.spconv_options_init.argtypes = [ctypes.POINTER(spconv_options)]
    lib.spconv_plan_get_info.restype = i32
    lib.spconv_plan_get_info.argtypes = [vp, ctypes.POINTER(spconv_plan_info)]
    lib.spconv_plan_unpack.restype = i32
    lib.spconv_plan_unpack.argtypes = [vp, vp, vp, vp, vp]
    lib.spconv_plan_unpack_interleaved.restype = i32
    lib.spconv_plan_unpack_interleaved.argtypes = [vp, vp, vp, vp]
    lib.spconv_plan_unpack_indexed.restype = i32
    lib.spconv_plan_unpack_indexed.argtypes = [vp, i32, vp, vp, vp]
    lib.spconv_plan_unpack_outer.restype = i32
    lib.spconv_plan_unpack_outer.argtypes = [vp, vp, vp, vp]
    lib.spconv_plan_create_static.restype = i32
    lib.spconv_plan_create_static.argtypes = [ctypes.POINTER(vp), i32, i32, i32, vp, vp, vp, vp, i32, i32,
                                              ctypes.POINTER(spconv_options)]
    lib.spconv_plan_check.restype = i32
    lib.spconv_plan_check.argtypes = [vp, ctypes.POINTER(i32), i32]
    lib.spconv_plan_set_wait_limit.restype = i32
    lib.spconv_plan_set_wait_limit.argtypes = [vp, i32]
    lib.spconv_detect_block_rows.restype = i32
    lib.spconv_detect_block_rows.argtypes = [i32, i32, vp, ctypes.POINTER(i32)]
    lib.spconv_dense_to_bcsr.restype = i32
    lib.spconv_dense_to_bcsr.argtypes = [i32, i32, vp, i32, vp, vp, vp, ctypes.c_int64, ctypes.POINTER(ctypes.c_int64)]
    lib.spconv_plan_create_dense.restype = i32
    lib.spconv_plan_create_dense.argtypes = [ctypes.POINTER(vp), i32, i32, vp, i32, vp, i32, i32]
    lib.spconv_plan_create_blocked.restype = i32
    lib.spconv_plan_create_blocked.argtypes = [ctypes.POINTER(vp), i32, i32, i32, i32, vp, vp, vp, vp, i32, i32,
                                               ctypes.POINTER(spconv_options)]
    lib.spconv_detect_blocks.restype = i32
    lib.spconv_detect_blocks.argtypes = [i32, i32, vp, ctypes.POINTER(i32), ctypes.POINTER(i32)]
    lib.spconv_dense_to_bcsr_blocked.restype = i32
    lib.spconv_dense_to_bcsr_blocked.argtypes = [i32, i32, vp, i32, i32, vp, vp, vp, ctypes.c_int64,
                                                 ctypes.POINTER(ctypes.c_int64)]
    lib.spconv_plan_create_dense_blocked.restype = i32
    lib.spconv_plan_create_dense_blocked.argtypes = [ctypes.POINTER(vp), i32, i32, vp, i32, i32, vp, i32, i32]
    lib.spconv_plan_create_fused.restype = i32
    lib.spconv_plan_create_fused.argtypes = [ctypes.POINTER(vp), i32, i32, i32, vp, vp, vp, vp, i32, vp, vp, i32,
                                             i32, i32, ctypes.POINTER(spconv_options)]
    lib.spconv_conv3x3_hwc.restype = i32
    lib.spconv_conv3x3_hwc.argtypes = [vp, vp, vp, i32, i32, vp, i32, i32, i32, i32, i32, vp]
    lib.spconv_depthwise3x3.restype = i32
    lib.spconv_depthwise3x3.argtypes = [vp, vp, vp, i32, i32, vp, i32, i32, i32, i32, vp]
    lib.spconv_linear.restype = i32
    lib.spconv_linear.argtypes = [vp, vp, vp, i32, vp, i32, i32, i32, vp]
    lib.spconv_global_avg_pool.restype = i32
    lib.spconv_global_avg_pool.argtypes = [vp, vp, i32, i32, i32, i32, vp]
    if path is None:
        _lib = lib
    return lib


def _arr(a, dtype):
    if a is None:
        return None
    return np.ascontiguousarray(a, dtype=dtype)


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _check(status: int):
    if status != OK:
        raise SpconvError(status, spconv_last_error())


def spconv_last_error() -> str:
    return load_library().spconv_last_error().decode()


def spconv_options_init() -> spconv_options:
    o = spconv_options()
    load_library().spconv_options_init(ctypes.byref(o))
    return o


def spconv_plan_create(cout, cin, block_rows, row_ptr, col_idx, values, bias=None, act="none",
                       storage="f32", options: Optional[spconv_options] = None, check: bool = True):
    """Create a plan from host CSR / 1xk block-CSR arrays.  Returns the plan handle (int).

    With ``check=False`` returns ``(status, handle)`` instead of raising.
    """
    lib = load_library()
    rp = _arr(row_ptr, np.int32)
    ci = _arr(col_idx, np.int32)
    va = _arr(values, np.float32)
    bi = _arr(bias, np.float32)
    out = ctypes.c_void_p()
    a = _ACTS[act] if isinstance(act, str) else int(act)
    st = _DTYPES[storage] if isinstance(storage, str) else int(storage)
    if options is None:
        status = lib.spconv_plan_create(ctypes.byref(out), int(cout), int(cin), int(block_rows), _ptr(rp),
                                        _ptr(ci), _ptr(va), _ptr(bi), a, st)
    else:
        status = lib.spconv_plan_create_ex(ctypes.byref(out), int(cout), int(cin), int(block_rows), _ptr(rp),
                                           _ptr(ci), _ptr(va), _ptr(bi), a, st, ctypes.byref(options))
    if not check:
        return status, out.value
    _check(status)
    return out.value


SPCONV_STATIC_PLAN_BYTES = 32 << 20


def spconv_plan_create_static(cout, cin, block_rows, row_ptr, col_idx, values, bias=None, act="none",
                              storage="f32", options: Optional[spconv_options] = None, check: bool = True):
    """As spconv_plan_create, with the plan's device image in the library's
    static per-GPU array (no device allocation; only the last such plan on a
    device can run).  Returns the plan handle (or (status, handle))."""
    lib = load_library()
    rp = _arr(row_ptr, np.int32)
    ci = _arr(col_idx, np.int32)
    va = _arr(values, np.float32)
    bi = _arr(bias, np.float32)
    out = ctypes.c_void_p()
    a = _ACTS[act] if isinstance(act, str) else int(act)
    st = _DTYPES[storage] if isinstance(storage, str) else int(storage)
    status = lib.spconv_plan_create_static(ctypes.byref(out), int(cout), int(cin), int(block_rows), _ptr(rp),
                                           _ptr(ci), _ptr(va), _ptr(bi), a, st,
                                           ctypes.byref(options) if options is not None else None)
    if not check:
        return status, out.value
    _check(status)
    return out.value


def spconv_plan_create_blocked(cout, cin, block_rows, block_cols, row_ptr, col_idx, values, bias=None, act="none",
                               storage="f32", options: Optional[spconv_options] = None, check: bool = True):
    """Create a plan from block-CSR weights with block_rows output x block_cols
    input channels per block (values[(t * block_rows + i) * block_cols + j])."""
    lib = load_library()
    rp = _arr(row_ptr, np.int32)
    ci = _arr(col_idx, np.int32)
    va = _arr(values, np.float32)
    bi = _arr(bias, np.float32)
    out = ctypes.c_void_p()
    a = _ACTS[act] if isinstance(act, str) else int(act)
    st = _DTYPES[storage] if isinstance(storage, str) else int(storage)
    status = lib.spconv_plan_create_blocked(ctypes.byref(out), int(cout), int(cin), int(block_rows), int(block_cols),
                                            _ptr(rp), _ptr(ci), _ptr(va), _ptr(bi), a, st,
                                            ctypes.byref(options) if options is not None else None)
    if not check:
        return status, out.value
    _check(status)
    return out.value


def spconv_detect_block_rows(dense) -> int:
    """Largest k in (4, 2, 1) for which the dense [Cout, Cin] weight is 1 x k blocked."""
    d = _arr(dense, np.float32)
    k = ctypes.c_int32()
    _check(load_library().spconv_detect_block_rows(int(d.shape[0]), int(d.shape[1]), _ptr(d), ctypes.byref(k)))
    return k.value


def spconv_dense_to_bcsr(dense, block_rows: int):
    """Convert a dense [Cout, Cin] weight to 1 x block_rows block-CSR: (row_ptr, col_idx, values)."""
    lib = load_library()
    d = _arr(dense, np.float32)
    cout, cin = int(d.shape[0]), int(d.shape[1])
    n = ctypes.c_int64()
    _check(lib.spconv_dense_to_bcsr(cout, cin, _ptr(d), int(block_rows), None, None, None, 0, ctypes.byref(n)))
    k = int(block_rows)
    rp = np.zeros(cout // k + 1, np.int32)
    ci = np.zeros(max(n.value, 1), np.int32)
    va = np.zeros(max(n.value, 1) * k, np.float32)
    _check(lib.spconv_dense_to_bcsr(cout, cin, _ptr(d), k, _ptr(rp), _ptr(ci), _ptr(va), n.value, ctypes.byref(n)))
    return rp, ci[:n.value], va[:n.value * k]


def spconv_detect_blocks(dense):
    """(block_rows, block_cols) detected in a dense [Cout, Cin] weight."""
    d = _arr(dense, np.float32)
    kr, kc = ctypes.c_int32(), ctypes.c_int32()
    _check(load_library().spconv_detect_blocks(int(d.shape[0]), int(d.shape[1]), _ptr(d), ctypes.byref(kr),
                                               ctypes.byref(kc)))
    return kr.value, kc.value


def spconv_dense_to_bcsr_blocked(dense, block_rows: int, block_cols: int):
    """Convert a dense weight to block_rows x block_cols blocks: (row_ptr, col_idx, values)."""
    lib = load_library()
    d = _arr(dense, np.float32)
    cout, cin = int(d.shape[0]), int(d.shape[1])
    kr, kc = int(block_rows), int(block_cols)
    n = ctypes.c_int64()
    _check(lib.spconv_dense_to_bcsr_blocked(cout, cin, _ptr(d), kr, kc, None, None, None, 0, ctypes.byref(n)))
    rp = np.zeros(cout // kr + 1, np.int32)
    ci = np.zeros(max(n.value, 1), np.int32)
    va = np.zeros(max(n.value, 1) * kr * kc, np.float32)
    _check(lib.spconv_dense_to_bcsr_blocked(cout, cin, _ptr(d), kr, kc, _ptr(rp), _ptr(ci), _ptr(va), n.value,
                                            ctypes.byref(n)))
    return rp, ci[:n.value], va[:n.value * kr * kc]


def spconv_plan_create_dense_blocked(dense, block_rows: int = 0, block_cols: int = 0, bias=None, act="none",
                                     storage="f32", check: bool = True):
    """Plan from a dense weight with 2-D blocks (0, 0 = detect)."""
    d = _arr(dense, np.float32)
    bi = _arr(bias, np.float32)
    out = ctypes.c_void_p()
    a = _ACTS[act] if isinstance(act, str) else int(act)
    st = _DTYPES[storage] if isinstance(storage, str) else int(storage)
    status = load_library().spconv_plan_create_dense_blocked(ctypes.byref(out), int(d.shape[0]), int(d.shape[1]),
                                                             _ptr(d), int(block_rows), int(block_cols), _ptr(bi), a,
                                                             st)
    if not check:
        return status, out.value
    _check(status)
    return out.value


def spconv_plan_create_dense(dense, block_rows: int = 0, bias=None, act="none", storage="f32",
                             check: bool = True):
    """Create a plan from a dense [Cout, Cin] weight (block_rows 0 = detect).  Returns the handle."""
    d = _arr(dense, np.float32)
    bi = _arr(bias, np.float32)
    out = ctypes.c_void_p()
    a = _ACTS[act] if isinstance(act, str) else int(act)
    st = _DTYPES[storage] if isinstance(storage, str) else int(storage)
    status = load_library().spconv_plan_create_dense(ctypes.byref(out), int(d.shape[0]), int(d.shape[1]), _ptr(d),
                                                     int(block_rows), _ptr(bi), a, st)
    if not check:
        return status, out.value
    _check(status)
    return out.value


def spconv_plan_create_fused(cout, cin, block_rows, row_ptr, col_idx, values, bias, act, dw_weights, dw_bias=None,
                             dw_act="none", dw_stride=1, storage="f32", options: Optional[spconv_options] = None,
                             check: bool = True):
    """Create a plan for a depthwise 3x3 (weights [cin, 3, 3], zero padding 1,
    stride ``dw_stride``) followed by the sparse 1x1.  Returns the handle."""
    lib = load_library()
    rp = _arr(row_ptr, np.int32)
    ci = _arr(col_idx, np.int32)
    va = _arr(values, np.float32)
    bi = _arr(bias, np.float32)
    kw = _arr(dw_weights, np.float32)
    kb = _arr(dw_bias, np.float32)
    out = ctypes.c_void_p()
    a = _ACTS[act] if isinstance(act, str) else int(act)
    da = _ACTS[dw_act] if isinstance(dw_act, str) else int(dw_act)
    st = _DTYPES[storage] if isinstance(storage, str) else int(storage)
    status = lib.spconv_plan_create_fused(ctypes.byref(out), int(cout), int(cin), int(block_rows), _ptr(rp), _ptr(ci),
                                          _ptr(va), _ptr(bi), a, _ptr(kw), _ptr(kb), da, int(dw_stride), st,
                                          ctypes.byref(options) if options is not None else None)
    if not check:
        return status, out.value
    _check(status)
    return out.value


def _devptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def spconv_run(plan, x, y, n, h, w, stream=None, check: bool = True):
    """Queue y = act(W x + b) on ``stream`` (torch stream, raw hipStream_t int, or None for torch's current)."""
    lib = load_library()
    if stream is None:
        import torch
        stream = torch.cuda.current_stream().cuda_stream
    elif not isinstance(stream, int):
        stream = stream.cuda_stream
    status = lib.spconv_run(plan, _devptr(x), _devptr(y), int(n), int(h), int(w), stream or None)
    if check:
        _check(status)
    return status


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return stream if isinstance(stream, int) else stream.cuda_stream


def spconv_conv3x3_hwc(x, weight, bias, act, stride, y, n, h, w, cin, cout, stream=None, check: bool = True):
    """Queue the dense 3x3 HWC -> CHW convolution (device tensors or addresses)."""
    a = _ACTS[act] if isinstance(act, str) else int(act)
    status = load_library().spconv_conv3x3_hwc(_devptr(x), _devptr(weight), _devptr(bias), a, int(stride),
                                               _devptr(y), int(n), int(h), int(w), int(cin), int(cout),
                                               _stream(stream) or None)
    if check:
        _check(status)
    return status


def spconv_depthwise3x3(x, weight, bias, act, stride, y, n, c, h, w, stream=None, check: bool = True):
    """Queue a standalone depthwise 3x3 convolution on CHW tensors."""
    a = _ACTS[act] if isinstance(act, str) else int(act)
    status = load_library().spconv_depthwise3x3(_devptr(x), _devptr(weight), _devptr(bias), a, int(stride),
                                                _devptr(y), int(n), int(c), int(h), int(w), _stream(stream) or None)
    if check:
        _check(status)
    return status


def spconv_linear(x, weight, bias, act, y, n, cin, cout, stream=None, check: bool = True):
    """Queue the dense fully connected layer y = act(x W^T + b)."""
    a = _ACTS[act] if isinstance(act, str) else int(act)
    status = load_library().spconv_linear(_devptr(x), _devptr(weight), _devptr(bias), a, _devptr(y), int(n),
                                          int(cin), int(cout), _stream(stream) or None)
    if check:
        _check(status)
    return status


def spconv_global_avg_pool(x, y, n, c, h, w, stream=None, check: bool = True):
    """Queue global average pooling [N, C, H, W] -> [N, C]."""
    status = load_library().spconv_global_avg_pool(_devptr(x), _devptr(y), int(n), int(c), int(h), int(w),
                                                   _stream(stream) or None)
    if check:
        _check(status)
    return status


def spconv_destroy(plan):
    _check(load_library().spconv_destroy(plan))


def spconv_plan_get_info(plan) -> dict:
    info = spconv_plan_info()
    _check(load_library().spconv_plan_get_info(plan, ctypes.byref(info)))
    return info.as_dict()


def spconv_plan_unpack(plan):
    """Return (row_ptr, col_idx, values, perm) rebuilt from the plan's packed host image."""
    info = spconv_plan_get_info(plan)
    rows = info["cout"] // info["block_rows"]
    per = info["block_rows"] * info["block_cols"]
    rp = np.zeros(rows + 1, np.int32)
    ci = np.zeros(max(info["nnzb"], 1), np.int32)
    va = np.zeros(max(info["nnzb"] * per, 1), np.float32)
    perm = np.zeros(rows, np.int32)
    _check(load_library().spconv_plan_unpack(plan, _ptr(rp), _ptr(ci), _ptr(va), _ptr(perm)))
    return rp, ci[:info["nnzb"]], va[:info["nnzb"] * per], perm


def spconv_plan_unpack_interleaved(plan):
    """Return (row_ptr, col_idx, values) rebuilt from the pipelined kernel's interleaved streams."""
    info = spconv_plan_get_info(plan)
    rows = info["cout"] // info["block_rows"]
    per = info["block_rows"] * info["block_cols"]
    rp = np.zeros(rows + 1, np.int32)
    ci = np.zeros(max(info["nnzb"], 1), np.int32)
    va = np.zeros(max(info["nnzb"] * per, 1), np.float32)
    _check(load_library().spconv_plan_unpack_interleaved(plan, _ptr(rp), _ptr(ci), _ptr(va)))
    return rp, ci[:info["nnzb"]], va[:info["nnzb"] * per]


def spconv_plan_unpack_indexed(plan, from_pairs=False):
    """Return (row_ptr, col_idx, values) rebuilt from the register-indexed kernel's
    slot records (or, with from_pairs, its row-pair entries)."""
    info = spconv_plan_get_info(plan)
    rows = info["cout"] // info["block_rows"]
    per = info["block_rows"] * info["block_cols"]
    rp = np.zeros(rows + 1, np.int32)
    ci = np.zeros(max(info["nnzb"], 1), np.int32)
    va = np.zeros(max(info["nnzb"] * per, 1), np.float32)
    _check(load_library().spconv_plan_unpack_indexed(plan, int(bool(from_pairs)), _ptr(rp), _ptr(ci), _ptr(va)))
    return rp, ci[:info["nnzb"]], va[:info["nnzb"] * per]


def spconv_plan_unpack_outer(plan):
    """Return (row_ptr, col_idx, values) rebuilt from the outer-product kernel's records."""
    info = spconv_plan_get_info(plan)
    rows = info["cout"] // info["block_rows"]
    per = info["block_rows"] * info["block_cols"]
    rp = np.zeros(rows + 1, np.int32)
    ci = np.zeros(max(info["nnzb"], 1), np.int32)
    va = np.zeros(max(info["nnzb"] * per, 1), np.float32)
    _check(load_library().spconv_plan_unpack_outer(plan, _ptr(rp), _ptr(ci), _ptr(va)))
    return rp, ci[:info["nnzb"]], va[:info["nnzb"] * per]


SPCONV_FLAG_WAIT_GAVE_UP = 1


def spconv_plan_check(plan, clear: bool = False, check: bool = True):
    """The plan's device error word (bit 0: a bounded wait in a kernel gave up)
    after all work on its device finished; optionally reset it."""
    v = ctypes.c_int32(0)
    status = load_library().spconv_plan_check(plan, ctypes.byref(v), int(bool(clear)))
    if check:
        _check(status)
        return v.value
    return status, v.value


def spconv_plan_set_wait_limit(plan, sleeps: int, check: bool = True):
    """Test hook: bound every bounded wait of the plan's later launches (sleeps)."""
    status = load_library().spconv_plan_set_wait_limit(plan, int(sleeps))
    if check:
        _check(status)
    return status


class Plan:
    """Owning wrapper: ``Plan(...).run(x, y)`` with torch tensors [N, C, H, W]."""

    def __init__(self, cout, cin, block_rows, row_ptr, col_idx, values, bias=None, act="none",
                 storage="f32", **options):
        opts = None
        if options:
            opts = spconv_options_init()
            for k, v in options.items():
                setattr(opts, k, int(v))
        self.handle = spconv_plan_create(cout, cin, block_rows, row_ptr, col_idx, values, bias, act, storage,
                                         options=opts)
        self.cout, self.cin, self.storage, self.dw_stride = int(cout), int(cin), storage, 0

    @classmethod
    def from_dense(cls, dense, block_rows: int = 0, bias=None, act="none", storage="f32"):
        """Plan for a dense masked [Cout, Cin] weight (block_rows 0 = detect the block height)."""
        self = cls.__new__(cls)
        self.handle = spconv_plan_create_dense(dense, block_rows, bias, act, storage)
        self.cout, self.cin, self.storage, self.dw_stride = int(dense.shape[0]), int(dense.shape[1]), storage, 0
        return self

    @classmethod
    def blocked(cls, cout, cin, block_rows, block_cols, row_ptr, col_idx, values, bias=None, act="none",
                storage="f32", **options):
        """Plan for block_rows x block_cols blocks (output x input channels)."""
        self = cls.__new__(cls)
        opts = None
        if options:
            opts = spconv_options_init()
            for k, v in options.items():
                setattr(opts, k, int(v))
        self.handle = spconv_plan_create_blocked(cout, cin, block_rows, block_cols, row_ptr, col_idx, values, bias,
                                                 act, storage, options=opts)
        self.cout, self.cin, self.storage, self.dw_stride = int(cout), int(cin), storage, 0
        return self

    @classmethod
    def fused(cls, cout, cin, block_rows, row_ptr, col_idx, values, bias, act, dw_weights, dw_bias=None,
              dw_act="none", dw_stride=1, **options):
        """Plan for depthwise 3x3 (stride ``dw_stride``, zero padding 1) -> sparse 1x1, fp32."""
        self = cls.__new__(cls)
        opts = None
        if options:
            opts = spconv_options_init()
            for k, v in options.items():
                setattr(opts, k, int(v))
        self.handle = spconv_plan_create_fused(cout, cin, block_rows, row_ptr, col_idx, values, bias, act,
                                               dw_weights, dw_bias, dw_act, dw_stride, options=opts)
        self.cout, self.cin, self.storage, self.dw_stride = int(cout), int(cin), "f32", int(dw_stride)
        return self

    def out_hw(self, h, w):
        """Output spatial size for an h x w input."""
        if not self.dw_stride:
            return h, w
        s = self.dw_stride
        return ((h - 1) // s + 1 if h > 0 else 0), ((w - 1) // s + 1 if w > 0 else 0)

    @classmethod
    def from_layer(cls, layer, **options):
        if getattr(layer, "block_cols", 1) > 1:
            return cls.blocked(layer.cout, layer.cin, layer.block_rows, layer.block_cols, layer.row_ptr,
                               layer.col_idx, layer.values, layer.bias, layer.act, layer.storage, **options)
        return cls(layer.cout, layer.cin, layer.block_rows, layer.row_ptr, layer.col_idx, layer.values,
                   layer.bias, layer.act, layer.storage, **options)

    def check(self, clear: bool = False) -> int:
        """The device error word (0 when every bounded wait of every launch succeeded)."""
        return spconv_plan_check(self.handle, clear)

    def info(self) -> dict:
        return spconv_plan_get_info(self.handle)

    def run(self, x, y=None, stream=None):
        import torch
        n, c, h, w = x.shape
        if c != self.cin:
            raise ValueError("x has %d channels, plan expects %d" % (c, self.cin))
        if y is None:
            y = torch.empty((n, self.cout) + self.out_hw(h, w), dtype=x.dtype, device=x.device)
        spconv_run(self.handle, x, y, n, h, w, stream)
        return y

    def close(self):
        if self.handle:
            spconv_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
