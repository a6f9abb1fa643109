"""Helpers shared by the GPU tests: run the HIP library, compare with the oracle."""

from __future__ import annotations

import sys

import numpy as np

import oracle
from paper_1911_09723_amd import Plan


def device():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("GPU tests need a ROCm GPU (torch.cuda.is_available() is False)")
    return torch.device("cuda:0")


def to_gpu(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to(device())


def gpu_run(layer, x=None, **options):
    """Run the library on layer.x (or x) and return Y as a numpy array."""
    import torch
    x = layer.x if x is None else x
    plan = Plan.from_layer(layer, **options)
    try:
        xt = to_gpu(x)
        yt = plan.run(xt)
        torch.cuda.synchronize()
        y = yt.cpu().numpy()
        # every bounded wait inside the kernels succeeded
        assert plan.check() == 0, "a bounded wait gave up (plan error word set)"
        return y
    finally:
        plan.close()


def note(msg: str):
    """Name the case on stdout before the GPU runs it (flushed)."""
    print(msg, flush=True)
    sys.stdout.flush()


def assert_parity(layer, y_gpu, x=None, what=""):
    """Element-wise check against the oracle with the stated tolerance."""
    y_ref, _, scale = oracle.spconv_ref_layer(layer, x=x)
    assert y_gpu.shape == y_ref.shape and y_gpu.dtype == y_ref.dtype, (y_gpu.shape, y_ref.shape)
    tol = oracle.tolerance(y_ref, scale, layer.storage)
    err = np.abs(y_gpu.astype(np.float64) - y_ref.astype(np.float64))
    ratio = err / tol
    worst = float(ratio.max()) if ratio.size else 0.0
    bad = int((ratio > 1).sum())
    assert bad == 0, "%s: %d of %d elements outside tolerance (worst error/tolerance %.3g)" % (
        what, bad, ratio.size, worst)
    return worst


def gpu_run_fused(layer, dw_k, dw_b, dw_act, stride, x=None, **options):
    """Run a fused depthwise 3x3 -> sparse 1x1 plan on layer.x (the depthwise input)."""
    import torch
    x = layer.x if x is None else x
    plan = Plan.fused(layer.cout, layer.cin, layer.block_rows, layer.row_ptr, layer.col_idx, layer.values,
                      layer.bias, layer.act, dw_k, dw_b, dw_act, stride, **options)
    try:
        yt = plan.run(to_gpu(x))
        torch.cuda.synchronize()
        y = yt.cpu().numpy()
        assert plan.check() == 0, "a bounded wait gave up (plan error word set)"
        return y
    finally:
        plan.close()


def assert_fused_parity(layer, dw_k, dw_b, dw_act, stride, y_gpu, x=None, what=""):
    """Element-wise check of a fused run against the oracle, tolerance
    1e-5 * S + 1e-6 with S = sum |W * D| + |W| * SD (SD: the depthwise stage's
    sum of absolute terms), which bounds the fp32 error of both stages."""
    x = layer.x if x is None else x
    y_ref, _, scale = oracle.fused_ref(layer.cout, layer.cin, layer.block_rows, layer.row_ptr, layer.col_idx,
                                       layer.values, layer.bias, layer.act, x, dw_k, dw_b, dw_act, stride)
    assert y_gpu.shape == y_ref.shape and y_gpu.dtype == y_ref.dtype, (y_gpu.shape, y_ref.shape)
    tol = oracle.tolerance(y_ref, scale, "f32")
    ratio = np.abs(y_gpu.astype(np.float64) - y_ref.astype(np.float64)) / tol
    bad = int((ratio > 1).sum())
    assert bad == 0, "%s: %d of %d elements outside tolerance (worst error/tolerance %.3g)" % (
        what, bad, ratio.size, float(ratio.max()))
    return float(ratio.max()) if ratio.size else 0.0
