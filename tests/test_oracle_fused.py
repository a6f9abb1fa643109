"""Pins of the fused depthwise 3x3 -> sparse 1x1 oracle (no GPU).

The depthwise stage (a 3x3 convolution per channel, zero padding 1, stride 1
or 2: the MobileNet block order, paper Sec. 2; the library's CHW depthwise
kernels, Sec. 3.3) is checked against torch's grouped conv2d in fp64, an
independent library routine, and the fused output against the densified
weight applied to that convolution's output."""

import numpy as np
import pytest
import torch
from hypothesis import given, settings, strategies as st

import oracle
from synth import make_layer, densify


def _act(v, act):
    if act == "relu":
        return np.maximum(v, 0.0)
    if act == "relu6":
        return np.minimum(np.maximum(v, 0.0), 6.0)
    return v


def _conv(x, k, b, stride):
    c = x.shape[1]
    return torch.nn.functional.conv2d(torch.from_numpy(x).double(), torch.from_numpy(k).double()[:, None],
                                      None if b is None else torch.from_numpy(b).double(), stride=stride,
                                      padding=1, groups=c).numpy()


@settings(max_examples=40, deadline=None)
@given(c=st.integers(1, 6), h=st.integers(1, 9), w=st.integers(1, 9), n=st.integers(1, 2),
       stride=st.sampled_from([1, 2]), act=st.sampled_from(["none", "relu", "relu6"]),
       with_bias=st.booleans(), seed=st.integers(0, 2 ** 31 - 1))
def test_depthwise_matches_grouped_conv(c, h, w, n, stride, act, with_bias, seed):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((n, c, h, w)).astype(np.float32)
    k = rng.standard_normal((c, 3, 3)).astype(np.float32)
    b = rng.standard_normal(c).astype(np.float32) if with_bias else None
    d, sd = oracle.dw3x3_ref(x, k, b, act, stride)
    ref = _conv(x, k, b, stride)
    sref = _conv(np.abs(x), np.abs(k), None if b is None else np.abs(b), stride)
    assert d.shape == (n, c, (h - 1) // stride + 1, (w - 1) // stride + 1) == ref.shape
    assert np.all(np.abs(d - _act(ref, act)) <= 1e-12 * (sref + 1.0))
    assert np.allclose(sd, sref, rtol=1e-12, atol=0)


@pytest.mark.parametrize("k", [1, 2, 4])
@pytest.mark.parametrize("stride", [1, 2])
@pytest.mark.parametrize("dw_act", ["none", "relu6"])
def test_fused_matches_dense_product_of_conv(k, stride, dw_act):
    layer = make_layer(24, 32, 9, 10, 2, 0.7, block_rows=k, act="relu6", seed=40 + k)
    rng = np.random.default_rng(k + 7 * stride)
    kw = (rng.standard_normal((24, 3, 3)) * 0.3).astype(np.float32)
    kb = (rng.standard_normal(24) * 0.1).astype(np.float32)
    y, y64, s = oracle.fused_ref(32, 24, k, layer.row_ptr, layer.col_idx, layer.values, layer.bias, "relu6",
                                 layer.x, kw, kb, dw_act, stride)
    d = _act(_conv(layer.x, kw, kb, stride), dw_act)
    sd = _conv(np.abs(layer.x), np.abs(kw), np.abs(kb), stride)
    wd = densify(32, 24, k, layer.row_ptr, layer.col_idx, layer.values)
    n, _, ho, wo = d.shape
    ref = _act(np.matmul(wd[None], d.reshape(n, 24, -1)) + layer.bias.astype(np.float64)[None, :, None], "relu6")
    sref = np.matmul(np.abs(wd)[None], np.abs(d.reshape(n, 24, -1)) + sd.reshape(n, 24, -1))
    assert y.shape == (n, 32, ho, wo) and y.dtype == np.float32
    assert np.all(np.abs(y64.reshape(ref.shape) - ref) <= 1e-12 * (sref + 1.0))
    assert np.allclose(s.reshape(sref.shape), sref, rtol=1e-12, atol=0)
    assert np.array_equal(y, y64.astype(np.float32))


def test_identity_depthwise_reduces_to_the_plain_oracle():
    """Center tap 1, no bias, no activation, stride 1: the depthwise stage is the
    identity, so the fused result equals the plain 1x1 oracle's, and the scale
    gains exactly the |W| * |X| of the (exact) first stage."""
    layer = make_layer(16, 24, 7, 7, 2, 0.6, act="relu", seed=3)
    kw = np.zeros((16, 3, 3), np.float32)
    kw[:, 1, 1] = 1.0
    _, y64f, sf = oracle.fused_ref(24, 16, 1, layer.row_ptr, layer.col_idx, layer.values, layer.bias, "relu",
                                   layer.x, kw, None, "none", 1)
    _, y64, s = oracle.spconv_ref_layer(layer)
    assert np.array_equal(y64f, y64)
    assert np.allclose(sf, 2.0 * s, rtol=1e-15, atol=0)


def test_stride_two_corner_taps_read_zero_padding():
    """A 1x1 image: only the center tap lands inside, whatever the stride."""
    x = np.full((1, 2, 1, 1), 3.0, np.float32)
    k = np.arange(18, dtype=np.float32).reshape(2, 3, 3)
    for stride in (1, 2):
        d, _ = oracle.dw3x3_ref(x, k, None, "none", stride)
        assert d.shape == (1, 2, 1, 1) and d[0, 0, 0, 0] == 12.0 and d[0, 1, 0, 0] == 39.0
