"""Pins of the network-level oracle functions (no GPU).

The dense HWC -> CHW stem convolution (paper Sec. 3.1, Sec. 3.3), global
average pooling (Sec. 3.3), the double-input depthwise and 1x1 stages and the
whole-network chain are checked against torch / numpy library routines in
fp64: an independent evaluation of the same definitions."""

import numpy as np
import pytest
import torch
from hypothesis import given, settings, strategies as st

import oracle
from synth import make_layer, densify, make_mobilenet_v1, make_image, MBV1_BLOCKS

F = torch.nn.functional


def _act(v, act):
    if act == "relu":
        return np.maximum(v, 0.0)
    if act == "relu6":
        return np.minimum(np.maximum(v, 0.0), 6.0)
    return v


@settings(max_examples=30, deadline=None)
@given(n=st.integers(1, 2), h=st.integers(1, 11), w=st.integers(1, 11), cin=st.integers(1, 4),
       cout=st.integers(1, 6), stride=st.sampled_from([1, 2]), act=st.sampled_from(["none", "relu", "relu6"]),
       with_bias=st.booleans(), seed=st.integers(0, 2 ** 31 - 1))
def test_stem_conv_matches_torch(n, h, w, cin, cout, stride, act, with_bias, seed):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((n, h, w, cin)).astype(np.float32)
    wt = rng.standard_normal((cout, 3, 3, cin)).astype(np.float32)
    b = rng.standard_normal(cout).astype(np.float32) if with_bias else None
    y, ys = oracle.conv3x3_hwc_ref(x, wt, b, act, stride)
    xt = torch.from_numpy(x).double().permute(0, 3, 1, 2)
    wtt = torch.from_numpy(wt).double().permute(0, 3, 1, 2)
    bt = None if b is None else torch.from_numpy(b).double()
    ref = F.conv2d(xt, wtt, bt, stride=stride, padding=1).numpy()
    sref = F.conv2d(xt.abs(), wtt.abs(), None if bt is None else bt.abs(), stride=stride, padding=1).numpy()
    assert y.shape == ref.shape == (n, cout, (h - 1) // stride + 1, (w - 1) // stride + 1)
    assert np.all(np.abs(y - _act(ref, act)) <= 1e-12 * (sref + 1))
    assert np.allclose(ys, sref, rtol=1e-12, atol=0)


def test_stem_output_size_and_padding_at_224():
    """224 x 224 with stride 2 gives 112 x 112; the top-left output sees only
    the 2 x 2 taps at the image corner (zero padding above and left)."""
    x = np.ones((1, 224, 224, 3), np.float32)
    wt = np.ones((2, 3, 3, 3), np.float32)
    y, _ = oracle.conv3x3_hwc_ref(x, wt, None, "none", 2)
    assert y.shape == (1, 2, 112, 112)
    assert y[0, 0, 0, 0] == 12.0 and y[0, 0, 1, 1] == 27.0 and y[0, 1, 111, 111] == 27.0


@pytest.mark.parametrize("shape", [(2, 3, 7, 7), (1, 5, 1, 1), (3, 2, 13, 4)])
def test_gap_matches_numpy_mean(shape):
    rng = np.random.default_rng(sum(shape))
    x = rng.standard_normal(shape)
    xs = np.abs(rng.standard_normal(shape))
    y, ys = oracle.gap_ref(x, xs)
    assert np.allclose(y, x.mean(axis=(2, 3)), rtol=1e-13, atol=1e-15)
    assert np.allclose(ys, (np.abs(x) + xs).mean(axis=(2, 3)), rtol=1e-13, atol=0)


def test_gap_of_a_constant_plane_is_exact():
    x = np.full((1, 2, 7, 7), 0.375)
    y, _ = oracle.gap_ref(x)
    assert np.all(y == 0.375)


@pytest.mark.parametrize("stride", [1, 2])
def test_dw64_matches_grouped_conv_and_carries_input_scale(stride):
    rng = np.random.default_rng(stride)
    x = rng.standard_normal((2, 5, 9, 8))
    xs = np.abs(rng.standard_normal(x.shape))
    k = rng.standard_normal((5, 3, 3)).astype(np.float32)
    b = rng.standard_normal(5).astype(np.float32)
    d, sd = oracle.dw3x3_ref64(x, xs, k, b, "relu", stride)
    kt = torch.from_numpy(k).double()[:, None]
    ref = F.conv2d(torch.from_numpy(x), kt, torch.from_numpy(b).double(), stride=stride, padding=1, groups=5)
    sref = F.conv2d(torch.from_numpy(np.abs(x) + xs), kt.abs(), torch.from_numpy(np.abs(b)).double(),
                    stride=stride, padding=1, groups=5)
    assert np.allclose(d, np.maximum(ref.numpy(), 0), rtol=1e-12, atol=1e-12)
    assert np.allclose(sd, sref.numpy(), rtol=1e-12, atol=0)


@pytest.mark.parametrize("k", [1, 4])
def test_spmm64_matches_dense_product(k):
    layer = make_layer(24, 16, 3, 5, 2, 0.7, block_rows=k, act="relu6", seed=9)
    rng = np.random.default_rng(4)
    x = rng.standard_normal((2, 24, 3, 5))
    xs = np.abs(rng.standard_normal(x.shape))
    y, sc = oracle.spmm_ref64(16, 24, k, layer.row_ptr, layer.col_idx, layer.values, layer.bias, "relu6", x, xs)
    wd = densify(16, 24, k, layer.row_ptr, layer.col_idx, layer.values)
    ref = np.einsum("rc,ncp->nrp", wd, x.reshape(2, 24, -1)) + layer.bias.astype(np.float64)[None, :, None]
    sref = np.einsum("rc,ncp->nrp", np.abs(wd), np.abs(x.reshape(2, 24, -1)) + xs.reshape(2, 24, -1))
    assert np.allclose(y.reshape(2, 16, -1), _act(ref, "relu6"), rtol=1e-12, atol=1e-12)
    assert np.allclose(sc.reshape(2, 16, -1), sref, rtol=1e-12, atol=0)


def _torch_mobilenet(net, x):
    """The same network from torch library routines in fp64."""
    t = torch.from_numpy(x).double().permute(0, 3, 1, 2)
    t = F.conv2d(t, torch.from_numpy(net.stem_w).double().permute(0, 3, 1, 2), torch.from_numpy(net.stem_b).double(),
                 stride=2, padding=1).clamp(0, 6)
    for blk in net.blocks:
        t = F.conv2d(t, torch.from_numpy(blk.dw_k).double()[:, None], torch.from_numpy(blk.dw_b).double(),
                     stride=blk.stride, padding=1, groups=blk.cin).clamp(0, 6)
        pw = blk.pw
        wd = torch.from_numpy(densify(pw.cout, pw.cin, pw.block_rows, pw.row_ptr, pw.col_idx, pw.values))
        t = F.conv2d(t, wd[:, :, None, None], torch.from_numpy(pw.bias).double()).clamp(0, 6)
    g = t.mean(dim=(2, 3))
    return (g @ torch.from_numpy(net.fc_w).double().T + torch.from_numpy(net.fc_b).double()).numpy()


def test_mobilenet_chain_matches_torch_at_small_size():
    """Full 13-block chain on 32 x 32 images (the strides still take it to 1 x 1)."""
    net = make_mobilenet_v1(seed=3, sparsity=0.9, classes=10)
    x = make_image(2, 32, 32, seed=3)
    y, s = oracle.mobilenet_v1_ref(net, x)
    ref = _torch_mobilenet(net, x)
    assert y.shape == (2, 10)
    assert np.allclose(y, ref, rtol=1e-10, atol=1e-12)
    assert np.all(s >= np.abs(y) - 1e-9)


def test_mobilenet_architecture():
    net = make_mobilenet_v1(seed=0)
    assert [(b.cin, b.cout, b.stride) for b in net.blocks] == MBV1_BLOCKS
    assert net.stem_w.shape == (32, 3, 3, 3) and net.fc_w.shape == (1000, 1024)
    for b in net.blocks:
        assert b.pw.nnz == round(0.1 * b.cin * b.cout)
