"""Pins for the CPU oracle (no GPU).

The paper prints no numeric example for its kernels, so the oracle is pinned
to things fixed by the mathematics of the definition in Sec. 3.2 / Fig. 2
(1x1 convolution = sparse W times dense CHW activations, 1xk output blocks
sharing one pattern, block-CSR storage of Sec. 3.3):

* hand-derived worked examples with exact dyadic values (tests/golden);
* brute force: the densified weight times X with a library matmul / conv;
* identity weights, all-zero weights, power-of-two scaling, single nonzeros;
* block semantics (1x4 BCSR equals its CSR expansion), row permutations,
  batch splitting;
* the binary16 decoder against numpy on all 65536 bit patterns.
"""

import json
import os

import numpy as np
import pytest
import torch
from hypothesis import given, settings, strategies as st

import oracle
from synth import make_layer, densify, expand_blocks_to_csr

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")


def _act(v, act):
    if act == "relu":
        return np.maximum(v, 0.0)
    if act == "relu6":
        return np.minimum(np.maximum(v, 0.0), 6.0)
    return v


def _brute(layer, x=None):
    """Dense float64 reference: densified W times X with a library matmul."""
    x = layer.x if x is None else x
    wd = densify(layer.cout, layer.cin, layer.block_rows, layer.row_ptr, layer.col_idx, layer.values)
    x64 = x.astype(np.float64).reshape(x.shape[0], layer.cin, -1)
    pre = np.matmul(wd[None], x64) + layer.bias.astype(np.float64)[None, :, None]
    s = np.matmul(np.abs(wd)[None], np.abs(x64))
    return _act(pre, layer.act), s


@pytest.mark.parametrize("case", json.load(open(GOLDEN))["cases"], ids=lambda c: c["name"])
@pytest.mark.parametrize("act", ["none", "relu", "relu6"])
def test_hand_examples(case, act):
    x = np.asarray(case["x"], dtype=np.float32)[None]
    y, y64, s = oracle.spconv_ref(case["cout"], case["cin"], case["block_rows"], case["row_ptr"],
                                  case["col_idx"], case["values"], case["bias"], act, x)
    assert np.array_equal(y64[0], np.asarray(case["y_" + act], dtype=np.float64))
    assert np.array_equal(s[0], np.asarray(case["scale"], dtype=np.float64))
    # the CSR arrays of the fixture really encode its dense matrix
    wd = densify(case["cout"], case["cin"], case["block_rows"], np.asarray(case["row_ptr"]),
                 np.asarray(case["col_idx"]), np.asarray(case["values"], dtype=np.float32))
    assert np.array_equal(wd, np.asarray(case["dense_w"], dtype=np.float64))


@pytest.mark.parametrize("k", [1, 2, 4])
@pytest.mark.parametrize("sparsity", [0.0, 0.5, 0.9, 1.0])
@pytest.mark.parametrize("act", ["none", "relu", "relu6"])
@pytest.mark.parametrize("storage", ["f32", "f16"])
def test_brute_force_small(k, sparsity, act, storage):
    layer = make_layer(12, 16, 3, 5, 2, sparsity, block_rows=k, storage=storage, act=act,
                       seed=17 + k + int(sparsity * 10))
    y, y64, s = oracle.spconv_ref_layer(layer)
    ref, sref = _brute(layer)
    assert np.all(np.abs(y64 - ref.reshape(y64.shape)) <= 1e-12 * (sref.reshape(y64.shape) + 1.0))
    assert np.allclose(s, sref.reshape(s.shape), rtol=1e-12, atol=0)
    # storage rounding: one round-to-nearest-even step from the double result
    assert np.array_equal(y, y64.astype(y.dtype))


@settings(max_examples=60, deadline=None)
@given(cin=st.integers(1, 16), cout4=st.integers(1, 4), k=st.sampled_from([1, 2, 4]),
       hw=st.integers(1, 20), n=st.integers(1, 3),
       sparsity=st.sampled_from([0.0, 0.5, 0.9, 1.0]), act=st.sampled_from(["none", "relu", "relu6"]),
       seed=st.integers(0, 2 ** 31 - 1))
def test_brute_force_property(cin, cout4, k, hw, n, sparsity, act, seed):
    layer = make_layer(cin, 4 * cout4, 1, hw, n, sparsity, block_rows=k, act=act, seed=seed)
    _, y64, s = oracle.spconv_ref_layer(layer)
    ref, sref = _brute(layer)
    assert np.all(np.abs(y64 - ref.reshape(y64.shape)) <= 1e-12 * (sref.reshape(y64.shape) + 1.0))


def test_zero_sparsity_matches_dense_conv():
    """0% sparsity at a realistic size equals a dense fp64 1x1 convolution."""
    layer = make_layer(64, 128, 14, 14, 2, 0.0, act="none", seed=5)
    _, y64, s = oracle.spconv_ref_layer(layer)
    wd = densify(128, 64, 1, layer.row_ptr, layer.col_idx, layer.values)
    ref = torch.nn.functional.conv2d(torch.from_numpy(layer.x.astype(np.float64)),
                                     torch.from_numpy(wd).reshape(128, 64, 1, 1),
                                     torch.from_numpy(layer.bias.astype(np.float64))).numpy()
    assert layer.nnz == 64 * 128
    assert np.all(np.abs(y64 - ref) <= 1e-12 * (s + 1.0))


@pytest.mark.parametrize("storage", ["f32", "f16"])
@pytest.mark.parametrize("act", ["none", "relu"])
def test_identity_weight_returns_x(storage, act):
    c = 24
    rng = np.random.default_rng(3)
    x = np.maximum(rng.standard_normal((2, c, 7, 9)), 0).astype(np.float32)
    if storage == "f16":
        x = x.astype(np.float16)
    row_ptr = np.arange(c + 1, dtype=np.int32)
    col_idx = np.arange(c, dtype=np.int32)
    values = np.ones(c, dtype=np.float32)
    y, _, _ = oracle.spconv_ref(c, c, 1, row_ptr, col_idx, values, np.zeros(c, np.float32), act, x,
                                storage=storage)
    assert y.dtype == x.dtype and np.array_equal(y.view(np.uint8), x.view(np.uint8))


@pytest.mark.parametrize("storage", ["f32", "f16"])
@pytest.mark.parametrize("act", ["none", "relu", "relu6"])
@pytest.mark.parametrize("k", [1, 2, 4])
def test_all_zero_weight_gives_act_bias(storage, act, k):
    layer = make_layer(16, 32, 5, 5, 2, 1.0, block_rows=k, storage=storage, act=act, seed=9)
    layer.bias[:4] = np.float32([7.5, -3.0, 0.0, 6.0])
    assert layer.nnz == 0
    y, _, _ = oracle.spconv_ref_layer(layer)
    expect = _act(layer.bias.astype(np.float64), act).astype(y.dtype)
    assert np.array_equal(y, np.broadcast_to(expect[None, :, None, None], y.shape))


@pytest.mark.parametrize("k", [1, 2, 4])
def test_power_of_two_scaling(k):
    layer = make_layer(32, 64, 6, 6, 2, 0.7, block_rows=k, act="none", seed=11)
    y, y64, _ = oracle.spconv_ref_layer(layer)
    layer.values = layer.values * np.float32(2)
    layer.bias = layer.bias * np.float32(2)
    y2, y642, _ = oracle.spconv_ref_layer(layer)
    assert np.array_equal(y642, 2 * y64)
    assert np.array_equal(y2, 2 * y)


@pytest.mark.parametrize("k", [2, 4])
@pytest.mark.parametrize("storage", ["f32", "f16"])
def test_blocked_equals_expanded_csr(storage, k):
    layer = make_layer(40, 48, 4, 7, 2, 0.8, block_rows=k, storage=storage, act="relu6", seed=21)
    rp, ci, va = expand_blocks_to_csr(48, k, layer.row_ptr, layer.col_idx, layer.values)
    _, y64b, sb = oracle.spconv_ref_layer(layer)
    _, y64c, sc = oracle.spconv_ref(48, 40, 1, rp, ci, va, layer.bias, "relu6", layer.x, storage=storage)
    assert np.array_equal(y64b, y64c) and np.array_equal(sb, sc)
    # every block row of the expansion shares one column pattern
    for rb in range(48 // k):
        pats = [tuple(ci[rp[k * rb + i]:rp[k * rb + i + 1]]) for i in range(k)]
        assert len(set(pats)) == 1


def test_row_permutation_permutes_output():
    layer = make_layer(20, 30, 5, 4, 2, 0.6, act="relu", seed=31)
    perm = np.random.default_rng(0).permutation(30)
    rp, ci, va = [0], [], []
    for r in perm:
        s, e = layer.row_ptr[r], layer.row_ptr[r + 1]
        ci.extend(layer.col_idx[s:e])
        va.extend(layer.values[s:e])
        rp.append(len(ci))
    _, y64, _ = oracle.spconv_ref_layer(layer)
    _, y64p, _ = oracle.spconv_ref(30, 20, 1, rp, ci, va, layer.bias[perm], "relu", layer.x)
    assert np.array_equal(y64p, y64[:, perm])


def test_batch_split():
    layer = make_layer(16, 24, 7, 7, 3, 0.9, act="relu6", seed=41)
    _, y64, _ = oracle.spconv_ref_layer(layer)
    parts = [oracle.spconv_ref_layer(layer, x=layer.x[i:i + 1])[1] for i in range(3)]
    assert np.array_equal(np.concatenate(parts), y64)


@pytest.mark.parametrize("act", ["none", "relu", "relu6"])
def test_single_nonzero_per_row(act):
    cin, cout = 16, 32
    rng = np.random.default_rng(7)
    cols = rng.integers(0, cin, size=cout).astype(np.int32)
    vals = (rng.standard_normal(cout) * 3).astype(np.float32)
    bias = rng.standard_normal(cout).astype(np.float32)
    x = np.maximum(rng.standard_normal((2, cin, 3, 5)), 0).astype(np.float32) * 4
    y, y64, _ = oracle.spconv_ref(cout, cin, 1, np.arange(cout + 1, dtype=np.int32), cols, vals,
                                  bias, act, x)
    xr = x.astype(np.float64)[:, cols]                      # [n, cout, h, w]
    prod = vals.astype(np.float64)[None, :, None, None] * xr  # one rounding
    expect = _act(prod + bias.astype(np.float64)[None, :, None, None], act)  # one more
    assert np.array_equal(y64, expect)


def test_half_decoder_all_patterns():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ref = bits.view(np.float16).astype(np.float64)
    got = np.array([oracle.half_to_double(int(b)) for b in bits])
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(ref[~nan]))


def test_out_of_range_column_rejected():
    with pytest.raises(ValueError):
        oracle.spconv_ref(2, 3, 1, [0, 1, 1], [3], [1.0], None, "none", np.ones((1, 3, 2), np.float32))


def test_tolerance_formula():
    y = np.array([1.0, -2.0, 0.0])
    s = np.array([10.0, 0.0, 5.0])
    assert np.allclose(oracle.tolerance(y, s, "f32"), [1e-4 + 1e-6, 1e-6, 5e-5 + 1e-6])
    assert np.allclose(oracle.tolerance(y, s, "f16"), [2e-3 + 1e-4 + 1e-6, 4e-3 + 1e-6, 5e-5 + 1e-6])


FP16_GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "fp16_rounding.json")


@pytest.mark.parametrize("case", json.load(open(FP16_GOLDEN))["cases"], ids=lambda c: c["name"])
def test_fp16_output_rounds_once_to_nearest_even(case):
    """The oracle's fp16 result is the exact sum rounded once to binary16,
    ties to even: hand-derived bit patterns (tests/golden/fp16_rounding.json)
    that double rounding through fp32, truncation or ties-away would miss."""
    vals = np.array([float.fromhex(v) for v in case["values"]], np.float32)
    xs = np.array([float.fromhex(v) for v in case["x"]], np.float64)
    assert np.array_equal(xs.astype(np.float16).astype(np.float64), xs), "inputs must be fp16 values"
    cin = len(vals)
    x = xs.astype(np.float16).reshape(1, cin, 1, 1)
    y, y64, _ = oracle.spconv_ref(1, cin, 1, np.array([0, cin], np.int32), np.arange(cin, dtype=np.int32), vals,
                                  None, "none", x, storage="f16")
    assert y.dtype == np.float16
    assert int(y.reshape(-1).view(np.uint16)[0]) == int(case["y_bits"], 16), (
        case["name"], float(y64.reshape(-1)[0]).hex(), hex(int(y.reshape(-1).view(np.uint16)[0])))
