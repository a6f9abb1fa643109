"""The oracle's pins catch plausible mistakes (no GPU).

Each case plants one mistake in a copy of the oracle's C source (a wrong sign,
a dropped term, a wrong index, a transposed operand, a missing clamp, a wrong
binary16 decoding step), builds it with gcc into a temporary directory, and
checks that the pin battery below rejects it.  The unmodified source must pass
the same battery.
"""

import json
import os
import subprocess

import numpy as np
import pytest

import oracle
from synth import make_layer, densify
from blocks_util import dense_from_blocks, random_blocks

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle", "spconv_ref.c")
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")

MUTANTS = {
    "sign_of_term": ("acc[p] += prod;", "acc[p] -= prod;"),
    "block_value_index": ("values[((int64_t)t * k + i) * kc + j]", "values[((int64_t)t * k) * kc + j]"),
    "bias_index": ("(double)bias[r]", "(double)bias[rb]"),
    "x_transposed": ("(img * cin + c) * hw", "(c * n + img) * hw"),
    "dropped_first_term": ("t = row_ptr[rb]; t < row_ptr[rb + 1]", "t = row_ptr[rb] + 1; t < row_ptr[rb + 1]"),
    "dropped_bias": ("apply_act(acc[p] + b, act)", "apply_act(acc[p], act)"),
    "relu_unclamped": ("return v > 0.0 ? v : 0.0;", "return v;"),
    "relu6_unclamped": ("return v < 6.0 ? v : 6.0;", "return v;"),
    "scale_signed": ("s[p] += fabs(prod);", "s[p] += prod;"),
    "block_row_order": ("const int32_t r = rb * k + i;", "const int32_t r = rb + i * rows;"),
    "half_exponent_bias": ("expo - 25", "expo - 24"),
    "half_implicit_bit": ("(frac | 0x400)", "frac"),
    "half_subnormal_scale": ("ldexp((double)frac, -24)", "ldexp((double)frac, -25)"),
    "dw_tap_row_offset": ("spconv_ref_dw3x3", "oy * stride + dy - 1", "oy * stride + dy"),
    "dw_column_stride": ("spconv_ref_dw3x3", "ox * stride + dx - 1", "ox + dx - 1"),
    "dw_bias_dropped": ("spconv_ref_dw3x3", "d[o] = apply_act(acc + b, act);", "d[o] = apply_act(acc, act);"),
    "dw_kernel_transposed": ("spconv_ref_dw3x3", "kc[dy * 3 + dx]", "kc[dx * 3 + dy]"),
    "dw_scale_signed": ("spconv_ref_dw3x3", "            s += fabs(prod);", "            s += prod;"),
    "dw_border_taps_kept": ("spconv_ref_dw3x3", "if (ix < 0 || ix >= w)", "if (ix < 0 || ix > w)"),
    "input_scale_dropped": ("s[p] += fabs(wv) * xs[xrow + p];", "s[p] += 0.0;"),
    # input-channel blocks
    "input_block_channel": ("const int64_t c = (int64_t)col_idx[t] + j;", "const int64_t c = (int64_t)col_idx[t];"),
    "input_block_value_order": ("values[((int64_t)t * k + i) * kc + j]", "values[((int64_t)t * k + i) * kc + (kc - 1 - j)]"),
    "input_block_last_dropped": ("for (int32_t j = 0; j < kc; ++j)", "for (int32_t j = 0; j + 1 < kc; ++j)"),
    # the network-level stages: (function, anchor inside it, replacement)
    "dw64_tap_row_offset": ("spconv_ref_dw3x3_f64", "oy * stride + dy - 1", "oy * stride + dy"),
    "dw64_input_scale_dropped": ("spconv_ref_dw3x3_f64", "s += fabs(kv) * xs[plane + iy * w + ix];", "s += 0.0;"),
    "stem_tap_transposed": ("spconv_ref_conv3x3_hwc", "(int64_t)o * 9 + dy * 3 + dx", "(int64_t)o * 9 + dx * 3 + dy"),
    "stem_hwc_channel_stride": ("spconv_ref_conv3x3_hwc", "((img * h + iy) * w + ix) * cin + i",
                                "((img * h + iy) * w + ix) + i"),
    "stem_padding_shift": ("spconv_ref_conv3x3_hwc", "ox * stride + dx - 1", "ox * stride + dx"),
    "stem_bias_dropped": ("spconv_ref_conv3x3_hwc", "y[q] = apply_act(acc + b, act);", "y[q] = apply_act(acc, act);"),
    "gap_drops_last": ("spconv_ref_gap", "p < hw; ++p", "p < hw - 1; ++p"),
    "gap_divisor": ("spconv_ref_gap", "acc / (double)hw", "acc / (double)(hw + 1)"),
    "gap_input_scale_dropped": ("spconv_ref_gap", "s += xs[(img * c + ch) * hw + p];", "s += 0.0;"),
}


def _mutate(source, mutant):
    """Apply one planted mistake: (anchor, replacement), the anchor unique in
    the file, or (function, anchor, replacement), unique in that function."""
    if len(mutant) == 2:
        before, after = mutant
        assert source.count(before) == 1, "mutation anchor not found exactly once: " + before
        return source.replace(before, after)
    func, before, after = mutant
    start = source.index("\nint " + func + "(")
    end = source.index("\n}\n", start)
    body = source[start:end]
    assert body.count(before) == 1, "mutation anchor not found exactly once in %s: %s" % (func, before)
    return source[:start] + body.replace(before, after) + source[end:]


def _act(v, act):
    if act == "relu":
        return np.maximum(v, 0.0)
    if act == "relu6":
        return np.minimum(np.maximum(v, 0.0), 6.0)
    return v


def _battery(lib):
    """Return the names of the pins that fail for this build of the oracle."""
    failed = []
    for case in json.load(open(GOLDEN))["cases"]:
        x = np.asarray(case["x"], dtype=np.float32)[None]
        for act in ("none", "relu", "relu6"):
            _, y64, s = oracle.spconv_ref(case["cout"], case["cin"], case["block_rows"], case["row_ptr"],
                                          case["col_idx"], case["values"], case["bias"], act, x, lib=lib)
            if not np.array_equal(y64[0], np.asarray(case["y_" + act])):
                failed.append("hand:" + case["name"] + ":" + act)
            if not np.array_equal(s[0], np.asarray(case["scale"])):
                failed.append("hand-scale:" + case["name"])
    for k, storage in ((1, "f32"), (2, "f32"), (4, "f32"), (4, "f16")):
        layer = make_layer(12, 16, 3, 5, 2, 0.5, block_rows=k, storage=storage, act="relu6", seed=3)
        _, y64, s = oracle.spconv_ref(layer.cout, layer.cin, k, layer.row_ptr, layer.col_idx,
                                      layer.values, layer.bias, "relu6", layer.x, storage=storage, lib=lib)
        wd = densify(16, 12, k, layer.row_ptr, layer.col_idx, layer.values)
        x64 = layer.x.astype(np.float64).reshape(2, 12, -1)
        ref = _act(np.matmul(wd[None], x64) + layer.bias.astype(np.float64)[None, :, None], "relu6")
        sref = np.matmul(np.abs(wd)[None], np.abs(x64))
        if not np.all(np.abs(y64.reshape(ref.shape) - ref) <= 1e-12 * (sref + 1.0)):
            failed.append("brute:k%d:%s" % (k, storage))
        if not np.allclose(s.reshape(sref.shape), sref, rtol=1e-12, atol=0):
            failed.append("brute-scale:k%d:%s" % (k, storage))
    failed += _dw_battery(lib)
    failed += _net_battery(lib)
    failed += _block_battery(lib)
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ref = bits.view(np.float16).astype(np.float64)
    got = np.array([lib.spconv_ref_half_to_double(int(b)) for b in bits])
    ok = ~np.isnan(ref)
    if not np.array_equal(got[ok], ref[ok]):
        failed.append("half-decoder")
    return failed


def _dw_battery(lib):
    """Pins of the depthwise stage and the fused path: torch's grouped conv2d in
    fp64 (an independent library routine) for the outputs and, on absolute
    values, for the scale; the fused output against densified W applied to it."""
    import torch
    failed = []
    rng = np.random.default_rng(5)
    for stride, (h, w) in ((1, (5, 6)), (2, (7, 5)), (2, (6, 6))):
        x = rng.standard_normal((2, 4, h, w)).astype(np.float32)
        k = rng.standard_normal((4, 3, 3)).astype(np.float32)
        b = rng.standard_normal(4).astype(np.float32)
        d, sd = oracle.dw3x3_ref(x, k, b, "none", stride, lib=lib)
        conv = lambda xx, kk, bb: torch.nn.functional.conv2d(  # noqa: E731
            torch.from_numpy(xx).double(), torch.from_numpy(kk).double()[:, None],
            None if bb is None else torch.from_numpy(bb).double(), stride=stride, padding=1, groups=4).numpy()
        ref = conv(x, k, b)
        sref = conv(np.abs(x), np.abs(k), np.abs(b))
        if d.shape != ref.shape or not np.all(np.abs(d - ref) <= 1e-12 * (sref + 1.0)):
            failed.append("dw:s%d" % stride)
        elif not np.allclose(sd, sref, rtol=1e-12, atol=0):
            failed.append("dw-scale:s%d" % stride)
        layer = make_layer(4, 8, 1, 1, 1, 0.5, block_rows=2, act="relu", seed=stride, with_x=False)
        _, y64, s = oracle.fused_ref(8, 4, 2, layer.row_ptr, layer.col_idx, layer.values, layer.bias, "relu",
                                     x, k, b, "none", stride, lib=lib)
        wd = densify(8, 4, 2, layer.row_ptr, layer.col_idx, layer.values)
        d2 = ref.reshape(2, 4, -1)
        yref = _act(np.matmul(wd[None], d2) + layer.bias.astype(np.float64)[None, :, None], "relu")
        syref = np.matmul(np.abs(wd)[None], np.abs(d2)) + np.matmul(np.abs(wd)[None], sref.reshape(2, 4, -1))
        if not np.all(np.abs(y64.reshape(yref.shape) - yref) <= 1e-12 * (syref + 1.0)):
            failed.append("fused:s%d" % stride)
        elif not np.allclose(s.reshape(syref.shape), syref, rtol=1e-12, atol=1e-300):
            failed.append("fused-scale:s%d" % stride)
    return failed


def _block_battery(lib):
    """Input-channel (kc) and 2-D blocks against the dense product."""
    failed = []
    rng = np.random.default_rng(21)
    for kr, kc in ((1, 4), (2, 2), (1, 2), (4, 4)):
        cout, cin = 8, 16
        rp, ci, va = random_blocks(cout, cin, kr, kc, 0.5, rng)
        x = rng.standard_normal((2, cin, 3)).astype(np.float32)
        b = rng.standard_normal(cout).astype(np.float32)
        _, y64, s = oracle.spconv_ref(cout, cin, kr, rp, ci, va, b, "none", x, lib=lib, block_cols=kc)
        wd = dense_from_blocks(cout, cin, kr, kc, rp, ci, va)
        ref = np.einsum("rc,ncp->nrp", wd, x.astype(np.float64)) + b.astype(np.float64)[None, :, None]
        sref = np.einsum("rc,ncp->nrp", np.abs(wd), np.abs(x.astype(np.float64)))
        if not np.allclose(y64, ref, rtol=1e-12, atol=1e-12):
            failed.append("blocks:%dx%d" % (kr, kc))
        elif not np.allclose(s, sref, rtol=1e-12, atol=0):
            failed.append("blocks-scale:%dx%d" % (kr, kc))
    return failed


def _net_battery(lib):
    """Stem convolution, pooling and the double-input depthwise stage against
    torch / numpy in fp64, and the whole chain on 32 x 32 images."""
    import torch
    F = torch.nn.functional
    failed = []
    rng = np.random.default_rng(12)
    x = rng.standard_normal((2, 9, 8, 3)).astype(np.float32)
    wt = rng.standard_normal((4, 3, 3, 3)).astype(np.float32)
    b = rng.standard_normal(4).astype(np.float32)
    for stride in (1, 2):
        y, ys = oracle.conv3x3_hwc_ref(x, wt, b, "none", stride, lib=lib)
        xt = torch.from_numpy(x).double().permute(0, 3, 1, 2)
        wtt = torch.from_numpy(wt).double().permute(0, 3, 1, 2)
        ref = F.conv2d(xt, wtt, torch.from_numpy(b).double(), stride=stride, padding=1).numpy()
        if y.shape != ref.shape or not np.allclose(y, ref, rtol=1e-12, atol=1e-12):
            failed.append("stem:s%d" % stride)
    g = rng.standard_normal((2, 3, 5, 4))
    gs = np.abs(rng.standard_normal(g.shape))
    y, ys = oracle.gap_ref(g, gs, lib=lib)
    if not np.allclose(y, g.mean(axis=(2, 3)), rtol=1e-13, atol=1e-15):
        failed.append("gap")
    if not np.allclose(ys, (np.abs(g) + gs).mean(axis=(2, 3)), rtol=1e-13, atol=0):
        failed.append("gap-scale")
    d = rng.standard_normal((1, 3, 7, 6))
    ds = np.abs(rng.standard_normal(d.shape))
    k = rng.standard_normal((3, 3, 3)).astype(np.float32)
    for stride in (1, 2):
        o, os_ = oracle.dw3x3_ref64(d, ds, k, None, "none", stride, lib=lib)
        kt = torch.from_numpy(k).double()[:, None]
        ref = F.conv2d(torch.from_numpy(d), kt, None, stride=stride, padding=1, groups=3).numpy()
        sref = F.conv2d(torch.from_numpy(np.abs(d) + ds), kt.abs(), None, stride=stride, padding=1,
                        groups=3).numpy()
        if o.shape != ref.shape or not np.allclose(o, ref, rtol=1e-12, atol=1e-12):
            failed.append("dw64:s%d" % stride)
        elif not np.allclose(os_, sref, rtol=1e-12, atol=0):
            failed.append("dw64-scale:s%d" % stride)
    return failed


def _build(tmp_path, name, source):
    src = tmp_path / (name + ".c")
    so = tmp_path / ("lib" + name + ".so")
    src.write_text(source)
    subprocess.check_call(["gcc", "-O1", "-fopenmp", "-ffp-contract=off", "-fPIC", "-shared",
                           "-o", str(so), str(src), "-lm"])
    return oracle.load_library(str(so))


def test_unmodified_oracle_passes_battery(tmp_path):
    lib = _build(tmp_path, "pristine", open(SRC).read())
    assert _battery(lib) == []


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(tmp_path, name):
    lib = _build(tmp_path, name, _mutate(open(SRC).read(), MUTANTS[name]))
    assert _battery(lib), "planted mistake %r passed every pin" % name
