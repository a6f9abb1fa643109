"""Host-side checks of the fused depthwise 3x3 -> sparse 1x1 entry point (no GPU).

Plans are created with host_only = 1, so only the argument checks, the
planner and the packed image are exercised."""

import numpy as np
import pytest

import paper_1911_09723_amd as sp
from synth import make_layer, make_depthwise


def _opts(**kw):
    o = sp.spconv_options_init()
    o.host_only = 1
    for k, v in kw.items():
        setattr(o, k, v)
    return o


def _fused(layer, kw, kb=None, dw_act="relu6", stride=1, storage="f32", options=None):
    return sp.spconv_plan_create_fused(layer.cout, layer.cin, layer.block_rows, layer.row_ptr, layer.col_idx,
                                       layer.values, layer.bias, layer.act, kw, kb, dw_act, stride, storage,
                                       options=options or _opts(), check=False)


def _status(layer, kw, kb=None, **a):
    st, h = _fused(layer, kw, kb, **a)
    if h:
        sp.spconv_destroy(h)
    return st, sp.spconv_last_error()


@pytest.mark.parametrize("k", [1, 2, 4])
@pytest.mark.parametrize("stride", [1, 2])
def test_fused_host_plan(k, stride):
    layer = make_layer(96, 128, 2, 2, 1, 0.8, block_rows=k, act="relu", seed=3, with_x=False)
    kw, kb = make_depthwise(96, 4)
    st, h = _fused(layer, kw, kb, dw_act="relu6", stride=stride)
    assert st == sp.spconv.OK, sp.spconv_last_error()
    try:
        info = sp.spconv_plan_get_info(h)
        assert info["dw_stride"] == stride and info["dw_act"] == sp.spconv.ACT_RELU6
        assert info["kernel"] == 0 and info["pipe_sets"] == 0 and info["regions"] == 0
        rp, ci, va, _ = sp.spconv_plan_unpack(h)
        assert np.array_equal(rp, layer.row_ptr) and np.array_equal(ci, layer.col_idx)
        assert np.array_equal(va, layer.values)
        with pytest.raises(sp.SpconvError) as e:
            sp.spconv_plan_unpack_interleaved(h)
        assert e.value.status == sp.spconv.E_FORMAT
    finally:
        sp.spconv_destroy(h)


def test_plain_plan_reports_no_depthwise_stage():
    layer = make_layer(32, 64, 2, 2, 1, 0.8, seed=1, with_x=False)
    h = sp.spconv_plan_create(layer.cout, layer.cin, 1, layer.row_ptr, layer.col_idx, layer.values, layer.bias,
                              "relu", "f32", options=_opts())
    try:
        info = sp.spconv_plan_get_info(h)
        assert info["dw_stride"] == 0 and info["pipe_sets"] >= 1
    finally:
        sp.spconv_destroy(h)


def test_fused_arguments_checked():
    layer = make_layer(32, 64, 2, 2, 1, 0.8, seed=1, with_x=False)
    kw, kb = make_depthwise(32, 2)
    E = sp.spconv
    for stride in (0, 3, -1):
        st, msg = _status(layer, kw, kb, stride=stride)
        assert st == E.E_ARG and "dw_stride" in msg
    st, msg = _status(layer, None, kb)
    assert st == E.E_ARG and "dw_weights" in msg
    st, msg = _status(layer, kw, kb, dw_act=7)
    assert st == E.E_ARG and "dw_act" in msg
    st, msg = _status(layer, kw, kb, storage="f16")
    assert st == E.E_UNSUPPORTED and "fp32" in msg
    st, msg = _status(layer, kw, kb, options=_opts(kernel=2))
    assert st == E.E_UNSUPPORTED and "strip" in msg
    for o in (dict(pipe_sets=1), dict(regions=2)):
        st, msg = _status(layer, kw, kb, options=_opts(**o))
        assert st == E.E_UNSUPPORTED and "pipelined" in msg
    bad = kw.copy()
    bad[5, 2, 1] = np.nan
    st, msg = _status(layer, bad, kb)
    assert st == E.E_FORMAT and "dw_weights[5][2][1]" in msg
    badb = kb.copy()
    badb[7] = np.inf
    st, msg = _status(layer, kw, badb)
    assert st == E.E_FORMAT and "dw_bias[7]" in msg
    # a strip of 700 channels does not fit in LDS: no depthwise stage without it
    wide = make_layer(700, 16, 2, 2, 1, 0.9, seed=5, with_x=False)
    kw7, _ = make_depthwise(700, 6)
    st, msg = _status(wide, kw7)
    assert st == E.E_UNSUPPORTED and "LDS" in msg
    # the 1x1's own checks still apply
    layer.row_ptr = layer.row_ptr.copy()
    layer.row_ptr[0] = 1
    st, _ = _status(layer, kw, kb)
    assert st == E.E_FORMAT


def test_fused_bias_optional_and_out_null():
    layer = make_layer(16, 16, 2, 2, 1, 0.5, seed=8, with_x=False)
    kw, _ = make_depthwise(16, 9)
    st, h = _fused(layer, kw, None)
    assert st == sp.spconv.OK
    sp.spconv_destroy(h)
    lib = sp.load_library()
    rc = lib.spconv_plan_create_fused(None, 16, 16, 1, None, None, None, None, 0, None, None, 0, 1, 0, None)
    assert rc == sp.spconv.E_ARG


def test_out_hw():
    layer = make_layer(8, 8, 2, 2, 1, 0.5, seed=8, with_x=False)
    kw, _ = make_depthwise(8, 9)
    p = sp.Plan.__new__(sp.Plan)
    p.handle, p.dw_stride = None, 2
    assert p.out_hw(14, 14) == (7, 7) and p.out_hw(15, 1) == (8, 1) and p.out_hw(0, 5) == (0, 3)
    p.dw_stride = 1
    assert p.out_hw(13, 7) == (13, 7)
