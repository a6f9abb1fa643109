"""Host-side checks of weight blocks over input channels (no GPU): planning
with host_only = 1, round trips through the packed streams, errors."""

import numpy as np
import pytest

import paper_1911_09723_amd as sp
from blocks_util import random_blocks


def _opts(**kw):
    o = sp.spconv_options_init()
    o.host_only = 1
    for k, v in kw.items():
        setattr(o, k, v)
    return o


def _create(cout, cin, kr, kc, rp, ci, va, check=False, **opts):
    return sp.spconv_plan_create_blocked(cout, cin, kr, kc, rp, ci, va, None, "relu", "f32", options=_opts(**opts),
                                         check=check)


@pytest.mark.parametrize("kr,kc", [(1, 4), (2, 2), (1, 2), (4, 4), (2, 4), (4, 1)])
@pytest.mark.parametrize("opts", [dict(), dict(kernel=2), dict(group_lanes=16, reorder=0)])
def test_round_trip(kr, kc, opts):
    rng = np.random.default_rng(kr * 7 + kc)
    cout, cin = 64, 96
    rp, ci, va = random_blocks(cout, cin, kr, kc, 0.3, rng)
    h = _create(cout, cin, kr, kc, rp, ci, va, check=True, **opts)
    try:
        info = sp.spconv_plan_get_info(h)
        assert info["block_cols"] == kc and info["block_rows"] == kr and info["nnzb"] == len(ci)
        rp2, ci2, va2, _ = sp.spconv_plan_unpack(h)
        assert np.array_equal(rp2, rp) and np.array_equal(ci2, ci) and np.array_equal(va2, va)
        if info["kernel"] == 0:
            rp3, ci3, va3 = sp.spconv_plan_unpack_interleaved(h)
            assert np.array_equal(rp3, rp) and np.array_equal(ci3, ci) and np.array_equal(va3, va)
    finally:
        sp.spconv_destroy(h)


def test_unaligned_blocks_are_accepted():
    rp = np.array([0, 2], np.int32)
    ci = np.array([1, 6], np.int32)  # channels 1..4 and 6..9
    va = np.arange(8, dtype=np.float32)
    st, h = _create(1, 10, 1, 4, rp, ci, va)
    assert st == sp.spconv.OK
    sp.spconv_destroy(h)


@pytest.mark.parametrize("ci,expect,words", [
    ([4, 6], sp.spconv.E_FORMAT, "overlap"),     # second block starts inside the first
    ([0, 8], sp.spconv.E_FORMAT, "outside"),     # channels 8..11 past cin = 10
    ([-1, 4], sp.spconv.E_FORMAT, "outside"),
])
def test_bad_blocks_rejected(ci, expect, words):
    rp = np.array([0, 2], np.int32)
    st, h = _create(1, 10, 1, 4, rp, np.array(ci, np.int32), np.ones(8, np.float32))
    assert h is None and st == expect and words in sp.spconv_last_error()


def test_block_cols_checked():
    rp = np.array([0, 1], np.int32)
    for kc, expect in ((3, sp.spconv.E_UNSUPPORTED), (8, sp.spconv.E_UNSUPPORTED), (0, sp.spconv.E_ARG),
                       (-2, sp.spconv.E_ARG)):
        st, h = _create(1, 16, 1, kc, rp, np.array([0], np.int32), np.ones(8, np.float32))
        assert h is None and st == expect, kc


def test_non_finite_block_value_rejected():
    rp = np.array([0, 1], np.int32)
    va = np.ones(4, np.float32)
    va[3] = np.nan
    st, h = _create(1, 8, 1, 4, rp, np.array([4], np.int32), va)
    assert st == sp.spconv.E_FORMAT and "values[3]" in sp.spconv_last_error()


from hypothesis import given, settings, strategies as st


@settings(max_examples=60, deadline=None)
@given(kr=st.sampled_from([1, 2, 4]), kc=st.sampled_from([1, 2, 4]), rows=st.integers(1, 40),
       bcols=st.integers(1, 40), density=st.floats(0.0, 1.0), seed=st.integers(0, 2 ** 31 - 1),
       kernel=st.sampled_from([0, 2]))
def test_blocked_round_trip_property(kr, kc, rows, bcols, density, seed, kernel):
    """Any aligned block pattern survives planning and unpacking unchanged."""
    rng = np.random.default_rng(seed)
    cout, cin = rows * kr, bcols * kc
    rp, ci, va = random_blocks(cout, cin, kr, kc, density, rng)
    h = _create(cout, cin, kr, kc, rp, ci, va, check=True, kernel=kernel)
    try:
        rp2, ci2, va2, perm = sp.spconv_plan_unpack(h)
        assert np.array_equal(rp2, rp) and np.array_equal(ci2, ci) and np.array_equal(va2, va)
        assert sorted(perm.tolist()) == list(range(rows))
    finally:
        sp.spconv_destroy(h)


def test_oracle_layer_helper_reads_block_cols():
    """oracle.spconv_ref_layer on a layer with input-channel blocks applies them."""
    import oracle
    from synth import make_layer
    layer = make_layer(16, 8, 3, 3, 2, 0.5, block_rows=2, block_cols=4, seed=4)
    _, a, _ = oracle.spconv_ref_layer(layer)
    _, b, _ = oracle.spconv_ref(8, 16, 2, layer.row_ptr, layer.col_idx, layer.values, layer.bias, layer.act,
                                layer.x, block_cols=4)
    assert np.array_equal(a, b)
