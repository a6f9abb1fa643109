"""Host-only checks of the register-indexed kernel's streams (no GPU).

The planner lays every fp32 plan out a second time for the register-indexed
kernel: slot records per channel chunk with batch flags and ring offsets, and
row-pair entries for the columns left after the whole tiles.  Walking both
back into block-CSR with the kernel's own bookkeeping
(spconv_plan_unpack_indexed) must return the input exactly, for every block
shape, density and ragged size; malformed options are refused.
"""

import numpy as np
import pytest

import paper_1911_09723_amd as sp
from paper_1911_09723_amd import spconv as spmod
from synth import make_layer

E_ARG = 1  # SPCONV_E_ARG


def _host_plan(layer, **kw):
    o = sp.spconv_options_init()
    o.host_only = 1
    for k, v in kw.items():
        setattr(o, k, v)
    if getattr(layer, "block_cols", 1) > 1:
        return sp.spconv_plan_create_blocked(layer.cout, layer.cin, layer.block_rows, layer.block_cols,
                                             layer.row_ptr, layer.col_idx, layer.values, layer.bias, layer.act,
                                             layer.storage, options=o)
    return sp.spconv_plan_create(layer.cout, layer.cin, layer.block_rows, layer.row_ptr, layer.col_idx,
                                 layer.values, layer.bias, layer.act, layer.storage, options=o)


CASES = [
    # (cin, cout, sparsity, k, kc)
    (512, 512, 0.9, 1, 1),
    (512, 512, 0.9, 4, 1),
    (512, 512, 0.7, 2, 1),
    (96, 160, 0.95, 1, 1),     # most chunks of a slot empty: one weight-0 batch each
    (17, 20, 0.5, 1, 1),       # one ragged chunk, two slots, cout not a multiple of 16
    (200, 52, 0.85, 4, 1),     # ragged last chunk, a partial last slot
    (130, 64, 0.0, 1, 1),      # dense: records of 3 blocks everywhere
    (64, 48, 1.0, 1, 1),       # no stored blocks at all
    (256, 128, 0.9, 1, 4),     # 4x1 blocks, expanded to single channels
    (256, 128, 0.8, 2, 2),     # 2x2 blocks
]


@pytest.mark.parametrize("from_pairs", [False, True], ids=["records", "pairs"])
@pytest.mark.parametrize("case", CASES, ids=lambda c: "%d-%d-s%g-k%d-kc%d" % c)
def test_streams_unpack_to_the_input(case, from_pairs):
    cin, cout, s, k, kc = case
    layer = make_layer(cin, cout, 1, 1, 1, s, block_rows=k, block_cols=kc, seed=cin + cout, with_x=False)
    h = _host_plan(layer)
    try:
        rp, ci, va = sp.spconv_plan_unpack_indexed(h, from_pairs=from_pairs)
        assert np.array_equal(rp, layer.row_ptr)
        assert np.array_equal(ci, layer.col_idx)
        assert np.array_equal(va.view(np.uint32), layer.values.view(np.uint32))
    finally:
        sp.spconv_destroy(h)


def test_empty_rows_and_whole_empty_slot():
    layer = make_layer(160, 64, 1, 1, 1, 1.0, seed=3, with_x=False)
    rng = np.random.default_rng(3)
    rp, ci = [0], []
    for r in range(64):
        cols = [] if (r >= 48 or r % 5 == 0) else sorted(rng.choice(np.arange(32, 64), 3, replace=False).tolist())
        ci += cols
        rp.append(len(ci))
    layer.row_ptr = np.asarray(rp, np.int32)
    layer.col_idx = np.asarray(ci, np.int32)
    layer.values = rng.standard_normal(len(ci)).astype(np.float32)
    h = _host_plan(layer)
    try:
        for from_pairs in (False, True):
            rp2, ci2, va2 = sp.spconv_plan_unpack_indexed(h, from_pairs=from_pairs)
            assert np.array_equal(rp2, layer.row_ptr) and np.array_equal(ci2, layer.col_idx)
            assert np.array_equal(va2, layer.values)
    finally:
        sp.spconv_destroy(h)


def test_fp16_and_depthwise_plans_have_no_indexed_streams():
    layer = make_layer(64, 64, 1, 1, 1, 0.8, storage="f16", seed=4, with_x=False)
    h = _host_plan(layer)
    try:
        with pytest.raises(sp.SpconvError, match="E_FORMAT"):
            sp.spconv_plan_unpack_indexed(h)
    finally:
        sp.spconv_destroy(h)


@pytest.mark.parametrize("opts,status", [
    (dict(kernel=3, lane_cols=7), "E_ARG"),
    (dict(kernel=3, lane_cols=-1), "E_ARG"),
    (dict(kernel=6), "E_ARG"),
])
def test_bad_indexed_options_are_refused(opts, status):
    layer = make_layer(64, 64, 1, 1, 1, 0.8, seed=5, with_x=False)
    with pytest.raises(sp.SpconvError, match=status):
        sp.spconv_destroy(_host_plan(layer, **opts))


def test_indexed_kernel_refuses_fp16():
    layer = make_layer(64, 64, 1, 1, 1, 0.8, storage="f16", seed=6, with_x=False)
    with pytest.raises(sp.SpconvError, match="E_UNSUPPORTED"):
        sp.spconv_destroy(_host_plan(layer, kernel=3))


def test_error_word_calls_validate_their_arguments():
    layer = make_layer(64, 64, 1, 1, 1, 0.8, seed=7, with_x=False)
    h = _host_plan(layer)
    lib = spmod.load_library()
    try:
        st, _ = sp.spconv_plan_check(h, check=False)
        assert st == E_ARG          # a host-only plan has no device word
        assert sp.spconv_plan_set_wait_limit(h, -1, check=False) == E_ARG
        assert sp.spconv_plan_set_wait_limit(h, 0, check=False) == 0
        assert lib.spconv_plan_set_wait_limit(None, 5) == E_ARG
        assert lib.spconv_plan_check(None, None, 0) == E_ARG
    finally:
        sp.spconv_destroy(h)
