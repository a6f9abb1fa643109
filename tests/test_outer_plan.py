"""Host-only checks of the lockstep kernel's records (no GPU).

Plans of 1 x 4 blocks with at most 632 input channels (matrix mode) and
unstructured fp32 plans with at most 1264 (vector mode; 16-column tiles
above 632) are laid out again for the lockstep kernel: sets of block rows
in lockstep, per weight slot and quad of steps the weights, per lane group
and quad the LDS channel offsets, padding steps that read the zero row with
weight 0, and wave lists per tile parity.  Walking the records back into
block-CSR with the kernel's own bookkeeping (spconv_plan_unpack_outer, which
also checks the padding, ascending channels, offsets and wave lists) must
return the input exactly; plans the kernel cannot take carry no records, and
asking for the kernel there is refused.
"""

import numpy as np
import pytest

import paper_1911_09723_amd as sp
from synth import make_layer

E_FORMAT, E_UNSUPPORTED = 2, 4


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
    # (cin, cout, sparsity, kc); block_rows 4
    (512, 512, 0.9, 1),       # the 1x4 headline layer: 16 octs, one per wavefront and tile
    (512, 512, 0.7, 1),
    (632, 96, 0.9, 1),        # widest input; 3 octs, the last one partial
    (17, 20, 0.5, 1),         # cin not a multiple of 8, one partial oct of 5 block rows
    (200, 1024, 0.95, 1),     # 32 octs: two per wavefront per tile
    (130, 64, 0.0, 1),        # dense
    (64, 48, 1.0, 1),         # no stored blocks: every step is padding
    (256, 128, 0.8, 2),       # 4x2 blocks expanded to single channels
]

F16_CASES = [(320, 1280, 0.9), (40, 240, 0.9)]

VECTOR_CASES = [
    # (cin, cout, sparsity, kc); unstructured (block_rows 1)
    (512, 512, 0.9, 1),       # 32-column tiles, 64 sets of 8 rows
    (1024, 1024, 0.9, 1),     # 16-column tiles, sets of 16 rows
    (1264, 40, 0.8, 1),       # widest input, a partial set
    (17, 20, 0.5, 1),
    (64, 48, 1.0, 1),         # no stored blocks
    (256, 128, 0.9, 4),       # 4x1 input-channel blocks expanded to single channels
]


@pytest.mark.parametrize("case", VECTOR_CASES, ids=lambda c: "%d-%d-s%g-kc%d" % c)
def test_vector_mode_records_unpack_to_the_input(case):
    cin, cout, s, kc = case
    layer = make_layer(cin, cout, 1, 1, 1, s, block_rows=1, block_cols=kc, seed=cin + cout + 7, with_x=False)
    h = _host_plan(layer)
    try:
        rp, ci, va = sp.spconv_plan_unpack_outer(h)
        assert np.array_equal(rp, layer.row_ptr)
        assert np.array_equal(ci, layer.col_idx)
        assert np.array_equal(va.view(np.uint32), layer.values.view(np.uint32))
    finally:
        sp.spconv_destroy(h)


@pytest.mark.parametrize("case", CASES, ids=lambda c: "%d-%d-s%g-kc%d" % c)
def test_records_unpack_to_the_input(case):
    cin, cout, s, kc = case
    layer = make_layer(cin, cout, 1, 1, 1, s, block_rows=4, block_cols=kc, seed=cin + cout, with_x=False)
    h = _host_plan(layer)
    try:
        rp, ci, va = sp.spconv_plan_unpack_outer(h)
        assert np.array_equal(rp, layer.row_ptr)
        assert np.array_equal(ci, layer.col_idx)
        assert np.array_equal(va.view(np.uint32), layer.values.view(np.uint32))
    finally:
        sp.spconv_destroy(h)


@pytest.mark.parametrize("case", F16_CASES, ids=lambda c: "%d-%d-s%g" % c)
def test_fp16_records_hold_the_rounded_weights(case):
    """fp16 storage: the records carry each weight rounded once to fp16."""
    cin, cout, s = case
    layer = make_layer(cin, cout, 1, 1, 1, s, block_rows=4, storage="f16", seed=cin, with_x=False)
    h = _host_plan(layer)
    try:
        rp, ci, va = sp.spconv_plan_unpack_outer(h)
        assert np.array_equal(rp, layer.row_ptr)
        assert np.array_equal(ci, layer.col_idx)
        want = layer.values.astype(np.float16).astype(np.float32)
        assert np.array_equal(va.view(np.uint32), want.view(np.uint32))
    finally:
        sp.spconv_destroy(h)


@pytest.mark.parametrize("case", [(64, 64, 0.8, 2, "f32"), (640, 64, 0.9, 4, "f32"), (1280, 64, 0.9, 1, "f32"),
                                  (64, 64, 0.8, 1, "f16")],
                         ids=["k2", "k4-cin640", "k1-cin1280", "k1-f16"])
def test_plans_the_kernel_cannot_take(case):
    cin, cout, s, k, st = case
    layer = make_layer(cin, cout, 1, 1, 1, s, block_rows=k, storage=st, seed=5, with_x=False)
    h = _host_plan(layer)
    try:
        with pytest.raises(sp.SpconvError) as e:
            sp.spconv_plan_unpack_outer(h)
        assert e.value.args[0].startswith("SPCONV_E_FORMAT")
    finally:
        sp.spconv_destroy(h)
    with pytest.raises(sp.SpconvError) as e:
        _host_plan(layer, kernel=4)
    assert e.value.args[0].startswith("SPCONV_E_UNSUPPORTED")
