"""GPU parity of split rows: a row more than twice the median length (and at
least 32 nonzeros) is packed as two pieces, its even and its odd nonzeros, in
neighbouring lane groups whose partial sums are added before the epilogue.

Each case is compared with the oracle at the stated fp32 tolerance, and the
LDS-strip kernel bit for bit with the direct-load kernel at the same lane-group
width: the two share the packing, so they split the same rows and add the
pieces in the same order (the split decision depends on the layout, so at
different widths they may split differently)"""

import numpy as np
import pytest

from paper_1911_09723_amd import Plan
from synth import make_layer
from gpu_util import gpu_run, assert_parity, note

pytestmark = pytest.mark.gpu

# (cin, cout, h, w, n, sparsity, act, group_lanes): heavy-tailed (beta) rows,
# every lane-group width (the pieces' vectors differ by one rotation step),
# whole tiles and a ragged last tile, H*W a multiple of 4 and not
CASES = [
    (144, 24, 56, 56, 2, 0.85, "relu6", 16),
    (256, 48, 9, 9, 3, 0.85, "none", 4),
    (192, 32, 28, 28, 4, 0.85, "relu", 8),
    (192, 32, 28, 28, 4, 0.85, "relu", 16),
    (576, 96, 14, 14, 3, 0.85, "relu6", 8),
    (320, 40, 7, 7, 5, 0.85, "relu", 16),
]


@pytest.mark.parametrize("spec", CASES, ids=lambda s: "%d-%d-%dx%d-n%d-s%g-%s-g%d" % s)
def test_split_rows_match_oracle_and_direct_kernel(spec):
    cin, cout, h, w, n, s, act, g = spec
    layer = make_layer(cin, cout, h, w, n, s, pattern="beta", act=act, seed=cin * 7 + cout + g)
    plan = Plan.from_layer(layer, kernel=1, group_lanes=g)
    try:
        assert plan.info()["split_rows"] > 0, "the case must split at least one row"
    finally:
        plan.close()
    note("split rows %s" % (spec,))
    y1 = gpu_run(layer, kernel=1, group_lanes=g)
    assert_parity(layer, y1, what="split %s" % (spec,))
    y2 = gpu_run(layer, kernel=2, group_lanes=g)
    assert np.array_equal(y1.view(np.uint32), y2.view(np.uint32))


def test_uniform_rows_are_not_split():
    layer = make_layer(512, 512, 14, 14, 1, 0.9, act="relu", seed=1, with_x=False)
    plan = Plan.from_layer(layer)
    try:
        assert plan.info()["split_rows"] == 0
    finally:
        plan.close()
