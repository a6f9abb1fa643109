"""GPU parity of channel-range passes (kernel option 5: inputs wider than
one LDS strip, run as several LDS-strip launches over ranges of at most 512
input channels, each adding to the partial sums the earlier ones left in Y).

Every case is compared with the oracle at the stated fp32 tolerance and bit
for bit with the direct-load kernel (kernel option 2): both sum each output
over all channels in ascending order from zero."""

import numpy as np
import pytest

from synth import make_layer
from gpu_util import gpu_run, assert_parity, note, to_gpu

pytestmark = pytest.mark.gpu

# (cin, cout, h, w, n, act): two and three passes, MobileNet's 1024-channel
# layer at batch 64, the 960-channel layer of the heavy-tailed workload,
# planes that are not a multiple of the vector width (element path), a
# single image, no activation
CASES = [
    (1024, 1024, 7, 7, 64, "relu6"),
    (960, 160, 7, 7, 16, "relu6"),
    (1280, 320, 7, 7, 3, "relu"),
    (600, 64, 5, 5, 3, "none"),
    (1030, 48, 3, 3, 5, "relu"),
    (1024, 96, 8, 8, 1, "relu6"),
]


@pytest.mark.parametrize("spec", CASES, ids=lambda s: "%d-%d-%dx%d-n%d-%s" % s)
def test_channel_range_passes_match_oracle_and_direct_kernel(spec):
    cin, cout, h, w, n, act = spec
    layer = make_layer(cin, cout, h, w, n, 0.9, act=act, seed=cin + cout + n)
    note("passes %s" % (spec,))
    y5 = gpu_run(layer, kernel=5)
    assert_parity(layer, y5, what="passes %s" % (spec,))
    y2 = gpu_run(layer, kernel=2)
    assert np.array_equal(y5.view(np.uint32), y2.view(np.uint32))


def test_channel_range_passes_unaligned_pointers():
    """x and y one element off a 16-byte boundary: the element-wise paths."""
    import torch
    from paper_1911_09723_amd import Plan
    layer = make_layer(1024, 64, 7, 7, 4, 0.9, act="relu", seed=5)
    plan = Plan.from_layer(layer, kernel=5)
    try:
        note("passes unaligned")
        xb = to_gpu(np.concatenate([np.zeros(1, np.float32), layer.x.ravel()]))
        yb = torch.full((4 * 64 * 49 + 1,), float("nan"), device="cuda:0")
        from paper_1911_09723_amd import spconv_run
        spconv_run(plan.handle, xb[1:], yb[1:], 4, 7, 7)
        torch.cuda.synchronize()
        assert plan.check() == 0
        y = yb[1:].cpu().numpy().reshape(4, 64, 7, 7)
    finally:
        plan.close()
    assert_parity(layer, y, what="passes unaligned")


def test_automatic_choice_runs_passes_beyond_the_lockstep_limit():
    """1300 input channels: the automatic choice plans three ranges (512, 512,
    276) and gives the direct-load kernel's bits."""
    from paper_1911_09723_amd import Plan
    layer = make_layer(1300, 40, 7, 7, 2, 0.9, act="relu6", seed=13)
    plan = Plan.from_layer(layer)
    try:
        assert plan.info()["channel_passes"] == 3
    finally:
        plan.close()
    note("passes automatic 1300")
    y0 = gpu_run(layer)
    assert_parity(layer, y0, what="passes automatic 1300")
    assert np.array_equal(y0.view(np.uint32), gpu_run(layer, kernel=2).view(np.uint32))


def test_rows_empty_in_some_ranges_or_everywhere():
    """Row r keeps nonzeros only in range r % 3 of the three 512-channel
    ranges (its partial sum passes through the other two passes untouched),
    every 7th row has none at all (bias and activation of zero)."""
    layer = make_layer(1536, 42, 5, 5, 3, 0.9, act="relu", seed=21)
    rp, ci, va = [0], [], []
    for r in range(layer.cout):
        s, e = layer.row_ptr[r], layer.row_ptr[r + 1]
        keep = [] if r % 7 == 6 else [i for i in range(s, e) if layer.col_idx[i] // 512 == r % 3]
        ci += [int(layer.col_idx[i]) for i in keep]
        va += [float(layer.values[i]) for i in keep]
        rp.append(len(ci))
    layer.row_ptr = np.array(rp, np.int32)
    layer.col_idx = np.array(ci, np.int32)
    layer.values = np.array(va, np.float32)
    note("passes empty ranges")
    y5 = gpu_run(layer, kernel=5)
    assert_parity(layer, y5, what="passes empty ranges")
    assert np.array_equal(y5.view(np.uint32), gpu_run(layer, kernel=2).view(np.uint32))
