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
