"""GPU parity of the fused depthwise 3x3 -> sparse 1x1 plans (runs on an MI355X).

Each case calls through the C ABI (spconv_plan_create_fused, spconv_run) and
compares every output with the oracle's depthwise stage followed by its
sparse 1x1 (fp64), to |y_gpu - y_ref| <= 1e-5 * S + 1e-6 with
S = sum |W * D| + |W| * SD (SD the depthwise stage's sum of absolute terms).
"""

import zlib

import numpy as np
import pytest

from synth import make_layer, make_depthwise
from gpu_util import gpu_run, gpu_run_fused, assert_fused_parity, note

pytestmark = pytest.mark.gpu

# (cin, cout, h, w, n, sparsity, k, act, dw_act, stride): the MobileNet v1
# block shapes (stride 1 and 2), ragged tails, odd and tiny images, every
# block height, the widest strip, tiles that span several images.
CASES = [
    (32, 64, 56, 56, 1, 0.9, 1, "relu", "relu6", 1),
    (32, 64, 56, 56, 1, 0.9, 1, "relu", "relu6", 2),
    (24, 40, 7, 7, 3, 0.8, 1, "relu6", "relu", 2),
    (24, 40, 9, 11, 3, 0.8, 4, "none", "none", 1),
    (64, 36, 5, 5, 2, 0.5, 2, "none", "relu6", 2),
    (40, 48, 15, 9, 2, 0.7, 2, "relu6", "relu6", 2),
    (40, 48, 7, 9, 2, 0.7, 1, "relu6", "none", 1),
    (3, 4, 1, 1, 1, 0.5, 4, "none", "none", 1),
    (3, 4, 1, 1, 1, 0.5, 4, "none", "none", 2),
    (16, 8, 13, 1, 1, 0.0, 1, "relu", "none", 2),
    (16, 8, 1, 13, 1, 0.0, 1, "relu", "relu", 1),
    (128, 256, 56, 56, 2, 0.9, 1, "relu6", "relu6", 2),
    (256, 512, 28, 28, 2, 0.9, 1, "relu6", "relu6", 2),
    (512, 512, 14, 14, 3, 0.9, 1, "relu6", "relu6", 1),
    (512, 512, 14, 14, 3, 0.9, 4, "relu", "relu6", 1),
    (512, 1024, 14, 14, 2, 0.9, 2, "relu6", "relu6", 2),
    (600, 96, 7, 7, 2, 0.9, 1, "relu6", "relu6", 1),
    # input windows too wide for the LDS staging area: some tiles (row 1 of a
    # 3 x 2500 image), then every tile (2 rows of 4096), take the direct loads
    (512, 64, 3, 2500, 1, 0.9, 1, "relu", "relu6", 1),
    (512, 64, 3, 4096, 1, 0.9, 1, "relu", "none", 2),
]


def _case(spec):
    cin, cout, h, w, n, s, k, act, dw_act, stride = spec
    seed = zlib.crc32(repr(spec).encode()) % 1000
    layer = make_layer(cin, cout, h, w, n, s, block_rows=k, act=act, seed=seed)
    kw, kb = make_depthwise(cin, seed + 1)
    return layer, kw, kb, dw_act, stride


@pytest.mark.parametrize("spec", CASES, ids=lambda s: "%d-%d-%dx%d-n%d-s%g-k%d-%s-dw%s-s%d" % s)
def test_fused_small(spec):
    layer, kw, kb, dw_act, stride = _case(spec)
    note("fused %s" % (spec,))
    assert_fused_parity(layer, kw, kb, dw_act, stride, gpu_run_fused(layer, kw, kb, dw_act, stride), what=str(spec))


@pytest.mark.parametrize("stride", [1, 2])
def test_fused_headline_shape_full_batch(stride):
    """The 512 -> 512 layer at 14x14 output, batch 256, 90% sparse, every output."""
    h = 14 * stride
    layer = make_layer(512, 512, h, h, 256, 0.9, act="relu", seed=2020 + stride)
    kw, kb = make_depthwise(512, 77 + stride)
    note("fused 512x512 14x14 b256 stride %d" % stride)
    assert_fused_parity(layer, kw, kb, "relu6", stride, gpu_run_fused(layer, kw, kb, "relu6", stride),
                        what="fused headline s%d" % stride)


@pytest.mark.parametrize("k", [1, 2, 4])
def test_identity_depthwise_is_bitwise_the_plain_plan(k):
    """Center tap 1, bias 0, no activation, stride 1: the depthwise stage is
    exact, so the fused plan's output equals the plain 1x1 plan's bit for bit
    (each row sums in ascending channel order in every kernel)."""
    layer = make_layer(96, 128, 14, 14, 3, 0.8, block_rows=k, act="relu6", seed=31 + k)
    kw = np.zeros((96, 3, 3), np.float32)
    kw[:, 1, 1] = 1.0
    note("identity depthwise k%d" % k)
    y_f = gpu_run_fused(layer, kw, None, "none", 1)
    y_p = gpu_run(layer)
    assert np.array_equal(y_f.view(np.uint32), y_p.view(np.uint32))


@pytest.mark.parametrize("spec", [(32, 64, 56, 56, 2, 1), (64, 128, 28, 28, 2, 2), (512, 512, 14, 14, 3, 1),
                                  (512, 1024, 14, 14, 2, 2), (40, 48, 15, 9, 2, 2)],
                         ids=lambda s: "%d-%d-%dx%d-n%d-s%d" % s)
def test_fused_equals_standalone_depthwise_then_plain_plan(spec):
    """The fused plan against its two-launch form (spconv_depthwise3x3 into a
    buffer, then the plain plan with its automatic kernel choice): equal bit
    for bit, so a network may take either form."""
    import torch
    from paper_1911_09723_amd import Plan, spconv_depthwise3x3
    from gpu_util import to_gpu
    cin, cout, h, w, n, stride = spec
    layer = make_layer(cin, cout, h, w, n, 0.9, act="relu6", seed=cin + h)
    kw, kb = make_depthwise(cin, cin + 3)
    note("fused vs two launches %s" % (spec,))
    y_f = gpu_run_fused(layer, kw, kb, "relu6", stride)
    ho, wo = (h - 1) // stride + 1, (w - 1) // stride + 1
    mid = torch.empty((n, cin, ho, wo), device="cuda:0")
    spconv_depthwise3x3(to_gpu(layer.x), to_gpu(kw), to_gpu(kb), "relu6", stride, mid, n, cin, h, w)
    plan = Plan(cout, cin, layer.block_rows, layer.row_ptr, layer.col_idx, layer.values, layer.bias, "relu6")
    try:
        y_s = plan.run(mid)
        torch.cuda.synchronize()
        y_s = y_s.cpu().numpy()
    finally:
        plan.close()
    assert np.array_equal(y_f.view(np.uint32), y_s.view(np.uint32))


@pytest.mark.parametrize("n", [1, 3, 85])
def test_fused_shared_tail_tiles(n):
    """Batches whose last tiles are shared by several workgroups (each part
    computes the whole depthwise strip for its own rows)."""
    layer = make_layer(256, 256, 14, 14, n, 0.9, act="relu", seed=50 + n)
    kw, kb = make_depthwise(256, 60 + n)
    note("fused shared tail n=%d" % n)
    assert_fused_parity(layer, kw, kb, "relu", 1, gpu_run_fused(layer, kw, kb, "relu", 1), what="tail n%d" % n)


@pytest.mark.parametrize("opts", [dict(group_lanes=8), dict(group_lanes=16), dict(waves=5), dict(reorder=0),
                                  dict(kernel=1)], ids=lambda o: ",".join("%s=%s" % kv for kv in o.items()))
def test_fused_planning_does_not_change_bits(opts):
    layer = make_layer(128, 96, 14, 14, 4, 0.85, act="relu6", seed=71)
    kw, kb = make_depthwise(128, 72)
    note("fused options %s" % opts)
    y0 = gpu_run_fused(layer, kw, kb, "relu6", 2)
    y1 = gpu_run_fused(layer, kw, kb, "relu6", 2, **opts)
    assert np.array_equal(y0.view(np.uint32), y1.view(np.uint32))


def test_fused_unaligned_pointers_and_odd_output():
    """Output plane 5 x 4 = 20 columns (a multiple of 4) but a y offset by one
    element: the scalar store path; also an x offset by one element."""
    import torch
    from paper_1911_09723_amd import Plan
    from gpu_util import to_gpu
    layer = make_layer(40, 24, 9, 7, 3, 0.7, act="relu", seed=81)
    kw, kb = make_depthwise(40, 82)
    plan = Plan.fused(layer.cout, layer.cin, 1, layer.row_ptr, layer.col_idx, layer.values, layer.bias, "relu",
                      kw, kb, "relu", 2)
    try:
        note("fused unaligned")
        xb = to_gpu(np.concatenate([np.zeros(1, np.float32), layer.x.ravel()]))
        yb = torch.full((1 + 3 * 24 * 5 * 4,), float("nan"), device=xb.device)
        xv = xb[1:].view(3, 40, 9, 7)
        yv = yb[1:].view(3, 24, 5, 4)
        plan.run(xv, yv)
        torch.cuda.synchronize()
        y = yv.cpu().numpy()
    finally:
        plan.close()
    assert_fused_parity(layer, kw, kb, "relu", 2, y, what="unaligned")
