"""GPU parity of the register-indexed kernel (kernel=3) against the CPU oracle.

Every case calls through the C ABI and compares element by element with the
oracle to |y_gpu - y_ref| <= 1e-5 * sum|w*x| + 1e-6.  Beyond that, the
kernel sums each row in ascending input channel from zero like the
direct-load kernel, so the two give the same bits on finite inputs.

Cases cover every column count per lane (lane_cols 1 .. 6) with each block
height, both ring-copy paths (16-byte copies when every image's column count
is a multiple of 4, one dword per lane otherwise), channel counts that wrap
the 96-row ring many times or end in a ragged chunk, tiles that end inside an
image, the row-pair phase for columns left over after the whole tiles, and
every fp32 layer of the workloads at full size.
"""

import zlib

import numpy as np
import pytest

from synth import make_layer, config_layers
from synth.configs import build
from gpu_util import gpu_run, assert_parity, note, to_gpu, device

pytestmark = pytest.mark.gpu

# (cin, cout, h, w, n, sparsity, k, act)
SHAPES = [
    (64, 48, 14, 14, 3, 0.9, 1, "relu"),      # 16-byte copies
    (40, 40, 7, 7, 5, 0.8, 1, "relu6"),       # dword copies (49 columns per image)
    (200, 96, 6, 10, 4, 0.9, 1, "none"),      # ragged last chunk, ring wraps
    (1000, 64, 4, 4, 9, 0.95, 1, "relu"),     # 63 chunks; tiles span many images
    (96, 160, 5, 5, 7, 0.7, 2, "relu"),       # dword copies, 1x2 blocks
    (128, 64, 8, 8, 5, 0.9, 2, "none"),       # 16-byte copies, 1x2 blocks
    (72, 96, 14, 14, 2, 0.85, 4, "relu6"),    # 16-byte copies, 1x4 blocks
    (130, 52, 3, 3, 11, 0.9, 4, "none"),      # dword copies, 1x4 blocks, cout not a multiple of 16
    (17, 20, 2, 2, 3, 0.5, 1, "relu"),        # one chunk, two slots, tiny images
]


@pytest.mark.parametrize("lane_cols", [1, 2, 3, 4, 5, 6])
@pytest.mark.parametrize("spec", SHAPES, ids=lambda s: "%d-%d-%dx%d-n%d-s%g-k%d-%s" % s)
def test_lane_cols(spec, lane_cols):
    cin, cout, h, w, n, s, k, act = spec
    layer = make_layer(cin, cout, h, w, n, s, block_rows=k, act=act,
                       seed=zlib.crc32(repr(spec).encode()) % 1000)
    note("indexed %s lane_cols=%d" % (spec, lane_cols))
    y = gpu_run(layer, kernel=3, lane_cols=lane_cols)
    assert_parity(layer, y, what="%s C=%d" % (spec, lane_cols))
    assert np.array_equal(y, gpu_run(layer, kernel=2)), "not bitwise equal to the direct-load kernel"


def _fp32_workload_cases():
    cases = []
    for c in range(5):
        for spec in config_layers(c):
            if spec.get("storage", "f32") != "f32":
                continue
            cases.append(pytest.param(c, spec, id="c%d-%s" % (c, spec["name"].replace(" ", "_"))))
    return cases


@pytest.mark.parametrize("config,spec", _fp32_workload_cases())
def test_workload_full_size(config, spec):
    """Every fp32 layer of the workloads at its full batch, all outputs; the
    512 -> 512 layer at batch 256 runs one round of whole tiles plus the
    row-pair phase."""
    layer = build(config, spec)
    note("indexed workload c%d %s" % (config, spec["name"]))
    y = gpu_run(layer, kernel=3)
    assert_parity(layer, y, what=spec["name"])


@pytest.mark.parametrize("n", [1, 85, 128, 130, 256])
@pytest.mark.parametrize("k", [1, 4])
def test_row_pairs_and_rounds(n, k):
    """Batches around one round of whole tiles (128 tiles of 384 columns at
    512 output channels): uniform tiles, or one round plus row pairs."""
    layer = make_layer(512, 512, 14, 14, n, 0.9, block_rows=k, act="relu", seed=31 + n)
    note("indexed rounds n=%d k=%d" % (n, k))
    y = gpu_run(layer, kernel=3)
    assert_parity(layer, y, what="n=%d k=%d" % (n, k))
    assert np.array_equal(y, gpu_run(layer, kernel=2))


def test_row_pairs_dword_path():
    """Row pairs when the image's column count is not a multiple of 4."""
    layer = make_layer(256, 256, 7, 7, 1100, 0.9, act="relu6", seed=41)
    note("indexed row pairs 7x7 n=1100")
    y = gpu_run(layer, kernel=3)
    assert_parity(layer, y, what="pairs 7x7")


def test_unaligned_input_takes_dword_copies():
    import torch
    from paper_1911_09723_amd import Plan
    layer = make_layer(64, 64, 8, 8, 3, 0.8, act="relu", seed=42)
    note("indexed unaligned")
    ref = gpu_run(layer, kernel=3)
    plan = Plan.from_layer(layer, kernel=3)
    try:
        flat = to_gpu(np.concatenate([np.zeros(1, layer.x.dtype), layer.x.ravel()]))
        x = flat[1:].view(layer.x.shape)
        ybuf = torch.empty(1 + ref.size, dtype=flat.dtype, device=device())
        y = ybuf[1:].view(ref.shape)
        plan.run(x, y)
        torch.cuda.synchronize()
        assert np.array_equal(y.cpu().numpy(), ref)
    finally:
        plan.close()


def test_empty_rows_slots_and_chunks():
    """Rows without nonzeros, a slot whose rows are all empty, and input
    channel chunks no row of a slot touches."""
    cin, cout = 160, 64
    layer = make_layer(cin, cout, 6, 6, 3, 1.0, act="none", seed=43)
    rng = np.random.default_rng(43)
    rp = [0]
    ci = []
    for r in range(cout):
        if r >= 48 or r % 5 == 0:
            cols = []                               # rows 48.. (a whole slot) and every fifth row empty
        else:
            cols = sorted(rng.choice(np.arange(32, 64), size=3, replace=False).tolist())  # chunks 2, 3 only
        ci += cols
        rp.append(len(ci))
    layer.row_ptr = np.asarray(rp, np.int32)
    layer.col_idx = np.asarray(ci, np.int32)
    layer.values = rng.standard_normal(len(ci)).astype(np.float32)
    note("indexed empty rows/slots/chunks")
    y = gpu_run(layer, kernel=3)
    assert_parity(layer, y, what="empty parts")
    assert np.array_equal(y, gpu_run(layer, kernel=2))


@pytest.mark.parametrize("kernel", [0, 3], ids=["strip-pipeline", "indexed"])
def test_a_wait_that_gives_up_is_reported(kernel):
    """With the plan's wait bound at 0 every bounded wait that finds its data
    missing gives up at once (the kernels still finish); the plan's error word
    reports it.  Cleared and run with the default bound, the word stays 0 and
    the output matches the oracle."""
    import torch
    from paper_1911_09723_amd import Plan, spconv_plan_set_wait_limit, SPCONV_FLAG_WAIT_GAVE_UP
    layer = make_layer(512, 512, 14, 14, 256, 0.9, act="relu", seed=51)
    note("indexed forced give-up kernel=%d" % kernel)
    plan = Plan.from_layer(layer, kernel=kernel)
    try:
        x = to_gpu(layer.x)
        spconv_plan_set_wait_limit(plan.handle, 0)
        plan.run(x)
        torch.cuda.synchronize()
        assert plan.check(clear=True) & SPCONV_FLAG_WAIT_GAVE_UP
        spconv_plan_set_wait_limit(plan.handle, 1 << 22)
        y = plan.run(x)
        torch.cuda.synchronize()
        assert plan.check() == 0
        assert_parity(layer, y.cpu().numpy(), what="after a forced give-up")
    finally:
        plan.close()
