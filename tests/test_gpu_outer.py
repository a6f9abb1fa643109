"""GPU parity of the outer-product kernel (kernel=4, 1 x 4 blocks) against the oracle.

Every case calls through the C ABI and compares element by element with the
oracle to its tolerance (fp32: |y_gpu - y_ref| <= 1e-5 * sum|w*x| + 1e-6;
fp16 storage: the fp16 bound).  The matrix instruction
rounds each product-and-add once, like a fused multiply-add, and every row
still sums in ascending input channel from zero, so the results also equal
the direct-load kernel's bit for bit.

Cases: ragged last tiles and tiles that straddle images, octs of fewer than 8
block rows, zero and one tile per workgroup (fewer tiles than compute units)
and many, several octs per wavefront, inputs whose channel count is not a
multiple of 8, rows without stored blocks, every activation, the channel
offsets read from the workgroup's LDS copy and (widest input) from global
memory, and the 1x4 headline layer at full size.
"""

import zlib

import numpy as np
import pytest

from synth import make_layer
from gpu_util import gpu_run, assert_parity, note

pytestmark = pytest.mark.gpu

# (cin, cout, h, w, n, sparsity, act)
SHAPES = [
    (64, 64, 4, 4, 3, 0.8, "relu"),          # 48 columns: one whole and one ragged tile
    (72, 96, 14, 14, 2, 0.85, "relu6"),      # tiles straddle images; 3 octs
    (17, 20, 2, 2, 9, 0.5, "none"),          # cin not a multiple of 8; one partial oct of 5 rows
    (200, 1024, 2, 2, 16, 0.95, "relu"),     # 32 octs: two per wavefront and tile parity
    (632, 64, 4, 8, 5, 0.9, "none"),         # widest input: the offset table stays in global memory
    (512, 128, 28, 28, 2, 0.9, "relu"),      # 49 tiles over the compute units
    (128, 256, 8, 8, 300, 0.9, "relu"),      # 600 tiles: several per workgroup, both buffers refilled
]


@pytest.mark.parametrize("spec", SHAPES, ids=lambda s: "%d-%d-%dx%d-n%d-s%g-%s" % s)
def test_outer_matches_oracle_and_direct_kernel(spec):
    cin, cout, h, w, n, s, act = spec
    layer = make_layer(cin, cout, h, w, n, s, block_rows=4, act=act, seed=zlib.crc32(repr(spec).encode()) % 1000)
    note("outer %s" % (spec,))
    y = gpu_run(layer, kernel=4)
    assert_parity(layer, y, what=str(spec))
    assert np.array_equal(y, gpu_run(layer, kernel=2)), "not bitwise equal to the direct-load kernel"


def test_outer_rows_without_blocks():
    """Block rows with no stored block (their outputs are bias + activation)
    and a whole oct of them."""
    cin, cout = 96, 128
    layer = make_layer(cin, cout, 6, 6, 7, 1.0, block_rows=4, act="none", seed=43)
    rng = np.random.default_rng(43)
    rp = [0]
    ci = []
    for r in range(cout // 4):
        cols = [] if (r >= 24 or r % 3 == 0) else sorted(rng.choice(cin, size=5, replace=False).tolist())
        ci += cols
        rp.append(len(ci))
    layer.row_ptr = np.asarray(rp, np.int32)
    layer.col_idx = np.asarray(ci, np.int32)
    layer.values = rng.standard_normal(4 * len(ci)).astype(np.float32)
    note("outer empty rows")
    y = gpu_run(layer, kernel=4)
    assert_parity(layer, y, what="empty rows")
    assert np.array_equal(y, gpu_run(layer, kernel=2))


@pytest.mark.parametrize("n", [1, 64, 256])
def test_outer_headline_layer(n):
    """The 512 -> 512 layer at 14 x 14, 90% sparse 1 x 4 blocks; batch 256 is
    1568 tiles, six rounds of the grid plus 32 tiles."""
    layer = make_layer(512, 512, 14, 14, n, 0.9, block_rows=4, act="relu", seed=71 + n)
    note("outer headline n=%d" % n)
    y = gpu_run(layer, kernel=4)
    assert_parity(layer, y, what="n=%d" % n)
    assert np.array_equal(y, gpu_run(layer, kernel=2))


# (cin, cout, h, w, n, sparsity, act, storage): H*W not a multiple of 4 (4-column
# vectors straddle images, copied and stored element by element) and fp16
# storage (converted to fp32 on the way into LDS, rounded once on the way out)
STAGED = [
    (64, 64, 7, 7, 3, 0.8, "relu", "f32"),
    (130, 96, 5, 5, 17, 0.9, "none", "f32"),
    (40, 240, 28, 28, 2, 0.9, "relu6", "f16"),
    (112, 672, 14, 14, 3, 0.9, "relu6", "f16"),
    (320, 1280, 7, 7, 5, 0.9, "relu6", "f16"),
    (24, 36, 3, 3, 7, 0.7, "none", "f16"),
]


@pytest.mark.parametrize("spec", STAGED, ids=lambda s: "%d-%d-%dx%d-n%d-s%g-%s-%s" % s)
def test_outer_ragged_and_fp16(spec):
    cin, cout, h, w, n, s, act, st = spec
    layer = make_layer(cin, cout, h, w, n, s, block_rows=4, act=act, storage=st,
                       seed=zlib.crc32(repr(spec).encode()) % 1000)
    note("outer staged %s" % (spec,))
    y = gpu_run(layer, kernel=4)
    assert_parity(layer, y, what=str(spec))
    assert np.array_equal(y, gpu_run(layer, kernel=2)), "not bitwise equal to the direct-load kernel"


def test_outer_unaligned_pointers_take_the_staged_copy():
    """x and y 4 bytes off a 16-byte boundary: element copies and stores."""
    import torch
    from paper_1911_09723_amd import Plan
    from gpu_util import to_gpu, device
    layer = make_layer(64, 64, 8, 8, 3, 0.8, block_rows=4, act="relu", seed=42)
    note("outer unaligned")
    ref = gpu_run(layer, kernel=4)
    plan = Plan.from_layer(layer, kernel=4)
    try:
        flat = to_gpu(np.concatenate([np.zeros(1, layer.x.dtype), layer.x.ravel()]))
        x = flat[1:].view(layer.x.shape)
        ybuf = torch.empty(1 + ref.size, dtype=flat.dtype, device=device())
        y = ybuf[1:].view(ref.shape)
        plan.run(x, y)
        torch.cuda.synchronize()
        assert plan.check() == 0
        assert np.array_equal(y.cpu().numpy(), ref)
    finally:
        plan.close()


# (cin, cout, h, w, n, sparsity, act): unstructured layers on the vector mode
# (one fused multiply-add per lane and column per step): 32-column tiles up
# to 632 input channels, 16-column tiles above; ragged H*W; a partial set
VECTOR = [
    (64, 64, 4, 4, 3, 0.8, "relu"),
    (512, 512, 14, 14, 4, 0.9, "relu"),
    (96, 40, 7, 7, 9, 0.7, "relu6"),
    (1024, 1024, 7, 7, 8, 0.9, "relu6"),
    (960, 160, 7, 7, 6, 0.85, "none"),
    (1264, 24, 5, 5, 3, 0.9, "relu"),
    (17, 20, 2, 2, 9, 0.5, "none"),
]


@pytest.mark.parametrize("spec", VECTOR, ids=lambda s: "%d-%d-%dx%d-n%d-s%g-%s" % s)
def test_vector_mode_matches_oracle_and_direct_kernel(spec):
    cin, cout, h, w, n, s, act = spec
    layer = make_layer(cin, cout, h, w, n, s, block_rows=1, act=act, seed=zlib.crc32(repr(spec).encode()) % 1000)
    note("lockstep vector %s" % (spec,))
    y = gpu_run(layer, kernel=4)
    assert_parity(layer, y, what=str(spec))
    assert np.array_equal(y, gpu_run(layer, kernel=2)), "not bitwise equal to the direct-load kernel"


@pytest.mark.parametrize("n", [64, 256])
def test_vector_mode_headline_layer(n):
    layer = make_layer(512, 512, 14, 14, n, 0.9, block_rows=1, act="relu", seed=91 + n)
    note("lockstep vector headline n=%d" % n)
    y = gpu_run(layer, kernel=4)
    assert_parity(layer, y, what="n=%d" % n)
    assert np.array_equal(y, gpu_run(layer, kernel=2))
