"""GPU parity: the HIP library against the CPU oracle (runs on an MI355X).

Every case calls through the C ABI (libspconv.so via the ctypes binding) and
compares element by element with the oracle, to the tolerance
|y_gpu - y_ref| <= 1e-5 * sum|w*x| + 1e-6 (fp32) plus 2e-3 * |y_ref| (fp16).
"""

import zlib

import numpy as np
import pytest

from synth import make_layer, expand_blocks_to_csr, config_layers
from synth.configs import build
from gpu_util import gpu_run, assert_parity, note, to_gpu, device

pytestmark = pytest.mark.gpu

# (cin, cout, h, w, n, sparsity, k, storage, act): several tiles, ragged tails,
# odd spatial sizes, Cout not a multiple of a bundle, both kernels.
SMALL = [
    (32, 64, 56, 56, 1, 0.9, 1, "f32", "relu"),
    (24, 40, 7, 7, 3, 0.8, 1, "f32", "relu6"),
    (24, 40, 7, 7, 3, 0.8, 4, "f32", "none"),
    (64, 36, 5, 5, 2, 0.5, 1, "f32", "none"),
    (64, 36, 5, 5, 2, 0.5, 4, "f16", "relu6"),
    (16, 8, 13, 1, 1, 0.0, 1, "f32", "relu"),
    (16, 8, 13, 1, 1, 0.0, 4, "f16", "relu"),
    (3, 4, 1, 1, 1, 0.5, 4, "f32", "none"),
    (200, 120, 9, 9, 2, 0.9, 1, "f16", "relu"),
    (200, 120, 9, 9, 2, 0.9, 4, "f16", "none"),
    (512, 64, 14, 14, 3, 0.9, 1, "f32", "relu"),
    (600, 96, 7, 7, 2, 0.9, 1, "f32", "relu6"),     # largest strip
    (601, 96, 7, 7, 2, 0.9, 4, "f32", "relu6"),     # direct-load kernel from here on
    (700, 64, 7, 7, 2, 0.9, 1, "f32", "relu6"),
    (1280, 32, 7, 7, 2, 0.9, 4, "f32", "relu6"),
    (1500, 48, 6, 6, 2, 0.9, 1, "f32", "relu"),
    (1500, 48, 6, 6, 2, 0.9, 4, "f16", "relu"),
    (1300, 48, 8, 8, 2, 0.9, 1, "f16", "none"),
    (640, 32, 1, 3, 5, 0.9, 1, "f32", "relu"),      # direct, H*W < 4: element loads
    (640, 32, 3, 3, 7, 0.9, 2, "f32", "relu6"),     # direct, H*W = 9: paired loads, many straddles
    (640, 40, 5, 5, 9, 0.9, 4, "f32", "none"),
    # 1x2 output-channel blocks (the paper's 16x2 kernels)
    (24, 40, 7, 7, 3, 0.8, 2, "f32", "relu6"),
    (64, 36, 5, 5, 2, 0.5, 2, "f16", "none"),
    (200, 120, 9, 9, 2, 0.9, 2, "f16", "relu"),
    (512, 64, 14, 14, 3, 0.9, 2, "f32", "relu"),
    (601, 96, 7, 7, 2, 0.9, 2, "f32", "relu6"),
    (1500, 48, 6, 6, 2, 0.9, 2, "f16", "relu"),
    # LDS strip, fp32, H*W not a multiple of 4 (16-byte strip reads with a
    # second read where a vector straddles two images, element stores): every
    # residue of H*W mod 4, several images per tile, a ragged last tile
    (48, 40, 2, 3, 37, 0.7, 1, "f32", "relu"),
    (48, 40, 1, 5, 29, 0.8, 4, "f32", "relu6"),
    (96, 24, 3, 5, 11, 0.85, 2, "f32", "none"),
    (72, 33, 7, 7, 5, 0.9, 1, "f32", "relu6"),
]


@pytest.mark.parametrize("spec", SMALL, ids=lambda s: "%d-%d-%dx%d-n%d-s%g-k%d-%s-%s" % s)
def test_small_shapes(spec):
    cin, cout, h, w, n, s, k, storage, act = spec
    layer = make_layer(cin, cout, h, w, n, s, block_rows=k, storage=storage, act=act, seed=zlib.crc32(repr(spec).encode()) % 1000)
    note("small %s" % (spec,))
    assert_parity(layer, gpu_run(layer), what=str(spec))


def _workload_cases():
    cases = []
    for c in range(5):
        for spec in config_layers(c):
            cases.append(pytest.param(c, spec, id="c%d-%s" % (c, spec["name"].replace(" ", "_"))))
    return cases


@pytest.mark.parametrize("config,spec", _workload_cases())
def test_workload_full_size(config, spec):
    """Every layer of every workload at its full batch size, all outputs."""
    layer = build(config, spec)
    note("workload c%d %s" % (config, spec["name"]))
    assert_parity(layer, gpu_run(layer), what=spec["name"])


@pytest.mark.parametrize("storage", ["f32", "f16"])
def test_identity_weight_is_bitwise_x(storage):
    c = 96
    layer = make_layer(c, c, 14, 14, 2, 0.5, storage=storage, act="none", seed=5)
    layer.row_ptr = np.arange(c + 1, dtype=np.int32)
    layer.col_idx = np.arange(c, dtype=np.int32)
    layer.values = np.ones(c, dtype=np.float32)
    layer.bias = np.zeros(c, dtype=np.float32)
    note("identity %s" % storage)
    y = gpu_run(layer)
    assert np.array_equal(y.view(np.uint8), layer.x.view(np.uint8))


@pytest.mark.parametrize("k", [1, 2, 4])
@pytest.mark.parametrize("act", ["none", "relu", "relu6"])
def test_all_zero_weight_gives_act_bias(k, act):
    layer = make_layer(64, 128, 7, 7, 2, 1.0, block_rows=k, act=act, seed=6)
    layer.bias[:3] = np.float32([7.5, -2.0, 3.25])
    note("all-zero k%d %s" % (k, act))
    y = gpu_run(layer)
    b = layer.bias.astype(np.float64)
    if act == "relu":
        b = np.maximum(b, 0)
    elif act == "relu6":
        b = np.minimum(np.maximum(b, 0), 6)
    assert np.array_equal(y, np.broadcast_to(b.astype(np.float32)[None, :, None, None], y.shape))


def test_one_row_holds_all_nonzeros():
    cin, cout = 256, 64
    layer = make_layer(cin, cout, 14, 14, 2, 1.0, act="relu", seed=7)
    rp = np.zeros(cout + 1, np.int32)
    rp[6:] = cin                      # row 5 is dense, all others empty
    layer.row_ptr = rp
    layer.col_idx = np.arange(cin, dtype=np.int32)
    layer.values = (np.random.default_rng(0).standard_normal(cin) * 0.1).astype(np.float32)
    note("one dense row")
    assert_parity(layer, gpu_run(layer), what="one dense row")


def test_single_nonzero_per_row_is_exact_fma():
    cin, cout = 64, 128
    rng = np.random.default_rng(8)
    layer = make_layer(cin, cout, 7, 7, 2, 1.0, act="none", seed=8)
    layer.row_ptr = np.arange(cout + 1, dtype=np.int32)
    layer.col_idx = rng.integers(0, cin, cout).astype(np.int32)
    layer.values = rng.standard_normal(cout).astype(np.float32)
    note("single nonzero")
    y = gpu_run(layer)
    # fp32: w * x is rounded once (FMA into an exact zero), then + b is rounded once
    xs = layer.x[:, layer.col_idx]
    prod = (layer.values[None, :, None, None].astype(np.float64) * xs).astype(np.float32)
    expect = (prod + layer.bias[None, :, None, None]).astype(np.float32)
    assert np.array_equal(y, expect)


def test_run_is_deterministic_and_independent_of_planning():
    layer = make_layer(256, 256, 14, 14, 4, 0.85, act="relu", seed=9)
    note("determinism")
    base = gpu_run(layer)
    assert np.array_equal(base, gpu_run(layer))
    for opts in (dict(reorder=0), dict(group_lanes=8), dict(group_lanes=16), dict(kernel=2),
                 dict(kernel=2, group_lanes=16), dict(waves=1), dict(waves=5), dict(waves=12, reorder=0),
                 dict(group_lanes=8, waves=16), dict(pipe_sets=1), dict(regions=1), dict(regions=3),
                 dict(pipe_sets=1, regions=2), dict(pipe_sets=2, waves=7)):
        note("determinism %s" % opts)
        assert np.array_equal(base, gpu_run(layer, **opts)), opts


@pytest.mark.parametrize("n", [1, 3, 83, 84, 85, 128])
@pytest.mark.parametrize("k", [1, 2, 4])
def test_shared_tail_tiles(n, k):
    """Batch sizes around one round of tiles: the tiles left after the whole
    rounds are split by bundles over several workgroups."""
    layer = make_layer(512, 512, 14, 14, n, 0.9, block_rows=k, act="relu", seed=11 + n)
    note("tail split n=%d k=%d" % (n, k))
    assert_parity(layer, gpu_run(layer), what="tail n=%d k=%d" % (n, k))


@pytest.mark.parametrize("opts", [dict(), dict(pipe_sets=1), dict(regions=1), dict(regions=2),
                                  dict(pipe_sets=1, regions=3), dict(waves=9), dict(group_lanes=8)],
                         ids=lambda o: "-".join("%s%d" % kv for kv in o.items()) or "auto")
def test_pipelined_rounds_bitwise_equal_simple_path(opts):
    """Batch 256 of the 512 -> 512 layer: three whole rounds of tiles through
    the pipelined kernel plus a shared tail; every planner choice gives the
    same bits, and they match the oracle."""
    layer = make_layer(512, 512, 14, 14, 256, 0.9, act="relu", seed=21)
    note("pipelined rounds %s" % opts)
    y = gpu_run(layer, **opts)
    ref = gpu_run(layer, kernel=2)  # direct-load kernel: no strip, no pipeline
    assert np.array_equal(y, ref), opts
    assert_parity(layer, y, what="pipelined %s" % opts)


def test_split_does_not_change_bits():
    """The per-row summation order is fixed, so how tiles are shared between
    workgroups does not change a single bit: image i of a batch of 85 equals
    image i of a batch of 84 (different tail splits)."""
    big = make_layer(512, 512, 14, 14, 85, 0.9, act="none", seed=12)
    small = make_layer(512, 512, 14, 14, 84, 0.9, act="none", seed=12)
    small.x = np.ascontiguousarray(big.x[:84])
    note("split bits")
    assert np.array_equal(gpu_run(big)[:84], gpu_run(small))


@pytest.mark.parametrize("k", [2, 4])
def test_blocked_equals_expanded_csr_bitwise(k):
    layer = make_layer(128, 96, 14, 14, 2, 0.8, block_rows=k, act="relu6", seed=10)
    rp, ci, va = expand_blocks_to_csr(96, k, layer.row_ptr, layer.col_idx, layer.values)
    csr = make_layer(128, 96, 14, 14, 2, 0.8, act="relu6", seed=10)
    csr.row_ptr, csr.col_idx, csr.values, csr.bias, csr.x = rp, ci, va, layer.bias, layer.x
    note("blocked vs expanded k=%d" % k)
    assert np.array_equal(gpu_run(layer), gpu_run(csr))


def test_batch_split_bitwise():
    layer = make_layer(96, 160, 7, 7, 3, 0.9, act="relu6", seed=11)
    note("batch split")
    whole = gpu_run(layer)
    parts = [gpu_run(layer, x=layer.x[i:i + 1]) for i in range(3)]
    assert np.array_equal(whole, np.concatenate(parts))


@pytest.mark.parametrize("storage", ["f32", "f16"])
def test_unaligned_pointers_take_scalar_path(storage):
    """x and y offset by one element from 16-byte alignment give the same bits."""
    import torch
    from paper_1911_09723_amd import Plan
    layer = make_layer(64, 64, 8, 8, 2, 0.7, storage=storage, act="relu", seed=12)
    note("unaligned %s" % storage)
    ref = gpu_run(layer)
    plan = Plan.from_layer(layer)
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


def test_runs_on_caller_stream_and_empty_batch_is_noop():
    import torch
    from paper_1911_09723_amd import Plan, spconv_run
    layer = make_layer(48, 80, 10, 10, 2, 0.9, act="relu", seed=13)
    note("stream / empty")
    ref = gpu_run(layer)
    plan = Plan.from_layer(layer)
    try:
        s = torch.cuda.Stream()
        x = to_gpu(layer.x)
        torch.cuda.synchronize()
        with torch.cuda.stream(s):
            y = plan.run(x)
        s.synchronize()
        assert np.array_equal(y.cpu().numpy(), ref)
        sentinel = torch.full((4,), 7.0, device=device())
        spconv_run(plan.handle, x, sentinel, 0, 10, 10)
        spconv_run(plan.handle, x, sentinel, 2, 0, 10)
        torch.cuda.synchronize()
        assert torch.all(sentinel == 7.0)
    finally:
        plan.close()


def test_overlapping_x_y_rejected():
    import torch
    from paper_1911_09723_amd import Plan, SpconvError, spconv_run
    layer = make_layer(16, 16, 4, 4, 1, 0.5, seed=14, with_x=False)
    plan = Plan.from_layer(layer)
    try:
        buf = torch.zeros(16 * 16 + 8, device=device())
        with pytest.raises(SpconvError) as ei:
            spconv_run(plan.handle, buf, buf[8:], 1, 4, 4)
        assert ei.value.status == 1
    finally:
        plan.close()


@pytest.mark.parametrize("k", [1, 2, 4])
@pytest.mark.parametrize("storage", ["f32", "f16"])
def test_dense_weight_plan_matches_block_csr_plan(k, storage):
    """A plan built from the dense masked weight (block height detected, then
    converted) computes the same bits as the plan from the block-CSR arrays."""
    from paper_1911_09723_amd import Plan
    from synth import densify
    import torch
    layer = make_layer(160, 96, 7, 7, 3, 0.85, block_rows=k, storage=storage, act="relu6", seed=30 + k)
    dense = densify(96, 160, k, layer.row_ptr, layer.col_idx, layer.values).astype(np.float32)
    note("dense plan k=%d %s" % (k, storage))
    plan = Plan.from_dense(dense, 0, layer.bias, "relu6", storage)
    try:
        assert plan.info()["block_rows"] == k
        y = plan.run(to_gpu(layer.x))
        torch.cuda.synchronize()
        y = y.cpu().numpy()
    finally:
        plan.close()
    assert np.array_equal(y.view(np.uint8), gpu_run(layer).view(np.uint8))
    assert_parity(layer, y, what="dense k=%d" % k)


@pytest.mark.parametrize("kr,kc,storage", [(1, 4, "f32"), (2, 2, "f32"), (1, 2, "f16"), (4, 4, "f32"),
                                          (2, 4, "f16"), (1, 4, "f16")])
@pytest.mark.parametrize("cin,h,w", [(64, 14, 14), (1024, 7, 7), (96, 5, 3)])
def test_input_channel_blocks_match_oracle(kr, kc, storage, cin, h, w):
    """Blocks of kr output x kc input channels (4x1, 2x2, ...) against the
    block oracle, on the strip kernel, the direct-load kernel (cin = 1024) and
    a ragged H*W."""
    from paper_1911_09723_amd import Plan
    from blocks_util import random_blocks
    import oracle
    rng = np.random.default_rng(kr * 100 + kc * 10 + cin)
    cout = 128
    rp, ci, va = random_blocks(cout, cin, kr, kc, 0.1, rng)
    va = (va * np.sqrt(2.0 / (0.1 * cin))).astype(np.float32)
    if storage == "f16":
        va = va.astype(np.float16).astype(np.float32)
    b = (rng.standard_normal(cout) * 0.1).astype(np.float32)
    n = 3
    x = np.maximum(rng.standard_normal((n, cin, h, w)), 0).astype(np.float16 if storage == "f16" else np.float32)
    plan = Plan.blocked(cout, cin, kr, kc, rp, ci, va, b, "relu6", storage)
    try:
        note("blocks %dx%d %s cin %d %dx%d" % (kr, kc, storage, cin, h, w))
        yt = plan.run(to_gpu(x))
        import torch
        torch.cuda.synchronize()
        y = yt.cpu().numpy()
    finally:
        plan.close()
    y_ref, _, s = oracle.spconv_ref(cout, cin, kr, rp, ci, va, b, "relu6", x, storage=storage, block_cols=kc)
    tol = oracle.tolerance(y_ref, s, storage)
    assert y.shape == y_ref.shape
    assert np.all(np.abs(y.astype(np.float64) - y_ref.astype(np.float64)) <= tol)


def test_dense_weight_with_2x2_blocks_plans_like_the_blocked_arrays():
    """spconv_plan_create_dense_blocked (detecting 2 x 2) gives the same bits
    as spconv_plan_create_blocked on the same blocks."""
    from paper_1911_09723_amd import Plan, spconv
    from blocks_util import dense_from_blocks, random_blocks
    import torch
    rng = np.random.default_rng(5)
    cin, cout = 128, 96
    rp, ci, va = random_blocks(cout, cin, 2, 2, 0.1, rng)
    va[va == 0] = 0.25
    dense = dense_from_blocks(cout, cin, 2, 2, rp, ci, va).astype(np.float32)
    assert spconv.spconv_detect_blocks(dense) == (2, 2)
    b = rng.standard_normal(cout).astype(np.float32)
    x = np.maximum(rng.standard_normal((2, cin, 9, 9)), 0).astype(np.float32)
    p1 = Plan.blocked(cout, cin, 2, 2, rp, ci, va, b, "relu")
    p2 = Plan.__new__(Plan)
    p2.handle = spconv.spconv_plan_create_dense_blocked(dense, 0, 0, b, "relu")
    p2.cout, p2.cin, p2.storage, p2.dw_stride = cout, cin, "f32", 0
    try:
        note("dense 2x2 blocked plan")
        xt = to_gpu(x)
        y1 = p1.run(xt)
        y2 = p2.run(xt)
        torch.cuda.synchronize()
        assert p2.info()["block_cols"] == 2 and p2.info()["block_rows"] == 2
        assert torch.equal(y1, y2)
    finally:
        p1.close()
        p2.close()
