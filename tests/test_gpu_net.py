"""GPU parity of the network operators and of a whole MobileNet v1 forward
pass (runs on an MI355X).

Each operator is compared element by element with the oracle at
|y_gpu - y_ref| <= 1e-5 * S + 1e-6 (S the sum of absolute terms).  The whole
network is compared with the oracle's double-precision chain; its
propagated worst-case scale is astronomically loose after 27 layers, so the
chain test bounds the logits by 1e-4 * max |logit| instead: a wiring mistake
(a wrong stride, layer order or buffer) moves logits by the order of the
logits themselves, while fp32 rounding through the chain moves them by ~1e-6
relative.  Graph replays must equal eager runs bit for bit (the kernels are
deterministic).
"""

import numpy as np
import pytest

import oracle
from synth import make_mobilenet_v1, make_image, make_depthwise
from gpu_util import note, to_gpu

pytestmark = pytest.mark.gpu


def _sync_np(t):
    import torch
    torch.cuda.synchronize()
    return t.cpu().numpy()


def _check(y, y_ref, scale, what):
    tol = 1e-5 * scale + 1e-6
    err = np.abs(y.astype(np.float64) - y_ref)
    bad = int((err > tol).sum())
    assert y.shape == y_ref.shape, (y.shape, y_ref.shape)
    assert bad == 0, "%s: %d of %d outside tolerance (worst %.3g)" % (what, bad, err.size, float((err / tol).max()))


@pytest.mark.parametrize("n,h,w,cin,cout,stride,act,bias", [
    (2, 224, 224, 3, 32, 2, "relu6", True),
    (1, 17, 9, 3, 32, 2, "relu", True),
    (3, 8, 8, 1, 5, 1, "none", False),
    (1, 13, 11, 8, 24, 2, "relu6", True),
    (2, 5, 7, 4, 64, 1, "none", True),
    (1, 1, 1, 3, 7, 2, "relu", True),
    (1, 9, 30, 3, 600, 1, "relu", True),   # more weights than the old LDS copy held
])
def test_stem_conv_parity(n, h, w, cin, cout, stride, act, bias):
    import torch
    from paper_1911_09723_amd import spconv_conv3x3_hwc
    rng = np.random.default_rng(h * 31 + w + cin)
    x = rng.uniform(-1, 1, (n, h, w, cin)).astype(np.float32)
    wt = (rng.standard_normal((cout, 3, 3, cin)) * 0.3).astype(np.float32)
    b = (rng.standard_normal(cout) * 0.1).astype(np.float32) if bias else None
    ho, wo = (h - 1) // stride + 1, (w - 1) // stride + 1
    y = torch.full((n, cout, ho, wo), float("nan"), device="cuda:0")
    note("stem %s" % ((n, h, w, cin, cout, stride, act, bias),))
    spconv_conv3x3_hwc(to_gpu(x), to_gpu(wt), None if b is None else to_gpu(b), act, stride, y, n, h, w, cin, cout)
    y_ref, s = oracle.conv3x3_hwc_ref(x, wt, b, act, stride)
    _check(_sync_np(y), y_ref, s, "stem")


@pytest.mark.parametrize("n,c,h,w,stride,act", [
    (2, 1024, 7, 7, 1, "relu6"), (1, 64, 112, 112, 2, "relu"), (3, 5, 9, 4, 2, "none"), (1, 3, 1, 1, 1, "relu6"),
    # staged kernel: a 112 x 112 plane per workgroup, many 3 x 3 planes per
    # workgroup crossing image boundaries, width 1 (divisor 1), odd planes
    # with stride 2, the largest plane that fits its LDS (126 x 126), then
    # one past it (the direct kernel)
    (4, 32, 112, 112, 1, "relu6"), (3, 333, 3, 3, 1, "relu"), (2, 6, 7, 1, 1, "none"), (3, 17, 15, 13, 2, "relu6"),
    (2, 3, 126, 126, 1, "relu6"), (1, 3, 127, 127, 2, "relu"),
    # every lane width and stride: 4 and 2 columns per lane at stride 2
    # (w a multiple of 8, of 4 only), one column at stride 2 with w even,
    # the MobileNet planes 56 and 28 at stride 2; planes too wide for whole
    # planes per wavefront (one column per lane, 64-column parts), both strides
    (2, 8, 20, 200, 2, "relu6"), (2, 16, 28, 28, 2, "relu"), (3, 16, 14, 14, 2, "relu6"), (2, 16, 56, 56, 2, "none"),
    (2, 8, 30, 300, 1, "relu6"), (1, 4, 9, 301, 2, "relu"),
])
def test_standalone_depthwise_parity(n, c, h, w, stride, act):
    import torch
    from paper_1911_09723_amd import spconv_depthwise3x3
    rng = np.random.default_rng(c + h)
    x = np.maximum(rng.standard_normal((n, c, h, w)), 0).astype(np.float32)
    k, b = make_depthwise(c, c + w)
    ho, wo = (h - 1) // stride + 1, (w - 1) // stride + 1
    y = torch.full((n, c, ho, wo), float("nan"), device="cuda:0")
    note("depthwise %s" % ((n, c, h, w, stride, act),))
    spconv_depthwise3x3(to_gpu(x), to_gpu(k), to_gpu(b), act, stride, y, n, c, h, w)
    d, sd = oracle.dw3x3_ref(x, k, b, act, stride)
    _check(_sync_np(y), d, sd, "depthwise")


@pytest.mark.parametrize("stride", [1, 2])
def test_standalone_depthwise_unaligned_pointers(stride):
    """x and y one element off a 16-byte boundary: one column per lane."""
    import torch
    from paper_1911_09723_amd import spconv_depthwise3x3
    n, c, h, w = 2, 12, 28, 28
    rng = np.random.default_rng(9 + stride)
    x = rng.standard_normal((n, c, h, w)).astype(np.float32)
    k, b = make_depthwise(c, 3)
    ho, wo = (h - 1) // stride + 1, (w - 1) // stride + 1
    xb = to_gpu(np.concatenate([np.zeros(1, np.float32), x.ravel()]))[1:]
    yb = torch.full((n * c * ho * wo + 1,), float("nan"), device="cuda:0")
    note("depthwise unaligned stride %d" % stride)
    spconv_depthwise3x3(xb, to_gpu(k), to_gpu(b), "relu6", stride, yb[1:], n, c, h, w)
    d, sd = oracle.dw3x3_ref(x, k, b, "relu6", stride)
    _check(_sync_np(yb[1:]).reshape(n, c, ho, wo), d, sd, "depthwise unaligned")


@pytest.mark.parametrize("n,c,h,w", [(64, 1024, 7, 7), (3, 5, 1, 1), (2, 7, 13, 3)])
def test_global_avg_pool_parity(n, c, h, w):
    import torch
    from paper_1911_09723_amd import spconv_global_avg_pool
    rng = np.random.default_rng(n * c)
    x = rng.standard_normal((n, c, h, w)).astype(np.float32)
    y = torch.full((n, c), float("nan"), device="cuda:0")
    note("gap %s" % ((n, c, h, w),))
    spconv_global_avg_pool(to_gpu(x), y, n, c, h, w)
    g, gs = oracle.gap_ref(x)
    _check(_sync_np(y), g, gs, "gap")


@pytest.mark.parametrize("n,cin,cout,act,bias,offset", [
    (64, 1024, 1000, "none", True, 0), (3, 7, 130, "relu6", True, 0), (5, 64, 64, "relu", False, 1),
    (1, 1, 1, "none", True, 0),
    # several image and row tiles with ragged edges, channel chunks that end
    # inside a block of 8, a width that leaves most wavefronts without channels
    (70, 2052, 33, "relu", True, 0), (33, 12, 65, "none", True, 0), (2, 1030, 7, "relu6", False, 1),
])
def test_linear_parity(n, cin, cout, act, bias, offset):
    """Against the oracle's 1x1 over 1 x 1 images with the dense weight as CSR;
    offset 1 misaligns x (the element-by-element path)."""
    import torch
    from paper_1911_09723_amd import spconv_linear
    rng = np.random.default_rng(n + cin + cout)
    x = rng.standard_normal((n, cin)).astype(np.float32)
    wt = (rng.standard_normal((cout, cin)) / np.sqrt(cin)).astype(np.float32)
    b = rng.standard_normal(cout).astype(np.float32) if bias else None
    xb = to_gpu(np.concatenate([np.zeros(offset, np.float32), x.ravel()]))[offset:]
    y = torch.full((n, cout), float("nan"), device="cuda:0")
    note("linear %s" % ((n, cin, cout, act, bias, offset),))
    spconv_linear(xb, to_gpu(wt), None if b is None else to_gpu(b), act, y, n, cin, cout)
    rp = np.arange(0, cout * cin + 1, cin, dtype=np.int32)
    ci = np.tile(np.arange(cin, dtype=np.int32), cout)
    _, y64, s = oracle.spconv_ref(cout, cin, 1, rp, ci, wt.ravel(), b, act, x.reshape(n, cin, 1, 1))
    _check(_sync_np(y), y64.reshape(n, cout), s.reshape(n, cout), "linear")


def _engine_case(batch, hw, classes, seed, fuse="auto"):
    from paper_1911_09723_amd.mobilenet import MobileNetV1Engine
    net = make_mobilenet_v1(seed=seed, classes=classes)
    x = make_image(batch, hw, hw, seed=seed)
    return net, x, MobileNetV1Engine(net, batch, hw, hw, fuse=fuse)


@pytest.mark.parametrize("batch,hw,classes", [(2, 224, 1000), (3, 32, 10), (64, 224, 1000)])
def test_mobilenet_v1_forward_matches_oracle(batch, hw, classes):
    # batch 64 at 224 x 224 is the configuration bench.py times
    net, x, eng = _engine_case(batch, hw, classes, seed=batch)
    try:
        note("mobilenet v1 batch %d %dx%d (%d launches, %d fused blocks)" % (batch, hw, hw, eng.launches(),
                                                                             eng.fused_blocks))
        # every block is one launch when fused, two when not
        assert eng.launches() == 1 + 13 + (13 - eng.fused_blocks) + 2
        y = _sync_np(eng.forward(to_gpu(x)))
    finally:
        eng.close()
    y_ref, s = oracle.mobilenet_v1_ref(net, x)
    err = np.abs(y.astype(np.float64) - y_ref)
    assert np.all(err <= 1e-5 * s + 1e-6)
    bound = 1e-4 * np.abs(y_ref).max()
    print("max |logit error| %.3g, bound %.3g" % (err.max(), bound))
    assert err.max() <= bound
    assert np.array_equal(y.argmax(axis=1), y_ref.argmax(axis=1))


def test_mobilenet_v1_fusion_choice_does_not_change_bits():
    """Every block fused where possible, no block fused, and the timed
    choice: the same logits bit for bit (both forms of a block run the same
    fp32 operations in the same order)."""
    outs = {}
    for fuse in ("always", "never", "auto"):
        net, x, eng = _engine_case(4, 96, 10, seed=5, fuse=fuse)
        try:
            note("mobilenet v1 fuse=%s (%d fused blocks)" % (fuse, eng.fused_blocks))
            assert eng.fused_blocks == {"always": 12, "never": 0}.get(fuse, eng.fused_blocks)
            outs[fuse] = _sync_np(eng.forward(to_gpu(x))).copy()
        finally:
            eng.close()
    for fuse in ("never", "auto"):
        assert np.array_equal(outs[fuse].view(np.uint32), outs["always"].view(np.uint32)), fuse


def test_mobilenet_v1_graph_replays_equal_eager_runs():
    """Capture once, then alternate eager runs and replays on new inputs (with
    synchronizations between); every replay must equal the eager result."""
    import torch
    net, x, eng = _engine_case(4, 64, 16, seed=11)
    try:
        note("mobilenet v1 graph capture")
        ys = []
        for i in range(3):
            xi = to_gpu(make_image(4, 64, 64, seed=20 + i))
            eager = _sync_np(eng.forward(xi)).copy()
            if eng.graph is None:
                eng.capture()
                torch.cuda.synchronize()
            eng.x.copy_(xi)
            for _ in range(2):
                rep = _sync_np(eng.replay()).copy()
                assert np.array_equal(rep.view(np.uint32), eager.view(np.uint32)), "replay %d differs" % i
            ys.append(eager)
        assert not np.array_equal(ys[0], ys[1])
    finally:
        eng.close()


def test_library_loaded_before_torch_shares_its_runtime():
    """A fresh process that loads libspconv before importing torch (the
    binding imports torch first, so both use one HIP runtime) can plan and
    run; regression test for a second runtime instance finding no device."""
    import subprocess
    import sys
    import os
    code = ("import sys; sys.path.insert(0, %r)\n"
            "import paper_1911_09723_amd as P\n"
            "P.load_library()\n"
            "import numpy as np, torch\n"
            "from synth import make_layer\n"
            "l = make_layer(32, 16, 5, 5, 1, 0.5, seed=1)\n"
            "p = P.Plan.from_layer(l)\n"
            "y = p.run(torch.from_numpy(l.x).to('cuda:0'))\n"
            "torch.cuda.synchronize()\n"
            "print('ran', tuple(y.shape))\n") % os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    note("library before torch (subprocess)")
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=180)
    assert out.returncode == 0 and "ran (1, 16, 5, 5)" in out.stdout, out.stdout[-2000:] + out.stderr[-2000:]
