"""The C ABI and the host planner, without a GPU.

* libspconv.so loads and exports every function include/spconv.h declares;
* malformed CSR / block-CSR input is rejected with the documented status
  before any device work;
* host-only plans: the packed image unpacks back to the input exactly, the
  processing order is a permutation sorted by nonzero count, the wave
  assignment is balanced, fp16 storage rounds weights to nearest-even.
"""

import ctypes
import os
import re
import subprocess
import sys

import numpy as np
import pytest

import paper_1911_09723_amd as sp
from paper_1911_09723_amd import spconv as spmod
from synth import make_layer

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "spconv.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"\b(spconv_[a-z0-9_]+)\s*\(", text)
    return sorted(set(names))


def test_header_declares_the_boundary():
    names = _declared_functions()
    for required in ("spconv_plan_create", "spconv_run", "spconv_destroy", "spconv_last_error"):
        assert required in names
    assert set(names) == set(spmod.EXPORTED)


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(spmod.LIBRARY_PATH)
    for name in _declared_functions():
        assert hasattr(lib, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", spmod.LIBRARY_PATH], capture_output=True, text=True)
    exported = set(re.findall(r" T (spconv_\w+)", out.stdout))
    assert set(_declared_functions()) <= exported


def _host_opts(**kw):
    o = sp.spconv_options_init()
    o.host_only = 1
    for k, v in kw.items():
        setattr(o, k, v)
    return o


def _create(layer=None, check=True, **kw):
    args = dict(cout=64, cin=32, block_rows=1, row_ptr=None, col_idx=None, values=None, bias=None,
                act="relu", storage="f32")
    if layer is not None:
        args.update(cout=layer.cout, cin=layer.cin, block_rows=layer.block_rows, row_ptr=layer.row_ptr,
                    col_idx=layer.col_idx, values=layer.values, bias=layer.bias, act=layer.act,
                    storage=layer.storage)
    opts = kw.pop("options", None) or _host_opts()
    args.update(kw)
    return sp.spconv_plan_create(args["cout"], args["cin"], args["block_rows"], args["row_ptr"],
                                 args["col_idx"], args["values"], args["bias"], args["act"], args["storage"],
                                 options=opts, check=check)


def _status(**kw):
    layer = kw.pop("layer", None) or make_layer(32, 64, 2, 2, 1, 0.8, seed=1, with_x=False)
    st, h = _create(layer, check=False, **kw)
    if h:
        sp.spconv_destroy(h)
    return st, sp.spconv_last_error()


def test_valid_host_plan():
    st, msg = _status()
    assert st == sp.spconv.OK and msg == ""


@pytest.mark.parametrize("mutate,expect,words", [
    (lambda L: L.row_ptr.__setitem__(0, 1), sp.spconv.E_FORMAT, "row_ptr[0]"),
    (lambda L: L.row_ptr.__setitem__(5, L.row_ptr[4] - 1), sp.spconv.E_FORMAT, "decreases"),
    (lambda L: L.col_idx.__setitem__(3, 32), sp.spconv.E_FORMAT, "outside"),
    (lambda L: L.col_idx.__setitem__(0, -1), sp.spconv.E_FORMAT, "outside"),
    (lambda L: L.values.__setitem__(2, np.nan), sp.spconv.E_FORMAT, "not finite"),
    (lambda L: L.values.__setitem__(2, np.inf), sp.spconv.E_FORMAT, "not finite"),
    (lambda L: L.bias.__setitem__(2, np.inf), sp.spconv.E_FORMAT, "bias"),
])
def test_malformed_csr_rejected(mutate, expect, words):
    layer = make_layer(32, 64, 2, 2, 1, 0.8, seed=1, with_x=False)
    mutate(layer)
    st, msg = _status(layer=layer)
    assert st == expect and words in msg, (st, msg)


def test_duplicate_or_unsorted_columns_rejected():
    layer = make_layer(32, 64, 2, 2, 1, 0.8, seed=1, with_x=False)
    s = layer.row_ptr[3]
    assert layer.row_ptr[4] - s >= 2
    layer.col_idx[s + 1] = layer.col_idx[s]
    st, msg = _status(layer=layer)
    assert st == sp.spconv.E_FORMAT and "ascending" in msg


@pytest.mark.parametrize("kw,expect", [
    (dict(cout=63, block_rows=4), sp.spconv.E_SHAPE),
    (dict(cout=0), sp.spconv.E_SHAPE),
    (dict(cin=0), sp.spconv.E_SHAPE),
    (dict(block_rows=3), sp.spconv.E_UNSUPPORTED),
    (dict(block_rows=8), sp.spconv.E_UNSUPPORTED),
    (dict(block_rows=0), sp.spconv.E_ARG),
    (dict(act=7), sp.spconv.E_ARG),
    (dict(storage=5), sp.spconv.E_ARG),
    (dict(row_ptr=None), sp.spconv.E_ARG),
])
def test_bad_arguments(kw, expect):
    layer = make_layer(32, 64, 2, 2, 1, 0.8, seed=1, with_x=False)
    if kw.get("row_ptr", 1) is None:
        layer.row_ptr = None
        kw = {}
    st, msg = _status(layer=layer, **kw)
    assert st == expect and msg, (st, msg)


def test_null_arrays_with_nonzeros_rejected():
    layer = make_layer(32, 64, 2, 2, 1, 0.8, seed=1, with_x=False)
    layer.col_idx = None
    st, msg = _status(layer=layer)
    assert st == sp.spconv.E_ARG and "NULL" in msg


def test_options_validated():
    for kw in (dict(group_lanes=2), dict(group_lanes=12), dict(group_lanes=32), dict(group_lanes=-4),
               dict(waves=17), dict(waves=-1), dict(reorder=2), dict(host_only=3), dict(kernel=6),
               dict(kernel=-1), dict(pipe_sets=3), dict(pipe_sets=-1), dict(regions=5), dict(regions=-1)):
        st, msg = _status(options=_host_opts(**kw))
        assert st == sp.spconv.E_ARG, kw
    o = _host_opts()
    o.struct_size = 4
    st, msg = _status(options=o)
    assert st == sp.spconv.E_ARG and "struct_size" in msg


def test_out_null_and_destroy_null():
    lib = sp.load_library()
    assert lib.spconv_plan_create(None, 4, 4, 1, None, None, None, None, 0, 0) == sp.spconv.E_ARG
    assert lib.spconv_destroy(None) == sp.spconv.OK


def test_run_refuses_host_only_plan_and_null_plan():
    layer = make_layer(32, 64, 2, 2, 1, 0.8, seed=1, with_x=False)
    h = _create(layer)
    try:
        assert sp.spconv_run(h, 1 << 20, 2 << 20, 1, 2, 2, stream=0, check=False) == sp.spconv.E_ARG
        assert "host_only" in sp.spconv_last_error()
    finally:
        sp.spconv_destroy(h)
    assert sp.load_library().spconv_run(None, None, None, 1, 1, 1, None) == sp.spconv.E_ARG


def test_injected_allocation_failure_reports_nomem():
    code = ("import paper_1911_09723_amd as sp; from synth import make_layer;"
            "L = make_layer(32, 64, 2, 2, 1, 0.8, seed=1, with_x=False);"
            "st, h = sp.spconv_plan_create(L.cout, L.cin, 1, L.row_ptr, L.col_idx, L.values, L.bias,"
            " 'relu', 'f32', check=False);"
            "print(st, h, sp.spconv_last_error())")
    env = dict(os.environ, SPCONV_FAULT="alloc", PYTHONPATH=ROOT)
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env, cwd=ROOT)
    assert out.returncode == 0, out.stderr
    st, h, msg = out.stdout.split(" ", 2)
    assert int(st) == sp.spconv.E_NOMEM and h == "None" and "SPCONV_FAULT" in msg


@pytest.mark.parametrize("k", [1, 2, 4])
@pytest.mark.parametrize("pattern", ["uniform", "beta"])
@pytest.mark.parametrize("kernel,group_lanes", [(0, 0), (1, 4), (1, 8), (1, 16), (2, 0), (2, 8)])
def test_pack_unpack_round_trip_and_order(k, pattern, kernel, group_lanes):
    if pattern == "beta" and k > 1:
        pytest.skip("beta row densities are defined for unstructured masks")
    layer = make_layer(96, 160, 2, 2, 1, 0.85, block_rows=k, pattern=pattern, seed=4, with_x=False)
    h = _create(layer, options=_host_opts(kernel=kernel, group_lanes=group_lanes))
    try:
        info = sp.spconv_plan_get_info(h)
        rp, ci, va, perm = sp.spconv_plan_unpack(h)
        if info["kernel"] == 0:
            irp, ici, iva = sp.spconv_plan_unpack_interleaved(h)
        else:
            with pytest.raises(sp.SpconvError) as ei:
                sp.spconv_plan_unpack_interleaved(h)
            assert ei.value.status == sp.spconv.E_FORMAT
            irp, ici, iva = rp, ci, va
    finally:
        sp.spconv_destroy(h)
    assert np.array_equal(rp, layer.row_ptr) and np.array_equal(ci, layer.col_idx)
    assert np.array_equal(va, layer.values)
    assert np.array_equal(irp, rp) and np.array_equal(ici, ci) and np.array_equal(iva, va)
    rows = 160 // k
    assert sorted(perm.tolist()) == list(range(rows))
    counts = np.diff(layer.row_ptr)[perm]
    assert np.all(np.diff(counts) <= 0), "rows not in descending nonzero order"
    ties = [perm[i] < perm[i + 1] for i in range(rows - 1) if counts[i] == counts[i + 1]]
    assert all(ties), "equal-length rows not kept in index order"
    assert info["nnzb"] == layer.nnzb and info["slots"] >= layer.nnzb
    assert info["group_lanes"] in (4, 8, 16) and (group_lanes == 0 or info["group_lanes"] == group_lanes)
    assert info["bundle_rows"] * info["group_lanes"] == 64
    assert info["cols_per_lane"] == (16 // info["group_lanes"]) * 4
    assert info["kernel"] == (1 if kernel == 2 else 0)
    # whole steps of 4 slots for every group of a bundle
    assert info["slots"] % (4 * info["bundle_rows"]) == 0


@pytest.mark.parametrize("sets", [0, 1, 2])
@pytest.mark.parametrize("regions", [0, 1, 2, 3, 4])
@pytest.mark.parametrize("shape", [(512, 512, 1, "uniform", 1), (37, 80, 1, "uniform", 1),
                                   (200, 120, 1, "beta", 0), (3, 8, 1, "uniform", 1), (96, 64, 4, "uniform", 1),
                                   (601, 48, 1, "uniform", 1)])
def test_interleaved_streams_walk_back_to_the_input(shape, regions, sets):
    """The pipelined kernel's streams, walked with its own bookkeeping (set and
    last-step bits, strip parts between need and release events), give back
    every row's blocks in order."""
    cin, cout, k, pattern, reorder = shape
    layer = make_layer(cin, cout, 1, 1, 1, 0.85, block_rows=k, pattern=pattern, seed=cin + cout,
                       with_x=False)
    opts = _host_opts(pipe_sets=sets, regions=regions, reorder=reorder, group_lanes=16 if k == 4 else 0)
    st, h = _create(layer, options=opts, check=False)
    if sets == 2 and k == 4 and st == sp.spconv.E_UNSUPPORTED:
        return
    assert st == sp.spconv.OK, sp.spconv_last_error()
    try:
        info = sp.spconv_plan_get_info(h)
        rp, ci, va = sp.spconv_plan_unpack_interleaved(h)
    finally:
        sp.spconv_destroy(h)
    assert info["kernel"] == 0
    assert info["pipe_sets"] == (sets or info["pipe_sets"]) and info["pipe_sets"] in (1, 2)
    strip_rows = -(-cin // 4) * 4
    assert 1 <= info["regions"] <= min(regions or 4, strip_rows // 4)
    assert np.array_equal(rp, layer.row_ptr) and np.array_equal(ci, layer.col_idx)
    assert np.array_equal(va, layer.values)


@pytest.mark.parametrize("cin,parts", [(512, 3), (128, 1), (144, 1), (256, 2), (576, 3), (768, 4)])
def test_headline_plan_interleaves_two_bundles_over_strip_parts(cin, parts):
    """Two interleaved bundles per wavefront, and about one strip part per
    192 input channels (at most 4)."""
    layer = make_layer(cin, 512, 1, 1, 1, 0.9, seed=5, with_x=False)
    h = _create(layer)
    try:
        info = sp.spconv_plan_get_info(h)
    finally:
        sp.spconv_destroy(h)
    if info["kernel"] != 0 or info["regions"] == 0:
        pytest.skip("not a strip-kernel plan at cin %d" % cin)
    assert (info["group_lanes"], info["waves"], info["pipe_sets"], info["regions"]) == (4, 16, 2, parts)


def test_two_sets_refused_when_accumulators_do_not_fit():
    # 1x4 blocks take 8 lanes per block row: 4 x 8 accumulators per set
    layer = make_layer(256, 512, 1, 1, 1, 0.9, block_rows=4, seed=1, with_x=False)
    st, msg = _status(layer=layer, options=_host_opts(pipe_sets=2))
    assert st == sp.spconv.E_UNSUPPORTED and "accumulators" in msg
    st, msg = _status(layer=layer, options=_host_opts(pipe_sets=2, group_lanes=16))
    assert st == sp.spconv.OK


def test_natural_order_when_reorder_off():
    layer = make_layer(64, 64, 2, 2, 1, 0.8, seed=5, with_x=False)
    h = _create(layer, options=_host_opts(reorder=0))
    try:
        _, _, _, perm = sp.spconv_plan_unpack(h)
    finally:
        sp.spconv_destroy(h)
    assert np.array_equal(perm, np.arange(64))


def test_lpt_balance_on_uniform_rows():
    layer = make_layer(512, 512, 1, 1, 1, 0.9, seed=2020, with_x=False)
    h = _create(layer)
    try:
        info = sp.spconv_plan_get_info(h)
    finally:
        sp.spconv_destroy(h)
    # 32 bundles of 16 rows on 16 wavefronts: two each, longest paired with shortest
    assert info["group_lanes"] == 4 and info["waves"] == 16
    assert info["max_wave_cost"] <= 1.07 * info["sum_wave_cost"] / info["waves"]
    # bundles are whole steps of 4 slots padded to their longest row (rows sorted by length)
    assert info["slots"] <= 1.06 * layer.nnzb


def test_lpt_balance_on_heavy_tailed_rows():
    layer = make_layer(960, 160, 1, 1, 1, 0.85, pattern="beta", seed=3070, with_x=False)
    h = _create(layer)
    try:
        info = sp.spconv_plan_get_info(h)
    finally:
        sp.spconv_destroy(h)
    mean = info["sum_wave_cost"] / info["waves"]
    # LPT bound: max load <= mean + largest single job
    counts = np.sort(np.diff(layer.row_ptr))[::-1]
    largest_bundle = counts[0] + 3
    assert info["max_wave_cost"] <= mean + largest_bundle


def test_geometry_choice():
    def info_for(cin, cout, storage, k=1, **opts):
        layer = make_layer(cin, cout, 1, 1, 1, 0.9, block_rows=k, storage=storage, seed=1, with_x=False)
        h = _create(layer, options=_host_opts(**opts))
        try:
            return sp.spconv_plan_get_info(h)
        finally:
            sp.spconv_destroy(h)

    def table(cout, k, nb):
        # per bundle: the block row and the k biases of each of its nb groups, 16-byte rounded,
        # then 32 bytes of counters
        bundles = -(-(cout // k) // nb)
        return -(-(bundles * nb * (1 + k) * 4) // 16) * 16 + 32

    def check(i, kernel, g, tile_cols, cin, cout, k):
        nb = 64 // g
        assert (i["kernel"], i["group_lanes"], i["bundle_rows"], i["tile_cols"]) == (kernel, g, nb, tile_cols)
        # the strip's rows and one row of zeros for padding slots
        strip = 0 if kernel == 1 else (-(-cin // 4) * 4 + 1) * 256
        assert i["lds_bytes"] == strip + table(cout, k, nb)
        assert i["waves"] == min(16, -(-(cout // k) // nb))

    # unstructured fp32: 4 lanes per row, 16 columns per lane, 256-byte strip rows
    check(info_for(512, 512, "f32"), 0, 4, 64, 512, 512, 1)
    # 1x4 blocks: 4 x 16 accumulators would crowd the registers, so 8 lanes per row
    check(info_for(512, 512, "f32", 4), 0, 8, 64, 512, 512, 4)
    # 1x2 blocks: 2 x 16 accumulators fit, so 4 lanes per row
    check(info_for(512, 512, "f32", 2), 0, 4, 64, 512, 512, 2)
    # fp16: 128 columns per tile; 1x4 blocks take 16 lanes per row
    check(info_for(320, 1280, "f16", 4), 0, 16, 128, 320, 1280, 4)
    check(info_for(320, 1280, "f16", 1), 0, 4, 128, 320, 1280, 1)
    # few rows: wider lane groups keep enough bundles for the wavefronts
    check(info_for(24, 32, "f32"), 0, 16, 64, 24, 32, 1)
    check(info_for(144, 24, "f32"), 0, 16, 64, 144, 24, 1)
    # inputs too wide for an LDS strip: the direct-load kernel, 16 lanes per row
    check(info_for(1024, 256, "f32"), 1, 16, 64, 1024, 256, 1)
    check(info_for(600, 256, "f32"), 0, 4, 64, 600, 256, 1)
    check(info_for(640, 256, "f32"), 1, 16, 64, 640, 256, 1)
    check(info_for(1152, 192, "f16", 4), 1, 16, 128, 1152, 192, 4)
    # an explicit lane width still holds on the direct-load kernel
    assert info_for(1024, 256, "f32", group_lanes=4)["group_lanes"] == 4
    # forced choices
    i = info_for(512, 512, "f32", group_lanes=16, waves=7)
    assert i["group_lanes"] == 16 and i["waves"] == 7
    assert info_for(512, 512, "f32", kernel=2)["kernel"] == 1


def test_group_lanes_beyond_the_accumulator_limit_rejected():
    layer = make_layer(64, 64, 1, 1, 1, 0.9, block_rows=4, storage="f16", seed=1, with_x=False)
    st, msg = _status(layer=layer, options=_host_opts(group_lanes=4))
    assert st == sp.spconv.E_UNSUPPORTED and "accumulators" in msg
    st, msg = _status(layer=layer, options=_host_opts(group_lanes=8))
    assert st == sp.spconv.OK


def test_strip_refused_when_it_does_not_fit():
    layer = make_layer(1024, 64, 1, 1, 1, 0.9, seed=1, with_x=False)
    st, msg = _status(layer=layer, options=_host_opts(kernel=1))
    assert st == sp.spconv.E_UNSUPPORTED and "LDS" in msg


def test_f16_weights_rounded_to_nearest_even():
    rng = np.random.default_rng(0)
    special = np.array([1.0, 1 + 2 ** -11, 1 + 3 * 2 ** -11, 65504.0, 65519.0, 6e-8, 2.0 ** -25,
                        3 * 2.0 ** -26, -2.0 ** -24, 1e-10, 0.0, -0.0, 5.96e-8, 6.1e-5, 6.09e-5],
                       dtype=np.float32)
    vals = np.concatenate([special, (rng.standard_normal(4000) * rng.choice([1e-6, 1e-3, 1, 300], 4000))
                           .astype(np.float32)])
    n = vals.size
    cin = n
    rp = np.array([0, n], np.int32)
    ci = np.arange(n, dtype=np.int32)
    h = sp.spconv_plan_create(1, cin, 1, rp, ci, vals, None, "none", "f16", options=_host_opts())
    try:
        _, _, va, _ = sp.spconv_plan_unpack(h)
    finally:
        sp.spconv_destroy(h)
    expect = vals.astype(np.float16).astype(np.float32)
    assert np.array_equal(va.view(np.uint32), expect.view(np.uint32))


def test_network_operators_reject_bad_arguments():
    """Argument checks of the network operators run before any HIP call: the
    addresses below are never dereferenced (stream 0 keeps the binding off
    torch's device state, so this runs without a GPU)."""
    from paper_1911_09723_amd import (spconv, spconv_conv3x3_hwc, spconv_depthwise3x3, spconv_global_avg_pool,
                                      spconv_linear)
    kw = dict(stream=0, check=False)
    assert spconv_conv3x3_hwc(1 << 40, 1 << 41, None, "relu", 3, 1 << 42, 1, 4, 4, 3, 8, **kw) == spconv.E_ARG
    assert spconv_conv3x3_hwc(1 << 40, 1 << 41, None, "relu", 2, 1 << 42, 1, 4, 4, 9, 8, **kw) == \
        spconv.E_UNSUPPORTED
    assert spconv_conv3x3_hwc(None, None, None, "relu", 2, None, 0, 4, 4, 3, 8, **kw) == spconv.OK
    assert spconv_depthwise3x3(1 << 40, 1 << 41, None, "relu", 2, 1 << 40, 1, 4, 4, 4, **kw) == spconv.E_ARG
    assert spconv_global_avg_pool(1 << 40, 1 << 41, 1, 4, 0, 3, **kw) == spconv.E_SHAPE
    assert spconv_global_avg_pool(None, None, 0, 4, 3, 3, **kw) == spconv.OK
    assert spconv_linear(1 << 40, 1 << 41, None, "none", 1 << 42, 2, 0, 5, **kw) == spconv.E_SHAPE
    assert spconv_linear(1 << 40, 1 << 41, None, "none", 1 << 42, 300000, 4, 5, **kw) == spconv.E_SHAPE
    assert spconv_linear(None, None, None, "none", None, 0, 4, 5, **kw) == spconv.OK


@pytest.mark.parametrize("kernel", [0, 3])
@pytest.mark.parametrize("fused", [False, True])
def test_run_rejects_tiles_whose_images_span_2gib(fused, kernel):
    """Two 1024 x 1024 images of 300 channels: one tile touches both, 2.5 GB of
    x, beyond the kernels' 32-bit offsets, so spconv_run refuses the call.  The
    check runs before any HIP call, so a host-only plan reaches it; images of
    a quarter the size pass it and only then meet the host-only refusal."""
    from synth import make_depthwise
    if fused and kernel == 3:
        pytest.skip("the register-indexed kernel has no depthwise stage")
    layer = make_layer(300, 8, 1, 1, 1, 0.5, act="relu", seed=91, with_x=False)
    o = _host_opts(kernel=kernel)
    if fused:
        kw, kb = make_depthwise(300, 92)
        h = sp.spconv_plan_create_fused(8, 300, 1, layer.row_ptr, layer.col_idx, layer.values, layer.bias, "relu",
                                        kw, kb, "none", 1, options=o)
    else:
        h = _create(layer, options=o)
    try:
        st = sp.spconv_run(h, 1 << 44, 1 << 45, 2, 1024, 1024, stream=0, check=False)
        assert st == sp.spconv.E_UNSUPPORTED and "2^31" in sp.spconv_last_error()
        st = sp.spconv_run(h, 1 << 44, 1 << 45, 4, 512, 512, stream=0, check=False)
        assert st == sp.spconv.E_ARG and "host_only" in sp.spconv_last_error()
    finally:
        sp.spconv_destroy(h)


@pytest.mark.parametrize("cin,passes", [(1024, 2), (960, 2), (1280, 3), (512, 1), (100, 1)])
def test_channel_range_passes_split_wide_inputs(cin, passes):
    """Kernel option 5: ranges of at most 512 input channels, one pass each."""
    layer = make_layer(cin, 96, 1, 1, 1, 0.9, seed=cin, with_x=False)
    h = _create(layer, options=_host_opts(kernel=5))
    try:
        info = sp.spconv_plan_get_info(h)
        rp, ci, va, _ = sp.spconv_plan_unpack(h)
    finally:
        sp.spconv_destroy(h)
    assert info["channel_passes"] == passes
    assert np.array_equal(rp, layer.row_ptr) and np.array_equal(ci, layer.col_idx)
    assert np.array_equal(va, layer.values)


@pytest.mark.parametrize("kw", [dict(block_rows=4), dict(storage="f16")], ids=["1x4", "f16"])
def test_channel_range_passes_refused_outside_fp32_unstructured(kw):
    layer = make_layer(1024, 96, 1, 1, 1, 0.9, seed=7, with_x=False, **kw)
    st, h = _create(layer, check=False, options=_host_opts(kernel=5))
    assert st == sp.spconv.E_UNSUPPORTED and not h, st
    assert "channel-range" in sp.spconv_last_error()


@pytest.mark.parametrize("cin,passes", [(1280, 3), (1264, 0), (2048, 4)])
def test_automatic_choice_takes_passes_beyond_the_lockstep_width(cin, passes):
    """Kernel option 0: fp32 unstructured inputs wider than 1264 channels run
    as channel-range passes; narrower ones do not."""
    layer = make_layer(cin, 64, 1, 1, 1, 0.9, seed=cin, with_x=False)
    h = _create(layer, options=_host_opts())
    try:
        assert sp.spconv_plan_get_info(h)["channel_passes"] == passes
    finally:
        sp.spconv_destroy(h)
