"""Dense masked weights -> block-CSR (paper Sec. 3.3: the library converts a
dense pruned weight to a block compressed sparse row form for inference;
Sec. 3.2: output-channel blocks of 2 and 4).  Host only: checks the C ABI's
detection and conversion against a plain numpy walk of the same definition,
and the round trip back to the dense matrix."""

import numpy as np
import pytest

import paper_1911_09723_amd.spconv as sp
from synth import densify


def _dense(cout, cin, k, density, seed, zero_in_blocks=False):
    """A dense weight whose mask is 1 x k blocked (k = 1: unstructured)."""
    rng = np.random.default_rng(seed)
    mask = np.repeat(rng.random((cout // k, cin)) < density, k, axis=0)
    w = rng.standard_normal((cout, cin)).astype(np.float32) * mask
    return np.where(w == 0, np.float32(0), w).astype(np.float32)


def _reference(dense, k):
    """Block (b, c) is stored when any of rows b*k .. b*k+k-1 is nonzero in column c."""
    cout, cin = dense.shape
    rp, ci, va = [0], [], []
    for b in range(cout // k):
        blk = dense[b * k:(b + 1) * k]
        for c in range(cin):
            if np.any(blk[:, c] != 0):
                ci.append(c)
                va.extend(blk[:, c].tolist())
        rp.append(len(ci))
    return (np.asarray(rp, np.int32), np.asarray(ci, np.int32), np.asarray(va, np.float32))


@pytest.mark.parametrize("k", [1, 2, 4])
@pytest.mark.parametrize("density", [0.0, 0.1, 0.5, 1.0])
def test_detect_block_rows(k, density):
    d = _dense(48, 40, k, density, seed=k)
    got = sp.spconv_detect_block_rows(d)
    if density in (0.0, 1.0):
        assert got == 4  # an empty or full mask is blocked at every height
    else:
        assert got == k


def test_detect_respects_cout_divisibility():
    d = _dense(6, 20, 2, 0.3, seed=3)  # 6 rows: 1x2 blocked, 4 does not divide 6
    assert sp.spconv_detect_block_rows(d) == 2
    d = _dense(7, 20, 1, 0.3, seed=3)
    assert sp.spconv_detect_block_rows(d) == 1


def test_negative_zero_counts_as_zero():
    d = _dense(8, 16, 4, 0.4, seed=5)
    d[1][d[1] == 0] = -0.0  # one row of a block with -0.0 where the others have zeros
    assert sp.spconv_detect_block_rows(d) == 4
    rp, ci, va = sp.spconv_dense_to_bcsr(d, 4)
    assert len(ci) == int(np.count_nonzero(d[0::4]))


@pytest.mark.parametrize("mask_k", [1, 2, 4])
@pytest.mark.parametrize("k", [1, 2, 4])
def test_conversion_matches_reference_and_round_trips(mask_k, k):
    d = _dense(64, 37, mask_k, 0.2, seed=10 * mask_k + k)
    rp, ci, va = sp.spconv_dense_to_bcsr(d, k)
    erp, eci, eva = _reference(d, k)
    assert np.array_equal(rp, erp) and np.array_equal(ci, eci)
    assert np.array_equal(va.view(np.uint32), eva.view(np.uint32))
    assert np.array_equal(densify(64, 37, k, rp, ci, va), d.astype(np.float64))
    if k <= mask_k:
        # a block height the mask has: no stored zero
        assert np.count_nonzero(va) == len(va) == np.count_nonzero(d)


def test_count_only_and_capacity():
    lib = sp.load_library()
    d = _dense(16, 24, 2, 0.3, seed=2)
    n = sp.ctypes.c_int64(-1)
    rp = np.zeros(9, np.int32)
    st = lib.spconv_dense_to_bcsr(16, 24, sp._ptr(d), 2, sp._ptr(rp), None, None, 0, sp.ctypes.byref(n))
    erp, eci, _ = _reference(d, 2)
    assert st == sp.OK and n.value == len(eci) and np.array_equal(rp, erp)
    ci = np.zeros(max(n.value - 1, 1), np.int32)
    va = np.zeros(2 * max(n.value - 1, 1), np.float32)
    st = lib.spconv_dense_to_bcsr(16, 24, sp._ptr(d), 2, sp._ptr(rp), sp._ptr(ci), sp._ptr(va), n.value - 1,
                                  sp.ctypes.byref(n))
    assert st == sp.E_ARG and n.value == len(eci) and "capacity" in sp.spconv_last_error()


@pytest.mark.parametrize("cout,k,expect", [(6, 4, sp.E_SHAPE), (8, 3, sp.E_UNSUPPORTED), (8, 0, sp.E_ARG),
                                           (0, 1, sp.E_SHAPE)])
def test_bad_shapes(cout, k, expect):
    lib = sp.load_library()
    d = np.ones((max(cout, 1), 4), np.float32)
    n = sp.ctypes.c_int64()
    st = lib.spconv_dense_to_bcsr(cout, 4, sp._ptr(d), k, None, None, None, 0, sp.ctypes.byref(n))
    assert st == expect


def test_non_finite_rejected():
    d = _dense(8, 8, 1, 0.5, seed=1)
    d[3, 5] = np.nan
    with pytest.raises(sp.SpconvError) as ei:
        sp.spconv_detect_block_rows(d)
    assert ei.value.status == sp.E_FORMAT and "[3][5]" in ei.value.message
    with pytest.raises(sp.SpconvError) as ei:
        sp.spconv_dense_to_bcsr(d, 1)
    assert ei.value.status == sp.E_FORMAT
    lib = sp.load_library()
    k = sp.ctypes.c_int32()
    assert lib.spconv_detect_block_rows(8, 8, None, sp.ctypes.byref(k)) == sp.E_ARG


def test_converted_weight_plans_like_the_block_csr():
    """The converted arrays are a valid plan input: a host-only plan unpacks to them."""
    d = _dense(96, 50, 2, 0.15, seed=8)
    k = sp.spconv_detect_block_rows(d)
    rp, ci, va = sp.spconv_dense_to_bcsr(d, k)
    opts = sp.spconv_options_init()
    opts.host_only = 1
    h = sp.spconv_plan_create(96, 50, k, rp, ci, va, options=opts)
    try:
        urp, uci, uva, _ = sp.spconv_plan_unpack(h)
    finally:
        sp.spconv_destroy(h)
    assert k == 2 and np.array_equal(urp, rp) and np.array_equal(uci, ci) and np.array_equal(uva, va)


# ---- blocks over input channels (4x1, 2x2, ...) ----

from blocks_util import dense_from_blocks, random_blocks  # noqa: E402


@pytest.mark.parametrize("kr,kc", [(1, 4), (2, 2), (4, 4), (1, 2), (4, 1), (2, 4)])
def test_blocked_detection_and_conversion_round_trip(kr, kc):
    rng = np.random.default_rng(kr * 10 + kc)
    cout, cin = 8 * kr, 12 * kc
    rp, ci, va = random_blocks(cout, cin, kr, kc, 0.4, rng)
    va[va == 0] = 1.0
    dense = dense_from_blocks(cout, cin, kr, kc, rp, ci, va).astype(np.float32)
    got = sp.spconv_detect_blocks(dense)
    # the detected shape holds at least as many weights and also describes the mask
    assert got[0] * got[1] >= kr * kc
    rp2, ci2, va2 = sp.spconv_dense_to_bcsr_blocked(dense, kr, kc)
    assert np.array_equal(rp2, rp) and np.array_equal(ci2, ci) and np.array_equal(va2, va)
    rp3, ci3, va3 = sp.spconv_dense_to_bcsr_blocked(dense, *got)
    assert np.array_equal(dense_from_blocks(cout, cin, got[0], got[1], rp3, ci3, va3), dense)
    assert np.count_nonzero(va3) == np.count_nonzero(dense)  # the detected blocks store no zero


def test_detection_prefers_output_blocks_on_a_tie():
    """The most weights per block wins; among equals the output-channel block."""
    dense = np.zeros((8, 8), np.float32)
    dense[0:4, 0:4] = 1.0  # one 4x4 block: 4x4 wins
    assert sp.spconv_detect_blocks(dense) == (4, 4)
    dense = np.zeros((4, 6), np.float32)
    dense[:, 2] = 1.0  # 4 x 1 column: only output blocks of 4 (cin 6 is not a multiple of 4)
    assert sp.spconv_detect_blocks(dense) == (4, 1)
    dense = np.zeros((2, 2), np.float32)
    dense[0, 0] = 1.0  # no block shape fits
    assert sp.spconv_detect_blocks(dense) == (1, 1)


def test_blocked_conversion_errors():
    dense = np.ones((4, 6), np.float32)
    lib = sp.load_library()
    import ctypes
    n = ctypes.c_int64()
    assert lib.spconv_dense_to_bcsr_blocked(4, 6, dense.ctypes.data_as(ctypes.c_void_p), 1, 4, None, None, None, 0,
                                            ctypes.byref(n)) == sp.E_SHAPE
    assert lib.spconv_dense_to_bcsr_blocked(4, 6, dense.ctypes.data_as(ctypes.c_void_p), 1, 3, None, None, None, 0,
                                            ctypes.byref(n)) == sp.E_UNSUPPORTED
    st, h = sp.spconv_plan_create_dense_blocked(dense, 0, 2, check=False)
    assert st == sp.E_ARG and h is None


def test_tie_between_output_and_input_blocks():
    """A 4 x 4 mask block is also 4x1, 1x4 and 2x2 blocked: 4x4 wins; a 2 x 2
    block (2x2 vs nothing larger) reports (2, 2) over (2, 1) and (1, 2)."""
    dense = np.zeros((4, 4), np.float32)
    dense[0:2, 2:4] = 3.0
    assert sp.spconv_detect_blocks(dense) == (2, 2)
