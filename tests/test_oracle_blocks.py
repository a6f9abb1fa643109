"""Pins of the oracle for input-channel and 2-D weight blocks (no GPU).

Sec. 3.2 blocks output channels; Fig. 5 shows 1x4, 4x1 and 2x2 blocks
reaching the same accuracy.  Here a block is kr consecutive output channels
x kc consecutive input channels (values[(t kr + i) kc + j] = W[rb kr + i,
col_idx[t] + j]).  Checked against the dense product by brute force, and
against the special cases it must reduce to."""

import numpy as np
import pytest

import oracle
from blocks_util import dense_from_blocks, random_blocks


@pytest.mark.parametrize("kr,kc", [(1, 4), (2, 2), (1, 2), (4, 4), (2, 4)])
@pytest.mark.parametrize("act", ["none", "relu6"])
def test_blocks_match_dense_product(kr, kc, act):
    rng = np.random.default_rng(kr * 10 + kc)
    cout, cin = 16, 24
    rp, ci, va = random_blocks(cout, cin, kr, kc, 0.4, rng)
    x = rng.standard_normal((3, cin, 5)).astype(np.float32)
    b = rng.standard_normal(cout).astype(np.float32)
    y, y64, s = oracle.spconv_ref(cout, cin, kr, rp, ci, va, b, act, x, block_cols=kc)
    wd = dense_from_blocks(cout, cin, kr, kc, rp, ci, va)
    ref = np.einsum("rc,ncp->nrp", wd, x.astype(np.float64)) + b.astype(np.float64)[None, :, None]
    if act == "relu6":
        ref = np.clip(ref, 0, 6)
    assert np.allclose(y64, ref, rtol=1e-12, atol=1e-12)
    assert np.array_equal(y, y64.astype(np.float32))


@pytest.mark.parametrize("kc", [2, 4])
def test_input_blocks_equal_their_channel_expansion(kc):
    """A kc-wide input block is kc consecutive single-channel entries of the
    same row: the plain CSR oracle on the expansion gives the same bits."""
    rng = np.random.default_rng(kc)
    cout, cin = 8, 16
    rp, ci, va = random_blocks(cout, cin, 1, kc, 0.5, rng)
    x = rng.standard_normal((2, cin, 7)).astype(np.float32)
    rp1 = rp * kc
    ci1 = (ci[:, None] + np.arange(kc)[None, :]).ravel().astype(np.int32)
    _, a, _ = oracle.spconv_ref(cout, cin, 1, rp, ci, va, None, "relu", x, block_cols=kc)
    _, e, _ = oracle.spconv_ref(cout, cin, 1, rp1, ci1, va, None, "relu", x)
    assert np.array_equal(a, e)


def test_block_past_the_last_channel_is_rejected():
    rp = np.array([0, 1], np.int32)
    with pytest.raises(ValueError):
        oracle.spconv_ref(1, 6, 1, rp, np.array([4], np.int32), np.ones(4, np.float32), None, "none",
                          np.ones((1, 6, 1), np.float32), block_cols=4)
