"""The seeded input generator draws what the workloads describe (no GPU)."""

import numpy as np
import pytest

from synth import make_layer, CONFIGS, config_layers, layer_seed
from synth.configs import build


def _check_csr(layer):
    rp, ci = layer.row_ptr, layer.col_idx
    rows = layer.cout // layer.block_rows
    assert rp.dtype == np.int32 and ci.dtype == np.int32
    assert rp.shape == (rows + 1,) and rp[0] == 0 and np.all(np.diff(rp) >= 0)
    assert ci.shape == (rp[-1],) and np.all((ci >= 0) & (ci < layer.cin))
    for r in range(rows):
        seg = ci[rp[r]:rp[r + 1]]
        assert np.all(np.diff(seg) > 0)
    assert layer.values.shape == (rp[-1] * layer.block_rows,)


@pytest.mark.parametrize("k", [1, 4])
@pytest.mark.parametrize("s", [0.7, 0.8, 0.9, 0.95])
def test_exact_uniform_count(k, s):
    layer = make_layer(64, 96, 2, 2, 1, s, block_rows=k, seed=1)
    _check_csr(layer)
    assert layer.nnzb == round((1 - s) * (96 // k) * 64)


def test_beta_rows_exact_total_and_heavy_tail():
    layer = make_layer(960, 160, 1, 1, 1, 0.85, pattern="beta", seed=layer_seed(3, 7, 0), with_x=False)
    _check_csr(layer)
    counts = np.diff(layer.row_ptr)
    assert counts.sum() == round(0.15 * 960 * 160)
    assert counts.max() > 2.5 * counts.mean()


def test_values_and_x_distribution():
    layer = make_layer(200, 200, 16, 16, 4, 0.5, seed=2)
    std_w = np.sqrt(2 / (0.1 * 200))
    assert abs(layer.values.std() / std_w - 1) < 0.05
    assert abs(layer.bias.std() / 0.1 - 1) < 0.3
    assert layer.x.min() == 0 and abs((layer.x == 0).mean() - 0.5) < 0.01


def test_f16_values_are_representable():
    layer = make_layer(40, 240, 7, 7, 2, 0.9, block_rows=4, storage="f16", seed=3)
    assert layer.x.dtype == np.float16
    assert np.array_equal(layer.values.astype(np.float16).astype(np.float32), layer.values)


def test_deterministic():
    a = make_layer(32, 64, 5, 5, 2, 0.9, seed=123)
    b = make_layer(32, 64, 5, 5, 2, 0.9, seed=123)
    assert all(np.array_equal(getattr(a, f), getattr(b, f)) for f in ("row_ptr", "col_idx", "values", "bias", "x"))


def test_all_workloads_have_expected_nnz():
    expect_nnz = {0: [205], 2: [78643, 78644, 52429, 52428, 26214, 26216, 13107, 13108],
                  4: [960, 3840, 7528, 22120, 40960]}
    for c in CONFIGS:
        specs = config_layers(c)
        for i, spec in enumerate(specs):
            layer = build(c, spec, with_x=False)
            _check_csr(layer)
            if c in expect_nnz:
                assert layer.nnz == expect_nnz[c][i], (c, spec["name"])
    assert len(config_layers(1)) == 26 and len(config_layers(3)) == 9
