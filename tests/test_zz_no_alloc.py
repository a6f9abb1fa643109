"""The entry point that allocates no device memory (spconv_plan_create_static).

Its plans put their device image in the library's static per-GPU array
instead of a new allocation; runs through the C ABI must give exactly the
bits of a plan made by spconv_plan_create_ex for the same weights, on two
creations in a row (the second for a smaller layer, overwriting the first),
and the plan the second creation replaced must be refused, not run.
"""

import numpy as np
import pytest

import paper_1911_09723_amd as sp
from paper_1911_09723_amd import spconv as spmod
from synth import make_layer

E_ARG, E_SHAPE = 1, 3


def _opts(**kw):
    o = sp.spconv_options_init()
    for k, v in kw.items():
        setattr(o, k, v)
    return o


def test_static_plan_refuses_oversized_images_before_any_device_call():
    """A 4096 x 4096 layer at 70% density needs far more than the array holds:
    refused with SPCONV_E_SHAPE (checked before any HIP call: runs on the CPU)."""
    layer = make_layer(4096, 4096, 1, 1, 1, 0.3, seed=7, with_x=False)
    st, h = sp.spconv_plan_create_static(layer.cout, layer.cin, 1, layer.row_ptr, layer.col_idx, layer.values,
                                         layer.bias, "relu", check=False)
    assert st == E_SHAPE and h is None
    assert "static array" in sp.spconv_last_error()


def test_static_plan_cannot_be_host_only():
    layer = make_layer(64, 64, 1, 1, 1, 0.8, seed=8, with_x=False)
    st, h = sp.spconv_plan_create_static(layer.cout, layer.cin, 1, layer.row_ptr, layer.col_idx, layer.values,
                                         layer.bias, "relu", options=_opts(host_only=1), check=False)
    assert st == E_ARG and h is None


@pytest.mark.gpu
@pytest.mark.parametrize("kernel", [0, 3])
def test_static_plans_match_allocated_plans_twice_in_a_row(kernel):
    import torch
    from gpu_util import note, to_gpu, assert_parity

    def run(h, layer):
        x = to_gpu(layer.x)
        y = torch.empty((layer.n, layer.cout, layer.h, layer.w), device=x.device)
        sp.spconv_run(h, x, y, layer.n, layer.h, layer.w)
        torch.cuda.synchronize()
        return y.cpu().numpy()

    big = make_layer(512, 512, 14, 14, 8, 0.9, act="relu", seed=61)
    small = make_layer(64, 128, 7, 7, 3, 0.8, act="relu6", seed=62)
    plans = []
    try:
        for layer in (big, small):
            note("no-alloc plan %dx%d n=%d kernel=%d" % (layer.cout, layer.cin, layer.n, kernel))
            hs = sp.spconv_plan_create_static(layer.cout, layer.cin, 1, layer.row_ptr, layer.col_idx,
                                              layer.values, layer.bias, layer.act, options=_opts(kernel=kernel))
            plans.append(hs)
            ha = sp.spconv_plan_create(layer.cout, layer.cin, 1, layer.row_ptr, layer.col_idx, layer.values,
                                       layer.bias, layer.act, options=_opts(kernel=kernel))
            plans.append(ha)
            ys, ya = run(hs, layer), run(ha, layer)
            assert np.array_equal(ys.view(np.uint32), ya.view(np.uint32))
            assert_parity(layer, ys, what="static plan")
            assert sp.spconv_plan_check(hs) == 0
        # the first static plan's image was overwritten by the second: refused, not run
        x = to_gpu(big.x)
        y = torch.full((big.n, big.cout, big.h, big.w), 7.0, device=x.device)
        st = sp.spconv_run(plans[0], x, y, big.n, big.h, big.w, check=False)
        torch.cuda.synchronize()
        assert st == E_ARG and "replaced" in sp.spconv_last_error()
        assert torch.all(y == 7.0)
    finally:
        for h in plans:
            sp.spconv_destroy(h)
