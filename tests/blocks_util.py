"""Helpers for block-CSR weights with kr output x kc input channels per block
(tests only): values[(t * kr + i) * kc + j] = W[rb * kr + i, col_idx[t] + j]."""

import numpy as np


def dense_from_blocks(cout, cin, kr, kc, row_ptr, col_idx, values):
    """Scatter a block-CSR weight with kr x kc blocks into a dense fp64 matrix."""
    wd = np.zeros((cout, cin))
    for rb in range(cout // kr):
        for t in range(int(row_ptr[rb]), int(row_ptr[rb + 1])):
            for i in range(kr):
                for j in range(kc):
                    wd[rb * kr + i, int(col_idx[t]) + j] = values[(t * kr + i) * kc + j]
    return wd


def random_blocks(cout, cin, kr, kc, density, rng):
    """A random aligned kr x kc block-CSR weight."""
    rows, bcols = cout // kr, cin // kc
    mask = rng.random((rows, bcols)) < density
    row_ptr = np.concatenate([[0], np.cumsum(mask.sum(axis=1))]).astype(np.int32)
    col_idx = (np.nonzero(mask)[1] * kc).astype(np.int32)
    values = rng.standard_normal(int(mask.sum()) * kr * kc).astype(np.float32)
    return row_ptr, col_idx, values
