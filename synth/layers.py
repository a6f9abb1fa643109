"""Synthetic sparse 1x1-convolution layers with the shapes of the paper's networks.

The paper (Sec. 3.2, Fig. 2) treats a 1x1 convolution over a CHW activation
tensor as a sparse-weight x dense-activation product: W is Cout x Cin and
sparse, X is Cin x (H*W) and dense.  Sec. 3.2 also introduces output-channel
blocks: k consecutive output channels share one sparsity pattern.  Sec. 3.3
names a block-compressed-sparse-row (BCSR-like) weight format; that is the
layout produced here:

* ``row_ptr``  int32[Cout/k + 1]  -- block-row offsets into ``col_idx``
* ``col_idx``  int32[nnzb]        -- input channel of each block, ascending per row
* ``values``   float32[nnzb * k]  -- block-major: values[b*k + i] = W[rb*k + i, col_idx[b]]
* ``bias``     float32[Cout]
* ``x``        float32 or float16 [N, Cin, H, W]  (NCHW: each channel's H*W plane contiguous)

Value recipe (the paper trains on ImageNet; trained weights are not available,
so these seeded draws stand in for them):

* mask first, then weight values, then bias, then X, all from one
  ``numpy.random.Generator(PCG64(seed))``;
* uniform masks draw exactly round((1 - s) * (Cout/k) * Cin) block positions
  without replacement;
* "beta" masks draw a per-row density from Beta(1.5, 8.5), rescale it so the
  layer's total density is 1 - s, and integerise with largest-remainder
  rounding so the total count is exact; each row's columns are then uniform
  without replacement (rows may be empty);
* W ~ N(0, variance 2 / (0.1 * Cin)), bias ~ N(0, variance 0.01),
  X = max(0, N(0, 1)) (about half of X is exactly zero and is kept dense);
* fp16 storage: W values are rounded to the nearest fp16 value (kept as
  float32 so both sides see identical weights) and X is rounded to fp16.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional

import numpy as np

ACTS = ("none", "relu", "relu6")
STORAGES = ("f32", "f16")


@dataclass
class Layer:
    cin: int
    cout: int
    h: int
    w: int
    n: int
    block_rows: int
    sparsity: float
    pattern: str
    storage: str
    act: str
    seed: int
    row_ptr: np.ndarray = field(repr=False)
    col_idx: np.ndarray = field(repr=False)
    values: np.ndarray = field(repr=False)
    bias: np.ndarray = field(repr=False)
    x: Optional[np.ndarray] = field(default=None, repr=False)
    block_cols: int = 1  # input channels per block (values[(t * block_rows + i) * block_cols + j])

    @property
    def hw(self) -> int:
        return self.h * self.w

    @property
    def nnzb(self) -> int:
        return int(self.row_ptr[-1])

    @property
    def nnz(self) -> int:
        """Stored weight values (block_rows x block_cols per block)."""
        return self.nnzb * self.block_rows * self.block_cols

    @property
    def x_dtype(self):
        return np.float16 if self.storage == "f16" else np.float32

    def flops(self, n: Optional[int] = None) -> float:
        """Effective FLOPs 2 * nnz * H * W * N (bias and activation not counted)."""
        n = self.n if n is None else n
        return 2.0 * self.nnz * self.hw * n

    def alg_bytes(self, n: Optional[int] = None) -> float:
        """Algorithmic HBM bytes: X read once, Y written once, plus the weights.

        Weight bytes: one value per stored element at the storage width, one
        int32 index per block, int32 row pointers, fp32 bias.
        """
        n = self.n if n is None else n
        e = 2 if self.storage == "f16" else 4
        act_bytes = e * n * self.hw * (self.cin + self.cout)
        w_bytes = e * self.nnz + 4 * self.nnzb + 4 * (self.cout // self.block_rows + 1) + 4 * self.cout
        return float(act_bytes + w_bytes)


def _uniform_mask(rng, rows: int, cin: int, density: float):
    nnzb = int(round(density * rows * cin))
    pos = np.sort(rng.choice(rows * cin, size=nnzb, replace=False))
    r = (pos // cin).astype(np.int64)
    c = (pos % cin).astype(np.int32)
    counts = np.bincount(r, minlength=rows)
    row_ptr = np.zeros(rows + 1, dtype=np.int64)
    np.cumsum(counts, out=row_ptr[1:])
    return row_ptr.astype(np.int32), c


def _beta_counts(rng, rows: int, cin: int, density: float):
    """Per-row nonzero counts with Beta(1.5, 8.5) row densities, exact total."""
    total = int(round(density * rows * cin))
    p = rng.beta(1.5, 8.5, size=rows)
    target = density * rows  # sum of row densities
    scaled = p * (target / p.sum())
    # Clip to [0, 1]; hand the clipped excess back to the unclipped rows.
    for _ in range(64):
        over = scaled > 1.0
        if not over.any():
            break
        excess = (scaled[over] - 1.0).sum()
        scaled[over] = 1.0
        free = ~over & (scaled < 1.0)
        scaled[free] += excess * scaled[free] / scaled[free].sum()
    exact = scaled * cin
    counts = np.floor(exact).astype(np.int64)
    counts = np.minimum(counts, cin)
    short = total - int(counts.sum())
    if short > 0:
        rem = exact - counts
        rem[counts >= cin] = -1.0
        order = np.argsort(-rem, kind="stable")
        counts[order[:short]] += 1
    return counts


def _beta_mask(rng, rows: int, cin: int, density: float):
    counts = _beta_counts(rng, rows, cin, density)
    cols = [np.sort(rng.choice(cin, size=int(k), replace=False)) for k in counts]
    row_ptr = np.zeros(rows + 1, dtype=np.int64)
    np.cumsum(counts, out=row_ptr[1:])
    col = np.concatenate(cols).astype(np.int32) if len(cols) else np.zeros(0, np.int32)
    return row_ptr.astype(np.int32), col


def make_layer(
    cin: int,
    cout: int,
    h: int,
    w: int,
    n: int,
    sparsity: float,
    block_rows: int = 1,
    pattern: str = "uniform",
    storage: str = "f32",
    act: str = "relu",
    seed: int = 0,
    with_x: bool = True,
    block_cols: int = 1,
) -> Layer:
    """One seeded layer (recipe in the module docstring).  block_cols > 1
    draws the mask over aligned blocks of block_cols input channels (the
    uniform pattern only); block_cols = 1 gives exactly the draws of the
    unblocked recipe."""
    if cout % block_rows or cin % block_cols:
        raise ValueError("cout must be a multiple of block_rows and cin of block_cols")
    if act not in ACTS or storage not in STORAGES:
        raise ValueError("bad act/storage")
    rng = np.random.Generator(np.random.PCG64(seed))
    rows = cout // block_rows
    density = 1.0 - sparsity
    if pattern == "uniform":
        row_ptr, col_idx = _uniform_mask(rng, rows, cin // block_cols, density)
        col_idx = (col_idx * block_cols).astype(np.int32)
    elif pattern == "beta":
        if block_rows != 1 or block_cols != 1:
            raise ValueError("beta row densities are defined for unstructured masks")
        row_ptr, col_idx = _beta_mask(rng, rows, cin, density)
    else:
        raise ValueError(pattern)
    nnzb = int(row_ptr[-1])
    std_w = np.sqrt(2.0 / (0.1 * cin))
    values = (rng.standard_normal(nnzb * block_rows * block_cols) * std_w).astype(np.float32)
    if storage == "f16":
        values = values.astype(np.float16).astype(np.float32)
    bias = (rng.standard_normal(cout) * 0.1).astype(np.float32)
    x = None
    if with_x:
        x = np.maximum(rng.standard_normal((n, cin, h, w), dtype=np.float32), np.float32(0))
        if storage == "f16":
            x = x.astype(np.float16)
    return Layer(cin, cout, h, w, n, block_rows, sparsity, pattern, storage, act, seed,
                 row_ptr, col_idx, values, bias, x, block_cols)


def densify(cout: int, cin: int, block_rows: int, row_ptr, col_idx, values) -> np.ndarray:
    """Scatter a CSR/BCSR weight into a dense float64 [Cout, Cin] matrix."""
    k = block_rows
    wd = np.zeros((cout, cin), dtype=np.float64)
    rows = cout // k
    for rb in range(rows):
        for t in range(int(row_ptr[rb]), int(row_ptr[rb + 1])):
            c = int(col_idx[t])
            for i in range(k):
                wd[rb * k + i, c] = float(values[t * k + i])
    return wd


def expand_blocks_to_csr(cout: int, block_rows: int, row_ptr, col_idx, values):
    """Rewrite a 1xk BCSR weight as plain CSR over Cout rows (same column order)."""
    k = block_rows
    rows = cout // k
    rp = [0]
    cols, vals = [], []
    for rb in range(rows):
        s, e = int(row_ptr[rb]), int(row_ptr[rb + 1])
        for i in range(k):
            for t in range(s, e):
                cols.append(int(col_idx[t]))
                vals.append(values[t * k + i])
            rp.append(len(cols))
    return (np.asarray(rp, dtype=np.int32), np.asarray(cols, dtype=np.int32),
            np.asarray(vals, dtype=np.float32))


def make_depthwise(cin: int, seed: int):
    """Seeded depthwise 3x3 weights [cin, 3, 3] and biases [cin] for the stage
    that precedes a 1x1 in a MobileNet block (Sec. 2): taps ~ N(0, variance
    2 / 9) (fan-in 9), bias ~ N(0, variance 0.01), from
    ``numpy.random.Generator(PCG64(seed))``."""
    rng = np.random.Generator(np.random.PCG64(seed))
    k = (rng.standard_normal((cin, 3, 3)) * np.sqrt(2.0 / 9.0)).astype(np.float32)
    b = (rng.standard_normal(cin) * 0.1).astype(np.float32)
    return k, b
