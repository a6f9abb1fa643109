"""Seeded synthetic MobileNet v1 weights and images (no trained model is used).

Architecture (width 1.0, 224 x 224 input; the network of the paper's Table 1):
a dense 3x3 stride-2 convolution 3 -> 32 on the HWC image, then 13 blocks of
depthwise 3x3 (stride 1 or 2) -> pointwise 1x1, then global average pooling
and a dense fully connected classifier.  The paper keeps the first
convolution and the classifier dense and makes every 1x1 sparse (90% for
its sparse MobileNet v1; Sec. 3.1, Table 1).

Value recipe, all from one ``numpy.random.Generator(PCG64(seed))`` per
tensor group (seed + 1 for the stem, seed + 10 + b for block b, seed + 100
for the classifier):

* stem taps ~ N(0, 2 / 27), bias ~ N(0, 0.01);
* depthwise taps ~ N(0, 2 / 9), bias ~ N(0, 0.01) (``make_depthwise``);
* pointwise 1x1: ``make_layer`` masks and values (uniform mask, exact count,
  W ~ N(0, 2 / (0.1 Cin)), bias ~ N(0, 0.01)), so the variance of each
  activation stays of order one through the 13 blocks (He-style scaling for
  the ReLU6 between layers);
* classifier W ~ N(0, 1 / 1024), bias ~ N(0, 0.01);
* the image: uniform in [-1, 1], HWC.
This module draws numbers only; it holds none of the network's arithmetic.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

from .layers import Layer, make_layer, make_depthwise

# (cin, cout, depthwise stride) of the 13 blocks at width 1.0
MBV1_BLOCKS = [
    (32, 64, 1), (64, 128, 2), (128, 128, 1), (128, 256, 2), (256, 256, 1), (256, 512, 2),
    (512, 512, 1), (512, 512, 1), (512, 512, 1), (512, 512, 1), (512, 512, 1),
    (512, 1024, 2), (1024, 1024, 1),
]


@dataclass
class Block:
    cin: int
    cout: int
    stride: int
    dw_k: np.ndarray = field(repr=False)   # [cin, 3, 3]
    dw_b: np.ndarray = field(repr=False)   # [cin]
    pw: Layer = field(repr=False)          # the sparse 1x1 (row_ptr, col_idx, values, bias, block_rows)


@dataclass
class MobileNetV1:
    stem_w: np.ndarray = field(repr=False)  # [32, 3, 3, 3]: [cout][dy][dx][cin]
    stem_b: np.ndarray = field(repr=False)  # [32]
    blocks: List[Block] = field(repr=False)
    fc_w: np.ndarray = field(repr=False)    # [classes, 1024], dense
    fc_b: np.ndarray = field(repr=False)    # [classes]
    sparsity: float = 0.9
    seed: int = 0

    @property
    def classes(self) -> int:
        return int(self.fc_w.shape[0])


def make_mobilenet_v1(seed: int = 0, sparsity: float = 0.9, classes: int = 1000,
                      block_rows: Optional[dict] = None, blocks=MBV1_BLOCKS) -> MobileNetV1:
    """Synthetic weights; ``block_rows`` maps a block index (0-based) to the
    1xk output-block height of its pointwise layer (default 1: unstructured)."""
    block_rows = block_rows or {}
    rng = np.random.Generator(np.random.PCG64(seed + 1))
    c0 = blocks[0][0]
    stem_w = (rng.standard_normal((c0, 3, 3, 3)) * np.sqrt(2.0 / 27.0)).astype(np.float32)
    stem_b = (rng.standard_normal(c0) * 0.1).astype(np.float32)
    out = []
    for b, (cin, cout, stride) in enumerate(blocks):
        kw, kb = make_depthwise(cin, seed + 10 + b)
        pw = make_layer(cin, cout, 1, 1, 1, sparsity, block_rows=block_rows.get(b, 1), act="relu6",
                        seed=seed + 10 + b, with_x=False)
        out.append(Block(cin, cout, stride, kw, kb, pw))
    rng = np.random.Generator(np.random.PCG64(seed + 100))
    cl = blocks[-1][1]
    fc_w = (rng.standard_normal((classes, cl)) * np.sqrt(1.0 / cl)).astype(np.float32)
    fc_b = (rng.standard_normal(classes) * 0.1).astype(np.float32)
    return MobileNetV1(stem_w, stem_b, out, fc_w, fc_b, sparsity, seed)


def make_image(n: int, h: int = 224, w: int = 224, seed: int = 0) -> np.ndarray:
    """A batch of HWC images, uniform in [-1, 1], float32 [n, h, w, 3]."""
    rng = np.random.Generator(np.random.PCG64(seed + 7))
    return rng.uniform(-1.0, 1.0, size=(n, h, w, 3)).astype(np.float32)
