"""The benchmark workloads: 1x1 layers with MobileNet/EfficientNet shapes.

Each layer is (cin, cout, h, w, n, sparsity, block_rows, pattern, storage, act).
Seeds follow seed = 1000 * config + 10 * layer + variant, so every layer of
every workload is reproducible on its own.

* mbv1_c32_56_b1   -- one 32->64 @56x56 layer, fp32, batch 1, 90%, ReLU.
* mbv1_pointwise   -- the 13 pointwise layers of MobileNet v1 (width 1.0, 224x224),
                      fp32, 90% uniform, ReLU6, batch 1 (variant 0) and 64 (variant 1).
* sweep_512_14_b256 -- Cin = Cout = 512, 14x14, batch 256, fp32, ReLU, sparsity
                      70/80/90/95%, unstructured (variant 0) and 1x4 blocked (variant 1).
                      The 90% pair is the headline workload.
* mbv2_bottleneck  -- MobileNet-v2 expand/contract pairs, fp32, batch 128, 85%,
                      Beta(1.5, 8.5) row densities; ReLU6 on expand layers, none on
                      contract (linear bottleneck) layers.
* effnet_b0_f16    -- EfficientNet-B0-sized layers, fp16 storage / fp32 accumulate,
                      batch 512, 90%, 1x4 blocked, ReLU6.
"""

from __future__ import annotations

from .layers import make_layer

_MBV1 = [
    (32, 64, 112), (64, 128, 56), (128, 128, 56), (128, 256, 28), (256, 256, 28),
    (256, 512, 14), (512, 512, 14), (512, 512, 14), (512, 512, 14), (512, 512, 14),
    (512, 512, 14), (512, 1024, 7), (1024, 1024, 7),
]
_MBV2 = [
    (24, 144, 56), (144, 24, 56), (32, 192, 28), (192, 32, 28), (96, 576, 14),
    (576, 96, 14), (160, 960, 7), (960, 160, 7), (320, 1280, 7),
]
_EN = [(40, 240, 28), (80, 480, 14), (112, 672, 14), (192, 1152, 7), (320, 1280, 7)]


def _c0():
    return [dict(name="32->64@56 b1", cin=32, cout=64, h=56, w=56, n=1, sparsity=0.9,
                 block_rows=1, pattern="uniform", storage="f32", act="relu", layer=0, variant=0)]


def _c1():
    out = []
    for vi, n in enumerate((1, 64)):
        for li, (ci, co, s) in enumerate(_MBV1):
            out.append(dict(name=f"L{li + 1} {ci}->{co}@{s} b{n}", cin=ci, cout=co, h=s, w=s, n=n,
                            sparsity=0.9, block_rows=1, pattern="uniform", storage="f32",
                            act="relu6", layer=li, variant=vi))
    return out


def _c2():
    out = []
    for li, s in enumerate((0.7, 0.8, 0.9, 0.95)):
        for vi, k in enumerate((1, 4)):
            out.append(dict(name=f"512->512@14 b256 {int(round(s * 100))}% 1x{k}", cin=512, cout=512,
                            h=14, w=14, n=256, sparsity=s, block_rows=k, pattern="uniform",
                            storage="f32", act="relu", layer=li, variant=vi))
    return out


def _c3():
    out = []
    for li, (ci, co, s) in enumerate(_MBV2):
        out.append(dict(name=f"{ci}->{co}@{s} b128", cin=ci, cout=co, h=s, w=s, n=128, sparsity=0.85,
                        block_rows=1, pattern="beta", storage="f32",
                        act="relu6" if co > ci else "none", layer=li, variant=0))
    return out


def _c4():
    out = []
    for li, (ci, co, s) in enumerate(_EN):
        out.append(dict(name=f"{ci}->{co}@{s} b512 f16", cin=ci, cout=co, h=s, w=s, n=512, sparsity=0.9,
                        block_rows=4, pattern="uniform", storage="f16", act="relu6", layer=li,
                        variant=0))
    return out


CONFIGS = {
    0: ("mbv1_c32_56_b1", _c0),
    1: ("mbv1_pointwise", _c1),
    2: ("sweep_512_14_b256", _c2),
    3: ("mbv2_bottleneck", _c3),
    4: ("effnet_b0_f16", _c4),
}

# The headline layer: 512->512, 14x14, batch 256, 90% sparse (both variants).
TARGET = dict(config=2, layer=2)


def layer_seed(config: int, layer: int, variant: int) -> int:
    return 1000 * config + 10 * layer + variant


def config_layers(config: int):
    """Layer specs (dicts) of one workload."""
    return CONFIGS[config][1]()


def build(config: int, spec: dict, n=None, with_x=True):
    """Draw one layer of a workload (optionally at another batch size)."""
    return make_layer(spec["cin"], spec["cout"], spec["h"], spec["w"],
                      spec["n"] if n is None else n, spec["sparsity"],
                      block_rows=spec["block_rows"], pattern=spec["pattern"],
                      storage=spec["storage"], act=spec["act"],
                      seed=layer_seed(config, spec["layer"], spec["variant"]), with_x=with_x)
