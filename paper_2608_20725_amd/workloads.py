"""Seeded synthetic convolution layers: shapes, seeds and value recipes.

This module only describes workloads and draws their values; it computes
nothing of the convolution itself, so both the GPU path's tests and the CPU
oracle can take their inputs from it.

The layer shapes of the 12-layer sweep are those of the paper's benchmark
table (Table I, layers cv1 and cv3-cv12), plus a 1x1 layer with 1024 input and
output channels; all of them run at batch 128.  Values are synthetic.

Recipe: a ``torch.Generator('cpu')`` seeded with the layer's seed draws the
NHWC input (N, H, W, C_i) first, then the filter (K_h, K_w, C_i, C_o), both in
fp32; ``uniform`` is ``rand * 2 - 1`` (uniform on [-1, 1)), ``normal`` is
``randn`` (normal(0, 1)).  The fp16 path uses ``.half()`` of the same draws.
"""
from __future__ import annotations

from dataclasses import dataclass, asdict

import torch


@dataclass(frozen=True)
class Layer:
    name: str
    N: int
    C_i: int
    H: int
    W: int
    C_o: int
    K_h: int
    K_w: int
    stride: int
    seed: int
    dist: str = "uniform"      # "uniform" on [-1, 1) or "normal" (0, 1)
    dtypes: tuple = ("f32", "f16")
    note: str = ""

    def as_dict(self):
        return asdict(self)


def _sq(name, N, Ci, HW, Co, K, s, seed, dist="uniform", dtypes=("f32", "f16"), note=""):
    return Layer(name, N, Ci, HW, HW, Co, K, K, s, seed, dist, tuple(dtypes), note)


# The four named configurations.
CFG1 = _sq("cfg1_tiny_c3_32_3x3", 1, 3, 32, 16, 3, 1, 0,
           note="single small layer, output 1x30x30x16")
CFG2 = _sq("cfg2_n128_c64_56_3x3", 128, 64, 56, 64, 3, 1, 1,
           note="ResNet-style 3x3 layer, fp32 and fp16")
CFG3 = _sq("cfg3_stem_c3_227_11x11_s4", 128, 3, 227, 96, 11, 4, 2, dist="normal",
           note="large-kernel stem, normal(0,1) values")
CFG4 = _sq("cfg4_deep_c512_14_3x3", 128, 512, 14, 512, 3, 1, 3, dtypes=("f16", "f32"),
           note="deep low-resolution layer")

# The 12-layer sweep (Table I shapes, cv2 dropped as a near-duplicate of cv1,
# plus one 1x1 layer); seeds 101..112.
SWEEP = (
    _sq("S1_cv1", 128, 3, 227, 96, 11, 4, 101),
    _sq("S2_cv3", 128, 3, 227, 64, 7, 2, 102),
    _sq("S3_cv4", 128, 64, 224, 64, 7, 2, 103),
    _sq("S4_cv5", 128, 96, 24, 256, 5, 1, 104),
    _sq("S5_cv6", 128, 256, 12, 512, 3, 1, 105),
    _sq("S6_cv7", 128, 3, 224, 64, 3, 1, 106),
    _sq("S7_cv8", 128, 64, 112, 128, 3, 1, 107),
    _sq("S8_cv9", 128, 64, 56, 64, 3, 1, 108),
    _sq("S9_cv10", 128, 128, 28, 128, 3, 1, 109),
    _sq("S10_cv11", 128, 256, 14, 256, 3, 1, 110),
    _sq("S11_cv12", 128, 512, 7, 512, 3, 1, 111),
    _sq("S12_1x1", 128, 1024, 14, 1024, 1, 1, 112),
)

CONFIGS = (CFG1, CFG2, CFG3, CFG4)
ALL = CONFIGS + SWEEP
BY_NAME = {l.name: l for l in ALL}


def draw(N, C_i, H, W, C_o, K_h, K_w, seed, dist="uniform"):
    """Draw (input NHWC, filter KhKwCiCo) as fp32 CPU tensors from ``seed``."""
    g = torch.Generator("cpu").manual_seed(int(seed))
    if dist == "uniform":
        x = torch.rand((N, H, W, C_i), generator=g, dtype=torch.float32) * 2 - 1
        w = torch.rand((K_h, K_w, C_i, C_o), generator=g, dtype=torch.float32) * 2 - 1
    elif dist == "normal":
        x = torch.randn((N, H, W, C_i), generator=g, dtype=torch.float32)
        w = torch.randn((K_h, K_w, C_i, C_o), generator=g, dtype=torch.float32)
    elif dist == "int2":
        # integers in {-2..2}: every product and partial sum is exact in fp16
        # operands with fp32 accumulation, so any summation order agrees
        x = torch.randint(-2, 3, (N, H, W, C_i), generator=g).to(torch.float32)
        w = torch.randint(-2, 3, (K_h, K_w, C_i, C_o), generator=g).to(torch.float32)
    else:
        raise ValueError("unknown distribution %r" % dist)
    return x, w


def draw_layer(layer: Layer, N: int | None = None):
    """Inputs of ``layer`` (optionally with a smaller batch, same recipe)."""
    return draw(layer.N if N is None else N, layer.C_i, layer.H, layer.W, layer.C_o,
                layer.K_h, layer.K_w, layer.seed, layer.dist)
