"""Seeded synthetic workloads for the quaternion convolution + IQBN path.

The five layer configurations the library is measured and tested on: a tiny
fp32 layer, and CIFAR-, ImageNet-stage-, detection-backbone- and
deep-stage-shaped bf16 layers (the shapes of the quaternion Wide-ResNet and
YOLO11n networks of Section IV).  Synthetic N(0, 1) activations stand in for
the paper's image datasets (CIFAR-10/100, the ImageNet subset, COCO, DOTA),
which are not used.

This module only draws numbers.  It computes no part of the convolution or of
the normalisation, so both the GPU path and the CPU oracle can take their
inputs from it.

Conventions: ``N(0, v)`` below means variance v; every draw is float32 from
``numpy.random.default_rng(seed)`` (PCG64), in the order x, then for each layer
W_r, W_i, W_j, W_k, bias, gamma, beta.  bf16 workloads round the float32 draws
to bfloat16 with round-to-nearest-even (torch's conversion).
"""
from dataclasses import dataclass, field
from typing import List, Optional, Tuple

import numpy as np
import torch


@dataclass(frozen=True)
class ConvLayer:
    c_in: int                 # quaternion input channels
    c_out: int                # quaternion output channels
    k: int                    # square kernel size
    stride: int = 1
    pad: int = 0
    dilation: int = 1
    w_var: float = 1.0        # weights ~ N(0, w_var)
    bias: str = "none"        # "none" | "zero" | "normal" (N(0, bias_var))
    bias_var: float = 0.0
    gamma: str = "one"        # "one" | "uniform" (U(0.5, 1.5))
    beta: str = "zero"        # "zero" | "normal" (N(0, beta_var))
    beta_var: float = 0.0
    relu: bool = False        # ReLU after IQBN

    def out_hw(self, h: int, w: int) -> Tuple[int, int]:
        span = self.dilation * (self.k - 1) + 1
        return ((h + 2 * self.pad - span) // self.stride + 1,
                (w + 2 * self.pad - span) // self.stride + 1)


@dataclass(frozen=True)
class Workload:
    name: str
    description: str
    dtype: str                # "fp32" | "bf16"
    n: int
    h: int
    w: int
    layers: Tuple[ConvLayer, ...]
    seed: int
    eps: float = 1e-5

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "fp32" else torch.bfloat16

    def layer_dims(self) -> List[dict]:
        """Per layer: input/output spatial sizes and the implicit-GEMM sizes."""
        h, w = self.h, self.w
        dims = []
        for L in self.layers:
            ho, wo = L.out_hw(h, w)
            m = self.n * ho * wo
            dims.append(dict(h=h, w=w, ho=ho, wo=wo, m=m, n_gemm=4 * L.c_out,
                             k_gemm=4 * L.c_in * L.k * L.k,
                             useful_flops=2 * m * 4 * L.c_out * 4 * L.c_in * L.k * L.k))
            h, w = ho, wo
        return dims

    def useful_flops(self) -> int:
        return sum(d["useful_flops"] for d in self.layer_dims())


def _fan(c_in: int, k: int) -> float:
    return 1.0 / (4 * c_in * k * k)


WORKLOADS = {
    "tiny_fp32": Workload(
        "tiny_fp32", "single 3x3 quaternion conv, 4->4 channels, 2x16x16, fp32, then IQBN",
        "fp32", 2, 16, 16,
        (ConvLayer(4, 4, 3, 1, 1, w_var=_fan(4, 3), bias="zero"),), seed=0),
    "cifar": Workload(
        "cifar", "CIFAR-shaped 3x3 layer, 16->16 channels, 128x32x32, bias, IQBN + ReLU",
        "bf16", 128, 32, 32,
        (ConvLayer(16, 16, 3, 1, 1, w_var=_fan(16, 3), bias="normal", bias_var=0.01,
                   gamma="uniform", beta="normal", beta_var=0.1, relu=True),), seed=1),
    "imagenet_stage": Workload(
        "imagenet_stage", "ImageNet-ResNet-stage 3x3 layer, 64->64 channels, 64x56x56, IQBN",
        "bf16", 64, 56, 56,
        (ConvLayer(64, 64, 3, 1, 1, w_var=_fan(64, 3)),), seed=2),
    "detection_pair": Workload(
        "detection_pair", "detection-backbone pair: 3x3/s2 32->64 on 16x160x160, "
        "then 1x1 64->64 on 80x80, each followed by IQBN",
        "bf16", 16, 160, 160,
        (ConvLayer(32, 64, 3, 2, 1, w_var=_fan(32, 3)),
         ConvLayer(64, 64, 1, 1, 0, w_var=_fan(64, 1))), seed=3),
    "deep_stack": Workload(
        "deep_stack", "deep-stage stack: four 3x3 256->256 layers on 32x14x14, "
        "each with IQBN + ReLU",
        "bf16", 32, 14, 14,
        tuple(ConvLayer(256, 256, 3, 1, 1, w_var=_fan(256, 3), gamma="uniform",
                        beta="normal", beta_var=0.1, relu=True) for _ in range(4)), seed=4),
}

# The order the five configurations are listed in (smallest first).
WORKLOAD_ORDER = ["tiny_fp32", "cifar", "imagenet_stage", "detection_pair", "deep_stack"]


@dataclass
class LayerTensors:
    weight: torch.Tensor              # [4, Cout, Cin, k, k] (W_r, W_i, W_j, W_k), run dtype
    bias: Optional[torch.Tensor]      # [4, Cout] run dtype, or None
    gamma: torch.Tensor               # [4, Cout] float32
    beta: torch.Tensor                # [4, Cout] float32


@dataclass
class WorkloadTensors:
    x: torch.Tensor                   # [N, 4, Cin, H, W] run dtype, logical layout, CPU
    layers: List[LayerTensors] = field(default_factory=list)


def _normal(rng, shape, var):
    return rng.standard_normal(shape, dtype=np.float32) * np.float32(np.sqrt(var))


def generate(wl: Workload, seed: Optional[int] = None, n: Optional[int] = None) -> WorkloadTensors:
    """Draw the workload's tensors on the CPU (logical layout, run dtype).

    ``n`` overrides the batch size (same per-image distributions)."""
    rng = np.random.default_rng(wl.seed if seed is None else seed)
    dt = wl.torch_dtype
    nb = wl.n if n is None else n
    x = _normal(rng, (nb, 4, wl.layers[0].c_in, wl.h, wl.w), 1.0)
    out = WorkloadTensors(torch.from_numpy(x).to(dt))
    for L in wl.layers:
        ws = [_normal(rng, (L.c_out, L.c_in, L.k, L.k), L.w_var) for _ in range(4)]
        weight = torch.from_numpy(np.stack(ws)).to(dt)
        if L.bias == "none":
            bias = None
        elif L.bias == "zero":
            bias = torch.zeros(4, L.c_out, dtype=dt)
        else:
            bias = torch.from_numpy(_normal(rng, (4, L.c_out), L.bias_var)).to(dt)
        if L.gamma == "one":
            gamma = torch.ones(4, L.c_out)
        else:
            gamma = torch.from_numpy(rng.uniform(0.5, 1.5, (4, L.c_out)).astype(np.float32))
        if L.beta == "zero":
            beta = torch.zeros(4, L.c_out)
        else:
            beta = torch.from_numpy(_normal(rng, (4, L.c_out), L.beta_var))
        out.layers.append(LayerTensors(weight, bias, gamma, beta))
    return out


def random_case(rng: np.random.Generator, shape, dtype=torch.bfloat16, scale: float = 1.0):
    """A seeded N(0, scale^2) tensor of the given shape, rounded to ``dtype``."""
    return torch.from_numpy(_normal(rng, tuple(shape), scale * scale)).to(dtype)
