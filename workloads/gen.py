"""Seeded generators for weights and activations (no arithmetic of the method)."""
import math

import torch

from .configs import ConvLayer

_DT = {"f32": torch.float32, "bf16": torch.bfloat16}


def gen_weight(gen: torch.Generator, cout: int, cin: int, k: int) -> torch.Tensor:
    """He-normal (fan-in) float32 weight [cout][cin][k][k]."""
    std = math.sqrt(2.0 / (cin * k * k))
    return torch.randn((cout, cin, k, k), generator=gen, dtype=torch.float32) * std


def gen_activation(gen: torch.Generator, shape, act: str = "relu") -> torch.Tensor:
    """ReLU(N(0,1)) or ReLU6(N(0,1)) float32 activations."""
    x = torch.randn(shape, generator=gen, dtype=torch.float32)
    return x.clamp(0.0, 6.0) if act == "relu6" else x.clamp_min(0.0)


def gen_layer(layer: ConvLayer, batch: int, dtype: str = "f32", layout: str = "nchw"):
    """(W, X) for one layer: W drawn first, then X, from the layer's seed.

    Returns CPU tensors of the requested dtype; X is NCHW, or NHWC when asked."""
    gen = torch.Generator("cpu").manual_seed(layer.seed)
    w = gen_weight(gen, layer.cout, layer.cin, layer.k)
    x = gen_activation(gen, (batch, layer.cin, layer.H, layer.H), layer.act)
    w, x = w.to(_DT[dtype]), x.to(_DT[dtype])
    if layout == "nhwc":
        x = x.permute(0, 2, 3, 1).contiguous()
    return w, x


def gen_integer_layer(seed: int, cout: int, cin: int, k: int, batch: int, H: int, W: int = None,
                      wmax: int = 3, xmax: int = 3):
    """Small-integer-valued W in [-wmax, wmax] and X in [0, xmax] (float32).

    With these, every partial sum of a convolution is an integer far below
    2^24, so any summation order gives the exact result in fp32."""
    W = H if W is None else W
    gen = torch.Generator("cpu").manual_seed(seed)
    w = torch.randint(-wmax, wmax + 1, (cout, cin, k, k), generator=gen).to(torch.float32)
    x = torch.randint(0, xmax + 1, (batch, cin, H, W), generator=gen).to(torch.float32)
    return w, x
