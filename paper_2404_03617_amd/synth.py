"""Seeded synthetic inputs for the ConvFirst block and its stacks.

This module only draws random numbers and rounds them to the I/O dtypes; it
holds none of the block's arithmetic.  The GPU path and the CPU checker both
consume the tensors it returns (the checker after an exact widening to
float64), so both see bit-identical inputs.

Distributions (per tensor, drawn in float64 from
``numpy.random.default_rng(SeedSequence([seed, tensor_id]))``):
  x            ~ N(0, 1)
  weights      ~ N(0, 1/fan_in), fan_in = k*k (depth-wise), C (expand),
                 E*C (project), 4*Cin (2x2 down-sampling)
  biases       ~ N(0, bias_std^2), bias_std = 0.1 by default (variance 0.01)
  scales       = 1 ("ones") or ~ U(0.5, 1.5) ("uniform")
Activations and weights are rounded to fp16/bf16 with round-to-nearest-even;
scales and biases stay fp32.

Layouts (what the C ABI takes):
  x            [N, H, W, C]
  dw_w         [k, k, C]
  w1           [E*C, C]        w2 [C, E*C]
  wd           [Cout, 2, 2, Cin]
"""
from __future__ import annotations

import numpy as np
import torch

DTYPES = {"f16": torch.float16, "bf16": torch.bfloat16}


def draw(seed: int, tensor_id: int, shape, std: float = 1.0) -> np.ndarray:
    rng = np.random.default_rng(np.random.SeedSequence([int(seed), int(tensor_id)]))
    return rng.standard_normal(tuple(shape)) * std


def draw_uniform(seed: int, tensor_id: int, shape, lo: float, hi: float) -> np.ndarray:
    rng = np.random.default_rng(np.random.SeedSequence([int(seed), int(tensor_id)]))
    return rng.uniform(lo, hi, tuple(shape))


def to_io(a: np.ndarray, dtype: str) -> torch.Tensor:
    """float64 -> fp16/bf16 (round to nearest even), contiguous CPU tensor."""
    return torch.from_numpy(np.ascontiguousarray(a)).to(DTYPES[dtype]).contiguous()


def to_f32(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a)).to(torch.float32).contiguous()


def activations(seed: int, N: int, H: int, W: int, C: int, dtype: str = "f16",
                tensor_id: int = 0, std: float = 1.0) -> torch.Tensor:
    return to_io(draw(seed, tensor_id, (N, H, W, C), std), dtype)


def _vec(seed, tid, n, kind, bias_std, scales):
    if kind == "scale":
        if scales == "ones":
            return to_f32(np.ones(n))
        if scales == "uniform":
            return to_f32(draw_uniform(seed, tid, (n,), 0.5, 1.5))
        if scales == "none":
            return None
        raise ValueError(scales)
    if bias_std is None:
        return None
    return to_f32(draw(seed, tid, (n,), bias_std))


def block_params(seed: int, layer: int, C: int, E: int, k: int, dtype: str = "f16",
                 scales: str = "ones", bias_std: float | None = 0.1) -> dict:
    """Weights of one block; tensor ids 100*(layer+1) + 0..8."""
    base = 100 * (layer + 1)
    EC = E * C
    p = {
        "dw_w": to_io(draw(seed, base + 0, (k, k, C), (1.0 / (k * k)) ** 0.5), dtype),
        "s0": _vec(seed, base + 1, C, "scale", bias_std, scales),
        "b0": _vec(seed, base + 2, C, "bias", bias_std, scales),
        "w1": to_io(draw(seed, base + 3, (EC, C), (1.0 / C) ** 0.5), dtype),
        "s1": _vec(seed, base + 4, EC, "scale", bias_std, scales),
        "b1": _vec(seed, base + 5, EC, "bias", bias_std, scales),
        "w2": to_io(draw(seed, base + 6, (C, EC), (1.0 / EC) ** 0.5), dtype),
        "s2": _vec(seed, base + 7, C, "scale", bias_std, scales),
        "b2": _vec(seed, base + 8, C, "bias", bias_std, scales),
    }
    return p


def gblock_params(seed: int, layer: int, C: int, E: int, k: int = 3, dtype: str = "f16",
                  scales: str = "ones", bias_std: float | None = 0.1, gw: int = 8) -> dict:
    """Weights of one block of the paper's own form (grouped conv of group
    width gw first); tensor ids 100*(layer+1) + 0..8, the grouped taps
    [k, k, C, gw] ~ N(0, 1/(k*k*gw)) in place of the depth-wise ones."""
    p = block_params(seed, layer, C, E, k, dtype, scales, bias_std)
    del p["dw_w"]
    p["gw_w"] = to_io(draw(seed, 100 * (layer + 1) + 0, (k, k, C, gw), (1.0 / (k * k * gw)) ** 0.5), dtype)
    return p


def stem_params(seed: int, layer: int, C: int, dtype: str = "f16", scales: str = "ones",
                bias_std: float | None = 0.1) -> dict:
    """The network stem (3x3 stride-2 conv from 3 channels): taps [C, 3, 3, 3]
    ~ N(0, 1/27) (fan-in 27), ids 100*(layer+1) + 0..2."""
    base = 100 * (layer + 1)
    return {
        "sw": to_io(draw(seed, base + 0, (C, 3, 3, 3), (1.0 / 27) ** 0.5), dtype),
        "ss": _vec(seed, base + 1, C, "scale", bias_std, scales),
        "sb": _vec(seed, base + 2, C, "bias", bias_std, scales),
    }


def mbconv_params(seed: int, layer: int, C: int, E: int, R: int, dtype: str = "f16",
                  scales: str = "ones", bias_std: float | None = 0.1, gw: int = 8, K: int | None = None) -> dict:
    """Weights of one MBConv block with Squeeze & Excitation (expand, grouped
    3x3 conv of group width gw, squeeze to R, excitation, project to K
    channels, C unless given); tensor ids 100*(layer+1) + 0..12.  Weights ~
    N(0, 1/fan_in): C (expand), 9*gw (grouped conv), E*C (squeeze, project),
    R (excitation)."""
    base = 100 * (layer + 1)
    EC = E * C
    K = C if K is None else K
    return {
        "w1": to_io(draw(seed, base + 0, (EC, C), (1.0 / C) ** 0.5), dtype),
        "s1": _vec(seed, base + 1, EC, "scale", bias_std, scales),
        "b1": _vec(seed, base + 2, EC, "bias", bias_std, scales),
        "gw_w": to_io(draw(seed, base + 3, (3, 3, EC, gw), (1.0 / (9 * gw)) ** 0.5), dtype),
        "s2": _vec(seed, base + 4, EC, "scale", bias_std, scales),
        "b2": _vec(seed, base + 5, EC, "bias", bias_std, scales),
        "wr": to_io(draw(seed, base + 6, (R, EC), (1.0 / EC) ** 0.5), dtype),
        "br": _vec(seed, base + 7, R, "bias", bias_std, scales),
        "we": to_io(draw(seed, base + 8, (EC, R), (1.0 / R) ** 0.5), dtype),
        "be": _vec(seed, base + 9, EC, "bias", bias_std, scales),
        "w2": to_io(draw(seed, base + 10, (K, EC), (1.0 / EC) ** 0.5), dtype),
        "s3": _vec(seed, base + 11, K, "scale", bias_std, scales),
        "b3": _vec(seed, base + 12, K, "bias", bias_std, scales),
    }


def convfirst_s2_params(seed: int, layer: int, C: int, R: int, K: int, dtype: str = "f16",
                        scales: str = "ones", bias_std: float | None = 0.1, gw: int = 8) -> dict:
    """Weights of one stride-2 ConvFirst block (grouped 3x3 conv of group
    width gw, expand from the 2C concatenated channels to R, project to K);
    tensor ids 100*(layer+1) + 0..8.  Weights ~ N(0, 1/fan_in): 9*gw (conv),
    2C (expand), R (project)."""
    base = 100 * (layer + 1)
    return {
        "gw_w": to_io(draw(seed, base + 0, (3, 3, C, gw), (1.0 / (9 * gw)) ** 0.5), dtype),
        "s0": _vec(seed, base + 1, C, "scale", bias_std, scales),
        "b0": _vec(seed, base + 2, C, "bias", bias_std, scales),
        "w1": to_io(draw(seed, base + 3, (R, 2 * C), (1.0 / (2 * C)) ** 0.5), dtype),
        "s1": _vec(seed, base + 4, R, "scale", bias_std, scales),
        "b1": _vec(seed, base + 5, R, "bias", bias_std, scales),
        "w2": to_io(draw(seed, base + 6, (K, R), (1.0 / R) ** 0.5), dtype),
        "s2": _vec(seed, base + 7, K, "scale", bias_std, scales),
        "b2": _vec(seed, base + 8, K, "bias", bias_std, scales),
    }


def down_params(seed: int, layer: int, Cin: int, Cout: int, dtype: str = "f16",
                scales: str = "ones", bias_std: float | None = 0.1) -> dict:
    """Weights of one 2x2 stride-2 down-sampling layer; ids 100*(layer+1) + 0..2."""
    base = 100 * (layer + 1)
    return {
        "wd": to_io(draw(seed, base + 0, (Cout, 2, 2, Cin), (1.0 / (4 * Cin)) ** 0.5), dtype),
        "sd": _vec(seed, base + 1, Cout, "scale", bias_std, scales),
        "bd": _vec(seed, base + 2, Cout, "bias", bias_std, scales),
    }


def stack_layers(seed: int, depths, widths, E: int, k: int, dtype: str = "f16",
                 scales: str = "ones", bias_std: float | None = 0.1) -> list:
    """Stages of blocks with a down-sampling layer between consecutive stages.
    Returns [("block", params) | ("down", params), ...] in execution order."""
    layers = []
    li = 0
    for s, (d, c) in enumerate(zip(depths, widths)):
        if s > 0:
            layers.append(("down", down_params(seed, li, widths[s - 1], c, dtype, scales, bias_std)))
            li += 1
        for _ in range(d):
            layers.append(("block", block_params(seed, li, c, E, k, dtype, scales, bias_std)))
            li += 1
    return layers


def to_f64(t):
    """Exact widening for the checker (None passes through)."""
    if t is None:
        return None
    return t.detach().to("cpu").to(torch.float64).numpy()


def params_f64(p: dict) -> dict:
    return {k: to_f64(v) for k, v in p.items()}
