"""Conversion of torch.nn layers into the parameter layouts of the C ABI.

Done once, when a model's weights are loaded; nothing here runs per call.

Layouts (include/convfirst.h):
  depth-wise taps   nn.Conv2d(C, C, k, groups=C).weight [C, 1, k, k] -> [k, k, C]
  grouped taps      nn.Conv2d(C, C, k, groups=C/gw).weight [C, gw, k, k] -> [k, k, C, gw]
  point-wise        nn.Conv2d(Cin, Cout, 1).weight [Cout, Cin, 1, 1] -> [Cout, Cin]
                    (nn.Linear.weight [Cout, Cin] is already in that layout)
  2x2 stride 2      nn.Conv2d(Cin, Cout, 2, stride=2).weight [Cout, Cin, 2, 2] -> [Cout, 2, 2, Cin]

Batch norm in inference mode is an affine map per channel, so it folds into a
scale and a bias after the preceding convolution (the folding of the last
paragraph of Sec. 5.3.1 of Lavin, arXiv:2404.03617):
  BN(conv(x) + cb) = s * conv(x) + (s * (cb - mean) + beta),  s = gamma / sqrt(var + eps).
The ABI takes s and the bias as separate fp32 vectors and applies them to the
fp32 accumulator, so the weights themselves are not rescaled.
"""
from __future__ import annotations

import torch

__all__ = ["dw_weight_from_conv2d", "grouped_weight_from_conv2d", "pw_weight_from_conv2d",
           "down_weight_from_conv2d", "fold_batchnorm", "block_params_from_modules",
           "grouped_block_params_from_modules", "down_params_from_modules"]


def _weight(m):
    return m.weight.detach() if isinstance(m, torch.nn.Module) else m.detach()


def dw_weight_from_conv2d(w, dtype=None) -> torch.Tensor:
    """[C, 1, k, k] (a depth-wise nn.Conv2d or its weight) -> [k, k, C]."""
    w = _weight(w)
    if w.dim() != 4 or w.shape[1] != 1 or w.shape[2] != w.shape[3]:
        raise ValueError("depth-wise weight must be [C, 1, k, k], got %s" % tuple(w.shape))
    out = w[:, 0].permute(1, 2, 0).contiguous()
    return out if dtype is None else out.to(dtype).contiguous()


def grouped_weight_from_conv2d(w, dtype=None) -> torch.Tensor:
    """[C, gw, k, k] (a grouped nn.Conv2d with C in and out channels, group
    width gw) -> [k, k, C, gw]."""
    w = _weight(w)
    if w.dim() != 4 or w.shape[2] != w.shape[3]:
        raise ValueError("grouped weight must be [C, gw, k, k], got %s" % tuple(w.shape))
    out = w.permute(2, 3, 0, 1).contiguous()
    return out if dtype is None else out.to(dtype).contiguous()


def pw_weight_from_conv2d(w, dtype=None) -> torch.Tensor:
    """[Cout, Cin, 1, 1] (a 1x1 nn.Conv2d) or [Cout, Cin] (nn.Linear) -> [Cout, Cin]."""
    w = _weight(w)
    if w.dim() == 4:
        if w.shape[2:] != (1, 1):
            raise ValueError("point-wise weight must be [Cout, Cin, 1, 1], got %s" % tuple(w.shape))
        w = w[:, :, 0, 0]
    if w.dim() != 2:
        raise ValueError("point-wise weight must be [Cout, Cin], got %s" % tuple(w.shape))
    out = w.contiguous()
    return out if dtype is None else out.to(dtype).contiguous()


def down_weight_from_conv2d(w, dtype=None) -> torch.Tensor:
    """[Cout, Cin, 2, 2] (a 2x2 stride-2 nn.Conv2d) -> [Cout, 2, 2, Cin]."""
    w = _weight(w)
    if w.dim() != 4 or tuple(w.shape[2:]) != (2, 2):
        raise ValueError("down-sampling weight must be [Cout, Cin, 2, 2], got %s" % tuple(w.shape))
    out = w.permute(0, 2, 3, 1).contiguous()
    return out if dtype is None else out.to(dtype).contiguous()


def fold_batchnorm(bn, conv_bias=None, channels: int | None = None):
    """(scale, bias) as fp32 vectors for `s * conv(x) + bias`.

    bn: an inference-mode nn.BatchNorm2d or None.  conv_bias: the preceding
    convolution's bias or None.  With neither, returns (None, None): the ABI
    reads NULL as scale 1 and bias 0."""
    cb = None if conv_bias is None else conv_bias.detach().to(torch.float64)
    if bn is None:
        return None, (None if cb is None else cb.to(torch.float32).contiguous())
    if bn.training:
        raise ValueError("batch norm must be in inference mode (call .eval()) to be folded")
    if not bn.track_running_stats or bn.running_mean is None:
        raise ValueError("batch norm without running statistics cannot be folded")
    mean = bn.running_mean.detach().to(torch.float64)
    var = bn.running_var.detach().to(torch.float64)
    gamma = bn.weight.detach().to(torch.float64) if bn.affine else torch.ones_like(mean)
    beta = bn.bias.detach().to(torch.float64) if bn.affine else torch.zeros_like(mean)
    s = gamma / torch.sqrt(var + bn.eps)
    b = beta - s * mean if cb is None else beta + s * (cb - mean)
    if channels is not None and s.numel() != channels:
        raise ValueError("batch norm has %d channels, expected %d" % (s.numel(), channels))
    return s.to(torch.float32).contiguous(), b.to(torch.float32).contiguous()


def _pair(conv, bn, channels):
    return fold_batchnorm(bn, getattr(conv, "bias", None), channels)


def block_params_from_modules(dw: torch.nn.Conv2d, bn0, pw1, bn1, pw2, bn2, dtype=torch.float16) -> dict:
    """Parameters of cf_block_forward from the block's torch layers: depth-wise
    conv -> BN -> 1x1 expand -> BN -> phi -> 1x1 project -> BN, plus the
    residual.  pw1/pw2 may be 1x1 nn.Conv2d or nn.Linear."""
    C = dw.weight.shape[0]
    if dw.groups != C or dw.stride not in ((1, 1), 1) or dw.weight.shape[2] % 2 == 0:
        raise ValueError("dw must be a stride-1 depth-wise conv with an odd kernel")
    if dw.padding not in ((dw.weight.shape[2] // 2,) * 2, dw.weight.shape[2] // 2):
        raise ValueError("dw must use 'same' zero padding k // 2")
    EC = pw1.weight.shape[0]
    p = {"dw_w": dw_weight_from_conv2d(dw, dtype), "w1": pw_weight_from_conv2d(pw1, dtype),
         "w2": pw_weight_from_conv2d(pw2, dtype)}
    p["s0"], p["b0"] = _pair(dw, bn0, C)
    p["s1"], p["b1"] = _pair(pw1, bn1, EC)
    p["s2"], p["b2"] = _pair(pw2, bn2, C)
    return p


def grouped_block_params_from_modules(conv: torch.nn.Conv2d, bn0, pw1, bn1, pw2, bn2,
                                      dtype=torch.float16) -> dict:
    """Parameters of cf_gblock_forward: as block_params_from_modules, with a
    grouped conv (C in and out channels, group width C / conv.groups) first."""
    C = conv.weight.shape[0]
    if conv.in_channels != C or conv.stride not in ((1, 1), 1) or conv.weight.shape[2] % 2 == 0:
        raise ValueError("conv must be a stride-1 C -> C grouped conv with an odd kernel")
    if conv.padding not in ((conv.weight.shape[2] // 2,) * 2, conv.weight.shape[2] // 2):
        raise ValueError("conv must use 'same' zero padding k // 2")
    EC = pw1.weight.shape[0]
    p = {"gw_w": grouped_weight_from_conv2d(conv, dtype), "w1": pw_weight_from_conv2d(pw1, dtype),
         "w2": pw_weight_from_conv2d(pw2, dtype)}
    p["s0"], p["b0"] = _pair(conv, bn0, C)
    p["s1"], p["b1"] = _pair(pw1, bn1, EC)
    p["s2"], p["b2"] = _pair(pw2, bn2, C)
    return p


def stem_params_from_modules(conv: torch.nn.Conv2d, bn=None, dtype=torch.float16) -> dict:
    """Parameters of cf_stem_forward / cf_stem_gblock_forward from the stem's
    3 x 3 stride-2 conv (3 input channels, padding 1) and its BN: taps
    [C][3][3][3] (torch [C][3][3][3] permuted (0, 2, 3, 1)), folded scale and bias."""
    if (tuple(conv.weight.shape[1:]) != (3, 3, 3) or conv.stride not in ((2, 2), 2) or conv.groups != 1
            or conv.padding not in ((1, 1), 1)):
        raise ValueError("conv must be a 3x3 stride-2 conv from 3 channels with padding 1")
    p = {"sw": conv.weight.detach().permute(0, 2, 3, 1).contiguous().to(dtype)}
    p["ss"], p["sb"] = _pair(conv, bn, conv.weight.shape[0])
    return p


def down_params_from_modules(conv: torch.nn.Conv2d, bn=None, dtype=torch.float16) -> dict:
    """Parameters of cf_downsample_forward from a 2x2 stride-2 conv and its BN."""
    if tuple(conv.weight.shape[2:]) != (2, 2) or conv.stride not in ((2, 2), 2):
        raise ValueError("conv must be a 2x2 conv with stride 2")
    p = {"wd": down_weight_from_conv2d(conv, dtype)}
    p["sd"], p["bd"] = _pair(conv, bn, conv.weight.shape[0])
    return p
