"""The Python binding on a host without a GPU.

1. Argument checks: every tensor's shape, dtype, layout and device is checked
   before any pointer reaches the library, so a wrong argument raises
   ValueError here instead of handing the kernel a host or undersized buffer.
   The library is replaced by a stub that fails the test if it is touched.
2. Conversion of torch layers (nn.Conv2d, nn.Linear, inference-mode
   BatchNorm2d) into the ABI layouts: the oracle evaluated on the converted
   parameters equals the torch modules evaluated in float64.
"""
import numpy as np
import pytest
import torch
import torch.nn as nn
import torch.nn.functional as F

import oracle
import paper_2404_03617_amd as cf
from paper_2404_03617_amd import synth


@pytest.fixture
def no_library(monkeypatch):
    def boom():
        raise AssertionError("the library was called before the arguments were checked")
    monkeypatch.setattr(cf, "lib", boom)


def block(C=64, E=4, k=3, dtype="f16"):
    x = synth.activations(1, 2, 5, 6, C, dtype)
    p = synth.block_params(1, 0, C, E, k, dtype, scales="uniform", bias_std=0.1)
    return x, p


@pytest.mark.parametrize("key,bad", [
    ("dw_w", lambda p: p["dw_w"][:, :, :32].contiguous()),          # wrong C
    ("w1", lambda p: p["w1"][:128].contiguous()),                    # E*C rows inconsistent with w2
    ("w2", lambda p: p["w2"][:, :128].contiguous()),                 # too few hidden columns
    ("w2", lambda p: p["w2"].t().contiguous()),                      # transposed
    ("s1", lambda p: p["s1"][:64].contiguous()),                     # scale of the wrong length
    ("b0", lambda p: p["b0"].to(torch.float64)),                     # vectors must be fp32
    ("w1", lambda p: p["w1"].to(torch.bfloat16)),                    # weights in x's dtype
    ("w2", lambda p: p["w2"].t().contiguous().t()),                  # not contiguous
    ("extra", lambda p: torch.zeros(3)),                              # unknown key
])
def test_block_parameter_checks_fire_before_the_library(no_library, key, bad):
    x, p = block()
    p[key] = bad(p)
    with pytest.raises(ValueError):
        cf.block_forward(x, p)


def test_host_tensors_are_rejected_before_the_library(no_library):
    x, p = block()
    with pytest.raises(ValueError, match="GPU"):
        cf.block_forward(x, p)
    with pytest.raises(ValueError, match="GPU"):
        cf.block_forward_unfused(x, p)
    with pytest.raises(ValueError, match="GPU"):
        cf.block_forward_split(x, p)
    with pytest.raises(ValueError, match="GPU"):
        cf.stage_forward(x, [p, p])


def test_missing_required_parameter_and_bad_activation(no_library):
    x, p = block()
    q = dict(p)
    del q["w2"]
    with pytest.raises(ValueError, match="w2"):
        cf.block_forward(x, q)
    with pytest.raises(ValueError, match="act"):
        cf.block_forward(x, p, act="silu")


def test_x_checks(no_library):
    x, p = block()
    with pytest.raises(ValueError):
        cf.block_forward(x.permute(0, 2, 1, 3), p)                   # not contiguous
    with pytest.raises(ValueError):
        cf.block_forward(x.float(), p)                               # fp32 I/O
    with pytest.raises(ValueError):
        cf.block_forward(x[0], p)                                    # rank 3


def test_stage_blocks_must_share_a_shape(no_library):
    x, p = block()
    _, q = block(E=2)
    with pytest.raises(ValueError):
        cf.stage_forward(x, [p, q])


def test_downsample_parameter_checks(no_library):
    x = synth.activations(1, 2, 6, 6, 64, "f16")
    d = synth.down_params(1, 0, 64, 128, "f16")
    bad = dict(d, wd=d["wd"][:, :, :, :32].contiguous())             # Cin mismatch
    with pytest.raises(ValueError):
        cf.downsample_forward(x, bad)
    bad = dict(d, sd=d["sd"][:64].contiguous())
    with pytest.raises(ValueError):
        cf.downsample_forward(x, bad)
    with pytest.raises(ValueError, match="GPU"):
        cf.downsample_forward(x, d)


# ---------------------------------------------------------------- conversion
def _bn(C, seed):
    g = torch.Generator().manual_seed(seed)
    bn = nn.BatchNorm2d(C).double()
    with torch.no_grad():
        bn.weight.copy_(torch.rand(C, generator=g, dtype=torch.float64) + 0.5)
        bn.bias.copy_(torch.randn(C, generator=g, dtype=torch.float64) * 0.3)
        bn.running_mean.copy_(torch.randn(C, generator=g, dtype=torch.float64) * 0.2)
        bn.running_var.copy_(torch.rand(C, generator=g, dtype=torch.float64) + 0.5)
    return bn.eval()


def _rand_conv(conv, seed):
    g = torch.Generator().manual_seed(seed)
    with torch.no_grad():
        conv.weight.copy_(torch.randn(conv.weight.shape, generator=g, dtype=torch.float64) * 0.3)
        if conv.bias is not None:
            conv.bias.copy_(torch.randn(conv.bias.shape, generator=g, dtype=torch.float64) * 0.1)
    return conv


@pytest.mark.parametrize("conv_bias", [False, True])
@pytest.mark.parametrize("linear", [False, True])
def test_block_from_torch_modules_matches_the_modules(conv_bias, linear):
    """Depth-wise conv -> BN -> expand -> BN -> GELU -> project -> BN, plus the
    residual, as torch float64 modules; the same block through the layout
    conversion and BN folding, evaluated by the oracle."""
    C, E, k = 6, 3, 5
    dw = _rand_conv(nn.Conv2d(C, C, k, padding=k // 2, groups=C, bias=conv_bias).double(), 1)
    if linear:
        pw1 = _rand_conv(nn.Linear(C, E * C, bias=conv_bias).double(), 2)
        pw2 = _rand_conv(nn.Linear(E * C, C, bias=conv_bias).double(), 3)
    else:
        pw1 = _rand_conv(nn.Conv2d(C, E * C, 1, bias=conv_bias).double(), 2)
        pw2 = _rand_conv(nn.Conv2d(E * C, C, 1, bias=conv_bias).double(), 3)
    bn0, bn1, bn2 = _bn(C, 4), _bn(E * C, 5), _bn(C, 6)
    x = torch.randn(2, C, 7, 4, dtype=torch.float64, generator=torch.Generator().manual_seed(7))

    def pw(m, t):
        if isinstance(m, nn.Linear):
            return m(t.permute(0, 2, 3, 1)).permute(0, 3, 1, 2)
        return m(t)

    with torch.no_grad():
        h = F.gelu(bn1(pw(pw1, bn0(dw(x)))))
        ref = (x + bn2(pw(pw2, h))).permute(0, 2, 3, 1).numpy()
    p = cf.block_params_from_modules(dw, bn0, pw1, bn1, pw2, bn2, dtype=torch.float64)
    got = oracle.block_forward(x.permute(0, 2, 3, 1).numpy(), {kk: (None if v is None else v.numpy())
                                                                for kk, v in p.items()})
    # the folded scale/bias vectors are fp32 (the ABI type): compare at that precision
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-5 * np.abs(ref).max())


def test_grouped_block_from_torch_modules_matches_the_modules():
    C, E, gw = 16, 3, 8
    conv = _rand_conv(nn.Conv2d(C, C, 3, padding=1, groups=C // gw, bias=True).double(), 11)
    pw1 = _rand_conv(nn.Conv2d(C, E * C, 1, bias=False).double(), 12)
    pw2 = _rand_conv(nn.Conv2d(E * C, C, 1, bias=False).double(), 13)
    bn0, bn1, bn2 = _bn(C, 14), _bn(E * C, 15), _bn(C, 16)
    x = torch.randn(2, C, 5, 6, dtype=torch.float64, generator=torch.Generator().manual_seed(17))
    with torch.no_grad():
        ref = (x + bn2(pw2(F.relu(bn1(pw1(bn0(conv(x)))))))).permute(0, 2, 3, 1).numpy()
    p = cf.grouped_block_params_from_modules(conv, bn0, pw1, bn1, pw2, bn2, dtype=torch.float64)
    assert tuple(p["gw_w"].shape) == (3, 3, C, gw)
    got = oracle.gblock_forward(x.permute(0, 2, 3, 1).numpy(), {kk: (None if v is None else v.numpy())
                                                                 for kk, v in p.items()}, act="relu")
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-5 * np.abs(ref).max())


def test_downsample_from_torch_modules_matches_the_modules():
    conv = _rand_conv(nn.Conv2d(6, 10, 2, stride=2, bias=True).double(), 21)
    bn = _bn(10, 22)
    x = torch.randn(2, 6, 8, 6, dtype=torch.float64, generator=torch.Generator().manual_seed(23))
    with torch.no_grad():
        ref = bn(conv(x)).permute(0, 2, 3, 1).numpy()
    p = cf.down_params_from_modules(conv, bn, dtype=torch.float64)
    got = oracle.downsample(x.permute(0, 2, 3, 1).numpy(), p["wd"].numpy(), p["sd"].numpy(),
                            p["bd"].numpy())
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-5 * np.abs(ref).max())


def test_stem_from_torch_modules_matches_the_modules():
    """The stem conv (3 -> 24, 3x3, stride 2, padding 1) with its BN and ReLU,
    on an odd-sized image, against the oracle on the converted parameters."""
    conv = _rand_conv(nn.Conv2d(3, 24, 3, stride=2, padding=1, bias=True).double(), 31)
    bn = _bn(24, 32)
    x = torch.randn(2, 3, 9, 12, dtype=torch.float64, generator=torch.Generator().manual_seed(33))
    with torch.no_grad():
        ref = F.relu(bn(conv(x))).permute(0, 2, 3, 1).numpy()
    p = cf.stem_params_from_modules(conv, bn, dtype=torch.float64)
    assert tuple(p["sw"].shape) == (24, 3, 3, 3)
    got = oracle.stem_forward(x.permute(0, 2, 3, 1).numpy(), p["sw"].numpy(), p["ss"].numpy(), p["sb"].numpy())
    assert got.shape == (2, 5, 6, 24)
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-5 * np.abs(ref).max())
    with pytest.raises(ValueError):
        cf.stem_params_from_modules(nn.Conv2d(3, 16, 3, stride=1, padding=1))


def test_fold_batchnorm_rejects_training_mode():
    with pytest.raises(ValueError):
        cf.fold_batchnorm(nn.BatchNorm2d(4))


def test_layout_conversions_on_known_values():
    w = torch.arange(3 * 1 * 5 * 5).reshape(3, 1, 5, 5)
    d = cf.dw_weight_from_conv2d(w)
    assert d.shape == (5, 5, 3) and d[1, 4, 2] == w[2, 0, 1, 4]
    w = torch.arange(16 * 8 * 3 * 3).reshape(16, 8, 3, 3)
    g = cf.grouped_weight_from_conv2d(w)
    assert g.shape == (3, 3, 16, 8) and g[2, 0, 11, 5] == w[11, 5, 2, 0]
    w = torch.arange(4 * 6 * 2 * 2).reshape(4, 6, 2, 2)
    dn = cf.down_weight_from_conv2d(w)
    assert dn.shape == (4, 2, 2, 6) and dn[3, 1, 0, 5] == w[3, 5, 1, 0]
