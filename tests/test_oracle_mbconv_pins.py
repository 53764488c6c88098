"""Pins for the oracle's MBConv + Squeeze & Excitation block (Sec. 5.4,
5.4.1): expand + SiLU, grouped conv (group width 8) + SiLU, SE gate,
project, residual.  Checked against torch float64 library routines and the
special cases that fix each part of the SE layer.  CPU only."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle

RNG = np.random.default_rng(777)


def rand(*shape):
    return RNG.standard_normal(shape)


def params(C, E, R, k=3, gw=8, scales=True):
    EC = E * C
    p = {"w1": rand(EC, C) / np.sqrt(C), "gw_w": rand(k, k, EC, gw) / np.sqrt(k * k * gw),
         "wr": rand(R, EC) / np.sqrt(EC), "we": rand(EC, R) / np.sqrt(R), "w2": rand(C, EC) / np.sqrt(EC),
         "b1": rand(EC) * 0.5, "b2": rand(EC) * 0.5, "br": rand(R) * 0.5, "be": rand(EC) * 0.5, "b3": rand(C) * 0.5}
    if scales:
        p.update(s1=RNG.uniform(0.5, 1.5, EC), s2=RNG.uniform(0.5, 1.5, EC), s3=RNG.uniform(0.5, 1.5, C))
    return p


def torch_mbconv(x, p):
    t = lambda a: None if a is None else torch.from_numpy(np.asarray(a))
    xt = torch.from_numpy(x)
    EC = p["w1"].shape[0]
    k, _, _, gw = p["gw_w"].shape
    u = F.linear(xt, t(p["w1"]))
    if p.get("s1") is not None:
        u = u * t(p["s1"])
    u = F.silu(u + t(p["b1"]))
    wt = t(p["gw_w"]).permute(2, 3, 0, 1).contiguous()          # [EC, gw, k, k]
    v = F.conv2d(u.permute(0, 3, 1, 2), wt, padding=k // 2, groups=EC // gw)
    if p.get("s2") is not None:
        v = v * t(p["s2"])[:, None, None]
    v = F.silu(v + t(p["b2"])[:, None, None])                   # [N, EC, H, W]
    sq = F.adaptive_avg_pool2d(v, 1).flatten(1)                  # [N, EC]
    z = F.relu(F.linear(sq, t(p["wr"]), t(p["br"])))
    g = torch.sigmoid(F.linear(z, t(p["we"]), t(p["be"])))
    vg = (v * g[:, :, None, None]).permute(0, 2, 3, 1)
    out = F.linear(vg, t(p["w2"]))
    if p.get("s3") is not None:
        out = out * t(p["s3"])
    return (xt + out + t(p["b3"])).numpy()


@pytest.mark.parametrize("C,E,R,H,W", [(16, 4, 4, 5, 6), (8, 2, 2, 3, 3), (16, 1, 4, 1, 1), (24, 4, 6, 4, 7)])
def test_mbconv_matches_torch_composition(C, E, R, H, W):
    x = rand(2, H, W, C)
    p = params(C, E, R)
    np.testing.assert_allclose(oracle.mbconv_forward(x, p), torch_mbconv(x, p), rtol=0, atol=1e-11)


def test_mbconv_without_scales_matches_torch():
    x = rand(2, 4, 5, 16)
    p = params(16, 2, 4, scales=False)
    np.testing.assert_allclose(oracle.mbconv_forward(x, p), torch_mbconv(x, p), rtol=0, atol=1e-11)


def test_zero_project_weights_pass_the_residual():
    x = rand(2, 4, 4, 16)
    p = params(16, 4, 4)
    p["w2"] = np.zeros_like(p["w2"])
    p["b3"] = np.zeros(16)
    assert np.array_equal(oracle.mbconv_forward(x, p), x)


def test_excitation_bias_alone_sets_the_gate():
    """With zero excitation weights the gate is sigmoid(be) for every image:
    be = 0 halves the projection (checked through linearity in the gate),
    and a large be opens it fully -- the block is then MBConv without SE."""
    x = rand(2, 4, 5, 16)
    p = params(16, 2, 4)
    p["we"] = np.zeros_like(p["we"])
    q = dict(p, w2=np.zeros_like(p["w2"]))
    base = oracle.mbconv_forward(x, q)                           # x + b3 (scaled bias only)
    p["be"] = np.full(32, 40.0)                                   # sigmoid(40) == 1.0 in fp64
    full = oracle.mbconv_forward(x, p)
    p["be"] = np.zeros(32)
    half = oracle.mbconv_forward(x, p)
    np.testing.assert_allclose(half - base, 0.5 * (full - base), atol=1e-12)
    # the fully open gate equals the torch block with the SE removed
    t = lambda a: torch.from_numpy(np.asarray(a))
    u = F.silu(F.linear(t(x), t(p["w1"])) * t(p["s1"]) + t(p["b1"]))
    v = F.conv2d(u.permute(0, 3, 1, 2), t(p["gw_w"]).permute(2, 3, 0, 1).contiguous(), padding=1, groups=4)
    v = F.silu(v * t(p["s2"])[:, None, None] + t(p["b2"])[:, None, None]).permute(0, 2, 3, 1)
    ref = (t(x) + F.linear(v, t(p["w2"])) * t(p["s3"]) + t(p["b3"])).numpy()
    np.testing.assert_allclose(full, ref, rtol=0, atol=1e-11)


def test_squeeze_couples_the_pixels_of_one_image_only():
    """The SE gate depends on every pixel of an image: changing one pixel of
    image 0 changes outputs far from it (beyond the 3x3 reach), and leaves
    image 1 untouched."""
    x = rand(2, 6, 6, 16)
    p = params(16, 2, 4)
    y = oracle.mbconv_forward(x, p)
    x2 = x.copy()
    x2[0, 0, 0] += 3.0
    y2 = oracle.mbconv_forward(x2, p)
    assert np.array_equal(y[1], y2[1])
    assert not np.allclose(y[0, 5, 5], y2[0, 5, 5], rtol=0, atol=1e-14)


def test_gate_is_a_per_channel_scale_of_the_hidden_layer():
    """Scaling We and be by zero and shifting be changes the output only
    through the gate: with R = 1, wr = 0 and br < 0 the squeeze is 0 and the
    gate is sigmoid(be) whatever the input."""
    x = rand(1, 3, 4, 8)
    p = params(8, 2, 1)
    p["wr"] = np.zeros_like(p["wr"])
    p["br"] = np.array([-1.0])
    y1 = oracle.mbconv_forward(x, p)
    y2 = oracle.mbconv_forward(x * 2.0, p)    # input changes, gate does not
    p2 = dict(p, we=rand(16, 1))              # any We: z = 0, so g = sigmoid(be)
    np.testing.assert_allclose(oracle.mbconv_forward(x, p2), y1, atol=1e-12)
    assert not np.allclose(y1, y2)
