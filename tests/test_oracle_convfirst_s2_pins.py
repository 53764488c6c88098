"""Pins for the oracle's stride-2 ConvFirst block (Fig. f:convfirst-block
(c)) in the reading the speed-projection counts support: grouped conv C -> C
at the input size, BlurPool (Triangle-3) of the conv output and of the block
input, both concatenated (conv output first) into the expand, activation,
project to K, no residual.  Checked against a torch float64 composition,
cases that isolate each half of the concatenation and its order, the missing
residual, and every distinct stride-2 ConvFirst row of App. A (the expand
reads 2C channels at the output size).  CPU only."""
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
RNG = np.random.default_rng(2404)
TRI = np.array([0.25, 0.5, 0.25])


def rand(*shape):
    return RNG.standard_normal(shape)


def params(C, R, K, k=3, gw=8, scales=True):
    p = {"gw_w": rand(k, k, C, gw) / np.sqrt(k * k * gw), "w1": rand(R, 2 * C) / np.sqrt(2 * C),
         "w2": rand(K, R) / np.sqrt(R), "b0": rand(C) * 0.5, "b1": rand(R) * 0.5, "b2": rand(K) * 0.5}
    if scales:
        p.update(s0=RNG.uniform(0.5, 1.5, C), s1=RNG.uniform(0.5, 1.5, R), s2=RNG.uniform(0.5, 1.5, K))
    return p


def torch_blurpool(v):
    """v [N,Ch,H,W] -> reflect pad 1, per-channel 3x3 outer(TRI, TRI), stride 2."""
    Ch = v.shape[1]
    w = torch.from_numpy(np.outer(TRI, TRI))[None, None].repeat(Ch, 1, 1, 1)
    return F.conv2d(F.pad(v, (1, 1, 1, 1), mode="reflect"), w, stride=2, groups=Ch)


def torch_convfirst_s2(x, p, act="relu"):
    t = lambda a: None if a is None else torch.from_numpy(np.asarray(a))
    xt = torch.from_numpy(x).permute(0, 3, 1, 2)
    C = xt.shape[1]
    k, _, _, gw = p["gw_w"].shape
    wt = t(p["gw_w"]).permute(2, 3, 0, 1).contiguous()
    d = F.conv2d(xt, wt, padding=k // 2, groups=C // gw)
    if p.get("s0") is not None:
        d = d * t(p["s0"])[:, None, None]
    if p.get("b0") is not None:
        d = d + t(p["b0"])[:, None, None]
    z = torch.cat([torch_blurpool(d), torch_blurpool(xt)], dim=1).permute(0, 2, 3, 1)
    u = F.linear(z, t(p["w1"]))
    if p.get("s1") is not None:
        u = u * t(p["s1"])
    if p.get("b1") is not None:
        u = u + t(p["b1"])
    u = {"relu": F.relu, "gelu": F.gelu, "none": lambda v: v}[act](u)
    y = F.linear(u, t(p["w2"]))
    if p.get("s2") is not None:
        y = y * t(p["s2"])
    if p.get("b2") is not None:
        y = y + t(p["b2"])
    return y.numpy()


@pytest.mark.parametrize("act", ["relu", "gelu", "none"])
@pytest.mark.parametrize("C,R,K,H,W", [(16, 96, 32, 6, 6), (8, 24, 16, 5, 7), (24, 48, 8, 2, 2), (16, 32, 48, 9, 4)])
def test_convfirst_s2_matches_torch_composition(C, R, K, H, W, act):
    x = rand(2, H, W, C)
    p = params(C, R, K)
    y = oracle.convfirst_s2_forward(x, p, act)
    assert y.shape == (2, (H + 1) // 2, (W + 1) // 2, K)
    np.testing.assert_allclose(y, torch_convfirst_s2(x, p, act), rtol=0, atol=1e-11)


def test_convfirst_s2_without_scales_and_biases_matches_torch():
    x = rand(2, 7, 6, 16)
    p = params(16, 32, 16, scales=False)
    for key in ("b0", "b1", "b2"):
        p[key] = None
    np.testing.assert_allclose(oracle.convfirst_s2_forward(x, p), torch_convfirst_s2(x, p), rtol=0, atol=1e-11)


def identity_case(C, which):
    """Identity weights routed through one half of the concatenation: W1 =
    [I | 0] (the conv half) or [0 | I] (the input half), no activation, W2 =
    I, no norms; the conv taps are the identity (centre tap, own channel)."""
    a = np.zeros((3, 3, C, 8))
    for c in range(C):
        a[1, 1, c, c % 8] = 1.0
    w1 = np.zeros((C, 2 * C))
    w1[:, (0 if which == "conv" else C):(C if which == "conv" else 2 * C)] = np.eye(C)
    return {"gw_w": a, "w1": w1, "w2": np.eye(C)}


def test_each_half_of_the_concatenation_is_the_blurred_map():
    """With identity taps D = X, so either half alone gives BlurPool(X)."""
    x = rand(2, 7, 6, 16)
    bp = oracle.blurpool_tri3(x)
    for which in ("conv", "input"):
        y = oracle.convfirst_s2_forward(x, identity_case(16, which), act="none")
        np.testing.assert_allclose(y, bp, rtol=0, atol=1e-14)


def test_concatenation_order_conv_first():
    """Conv half first: with s0 = 0 the conv output is the constant b0, so
    W1 = [I | 0] gives b0 everywhere (BlurPool keeps constants) and
    W1 = [0 | I] gives BlurPool(X)."""
    x = rand(1, 6, 8, 16)
    b0 = rand(16)
    p = identity_case(16, "conv")
    p.update(s0=np.zeros(16), b0=b0)
    y = oracle.convfirst_s2_forward(x, p, act="none")
    np.testing.assert_allclose(y, np.broadcast_to(b0, y.shape), rtol=0, atol=1e-14)
    p = identity_case(16, "input")
    p.update(s0=np.zeros(16), b0=b0)
    np.testing.assert_allclose(oracle.convfirst_s2_forward(x, p, act="none"), oracle.blurpool_tri3(x),
                               rtol=0, atol=1e-14)


def test_convfirst_s2_has_no_residual():
    x = rand(2, 6, 6, 16)
    p = params(16, 32, 16)
    p["w2"] = np.zeros_like(p["w2"])
    y = oracle.convfirst_s2_forward(x, p)
    np.testing.assert_array_equal(y, np.broadcast_to(p["b2"], y.shape))


def _rows():
    rows = []
    with open(os.path.join(ROOT, "tests", "golden", "convfirst_s2_projection_rows.txt")) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                v = line.split()
                rows.append(tuple(int(a) for a in v[:5]) + tuple(float(a) for a in v[5:]))
    return rows


@pytest.mark.parametrize("row", _rows(), ids=lambda r: "%dx%d_C%d_R%d_K%d" % r[:5])
def test_layer_sizes_reproduce_the_projection_tables(row):
    """Operations per image from the oracle's layer shapes (a 3 x 3 conv of
    group width 8 over C channels at H x W; W1 [R, 2C] and W2 [K, R] at the
    output size): every Conv, Exp and Prj value printed for a stride-2
    ConvFirst row.  An expand from C channels (the block without the input
    half) would give half the printed Exp."""
    H, W, C, R, K, conv, exp, prj, total = row
    p = params(C, R, K)
    Ho, Wo = (H + 1) // 2, (W + 1) // 2
    k, _, _, gw = p["gw_w"].shape
    assert 2 * H * W * C * k * k * gw / 1e6 == pytest.approx(conv, abs=0.005)
    assert 2 * Ho * Wo * p["w1"].size / 1e6 == pytest.approx(exp, abs=0.005)
    assert 2 * Ho * Wo * p["w2"].size / 1e6 == pytest.approx(prj, abs=0.005)
    assert (conv + exp + prj) == pytest.approx(total, abs=0.015)
    assert 2 * Ho * Wo * C * R / 1e6 == pytest.approx(exp / 2, abs=0.005)


@pytest.mark.parametrize("row", _rows(), ids=lambda r: "%dx%d_C%d_R%d_K%d" % r[:5])
def test_roofline_count_reproduces_the_projection_tables(row):
    """roofline.convfirst_s2_flops per image equals the printed row total."""
    from paper_2404_03617_amd import roofline as rl
    H, W, C, R, K, conv, exp, prj, total = row
    assert rl.convfirst_s2_flops(1, H, W, C, R, K) / 1e6 == pytest.approx(total, abs=0.015)
