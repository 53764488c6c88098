"""Pins for the oracle's stride-2 MBConv block (Fig. f:mbconv, stride 2;
Sec. 5.4): BlurPool with the Triangle-3 filter after the grouped conv, the
squeeze over the down-sampled map, the project to K channels and no
residual.  BlurPool is checked against torch (reflect padding + a strided
per-channel conv), closed forms and hand-computed values at the border; the
block against a torch float64 composition and the case that isolates the
missing residual.  CPU only."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle

RNG = np.random.default_rng(4242)
TRI = np.array([0.25, 0.5, 0.25])


def rand(*shape):
    return RNG.standard_normal(shape)


def torch_blurpool(x):
    """x [N,H,W,Ch] -> reflect pad 1, per-channel 3x3 outer(TRI, TRI), stride 2."""
    xt = torch.from_numpy(x).permute(0, 3, 1, 2)
    Ch = xt.shape[1]
    w = torch.from_numpy(np.outer(TRI, TRI))[None, None].repeat(Ch, 1, 1, 1)
    return F.conv2d(F.pad(xt, (1, 1, 1, 1), mode="reflect"), w, stride=2, groups=Ch).permute(0, 2, 3, 1).numpy()


@pytest.mark.parametrize("H,W", [(2, 2), (3, 5), (16, 16), (7, 2), (9, 12)])
def test_blurpool_matches_torch(H, W):
    x = rand(2, H, W, 5)
    y = oracle.blurpool_tri3(x)
    assert y.shape == (2, (H + 1) // 2, (W + 1) // 2, 5)
    np.testing.assert_allclose(y, torch_blurpool(x), rtol=0, atol=1e-14)


def test_blurpool_keeps_a_constant_image():
    """The taps sum to one and reflection repeats image pixels: a constant
    image stays constant, borders included."""
    x = np.full((1, 7, 6, 3), 2.5)
    np.testing.assert_array_equal(oracle.blurpool_tri3(x), np.full((1, 4, 3, 3), 2.5))


def test_blurpool_impulse_responses():
    """An impulse on an even pixel of the interior reaches one output with
    weight 1/4; on an odd pixel it reaches four outputs with 1/16 each; at the
    corner (0, 1) the reflected copy adds to the direct tap: output (0, 0)
    reads rows {1, 0, 1} and columns {1, 0, 1}, so pixel (0, 1) counts with
    weight t1 * (t0 + t2) = 1/4, and output (0, 1) reads columns {1, 2, 3}:
    t1 * t0 = 1/8."""
    x = np.zeros((1, 9, 9, 1))
    x[0, 4, 4, 0] = 1.0
    y = oracle.blurpool_tri3(x)[0, :, :, 0]
    exp = np.zeros((5, 5))
    exp[2, 2] = 0.25
    np.testing.assert_array_equal(y, exp)
    x = np.zeros((1, 9, 9, 1))
    x[0, 3, 5, 0] = 1.0
    y = oracle.blurpool_tri3(x)[0, :, :, 0]
    exp = np.zeros((5, 5))
    exp[1:3, 2:4] = 1.0 / 16
    np.testing.assert_array_equal(y, exp)
    x = np.zeros((1, 6, 6, 1))
    x[0, 0, 1, 0] = 1.0
    y = oracle.blurpool_tri3(x)[0, :, :, 0]
    exp = np.zeros((3, 3))
    exp[0, 0] = 0.25
    exp[0, 1] = 0.125
    np.testing.assert_array_equal(y, exp)


def params(C, E, R, K, k=3, gw=8, scales=True):
    EC = E * C
    p = {"w1": rand(EC, C) / np.sqrt(C), "gw_w": rand(k, k, EC, gw) / np.sqrt(k * k * gw),
         "wr": rand(R, EC) / np.sqrt(EC), "we": rand(EC, R) / np.sqrt(R), "w2": rand(K, EC) / np.sqrt(EC),
         "b1": rand(EC) * 0.5, "b2": rand(EC) * 0.5, "br": rand(R) * 0.5, "be": rand(EC) * 0.5, "b3": rand(K) * 0.5}
    if scales:
        p.update(s1=RNG.uniform(0.5, 1.5, EC), s2=RNG.uniform(0.5, 1.5, EC), s3=RNG.uniform(0.5, 1.5, K))
    return p


def torch_mbconv_s2(x, p, pool_before_blur=False):
    t = lambda a: None if a is None else torch.from_numpy(np.asarray(a))
    xt = torch.from_numpy(x)
    EC = p["w1"].shape[0]
    k, _, _, gw = p["gw_w"].shape
    u = F.linear(xt, t(p["w1"]))
    if p.get("s1") is not None:
        u = u * t(p["s1"])
    u = F.silu(u + t(p["b1"]))
    wt = t(p["gw_w"]).permute(2, 3, 0, 1).contiguous()
    v = F.conv2d(u.permute(0, 3, 1, 2), wt, padding=k // 2, groups=EC // gw)
    if p.get("s2") is not None:
        v = v * t(p["s2"])[:, None, None]
    v = F.silu(v + t(p["b2"])[:, None, None])
    bw = torch.from_numpy(np.outer(TRI, TRI))[None, None].repeat(EC, 1, 1, 1)
    sq_full = F.adaptive_avg_pool2d(v, 1).flatten(1)
    v = F.conv2d(F.pad(v, (1, 1, 1, 1), mode="reflect"), bw, stride=2, groups=EC)
    sq = sq_full if pool_before_blur else F.adaptive_avg_pool2d(v, 1).flatten(1)
    z = F.relu(F.linear(sq, t(p["wr"]), t(p["br"])))
    g = torch.sigmoid(F.linear(z, t(p["we"]), t(p["be"])))
    vg = (v * g[:, :, None, None]).permute(0, 2, 3, 1)
    out = F.linear(vg, t(p["w2"]))
    if p.get("s3") is not None:
        out = out * t(p["s3"])
    return (out + t(p["b3"])).numpy()


@pytest.mark.parametrize("C,E,R,K,H,W", [(16, 4, 4, 24, 6, 6), (8, 2, 2, 8, 3, 5), (16, 1, 4, 32, 2, 2),
                                          (24, 4, 6, 16, 7, 4)])
def test_mbconv_s2_matches_torch_composition(C, E, R, K, H, W):
    x = rand(2, H, W, C)
    p = params(C, E, R, K)
    y = oracle.mbconv_s2_forward(x, p)
    assert y.shape == (2, (H + 1) // 2, (W + 1) // 2, K)
    np.testing.assert_allclose(y, torch_mbconv_s2(x, p), rtol=0, atol=1e-11)


def test_mbconv_s2_without_scales_matches_torch():
    x = rand(2, 4, 5, 16)
    p = params(16, 2, 4, 8, scales=False)
    np.testing.assert_allclose(oracle.mbconv_s2_forward(x, p), torch_mbconv_s2(x, p), rtol=0, atol=1e-11)


def test_mbconv_s2_has_no_residual():
    """With zero project weights the output is b3 at every pixel (the
    stride-1 block would return x + b3)."""
    x = rand(2, 6, 6, 16)
    p = params(16, 4, 4, 16)
    p["w2"] = np.zeros_like(p["w2"])
    y = oracle.mbconv_s2_forward(x, p)
    np.testing.assert_array_equal(y, np.broadcast_to(p["b3"], y.shape))


def test_mbconv_s2_squeeze_reads_the_blurred_map():
    """The gates come from the mean of the down-sampled map: the oracle
    equals the composition that pools the blurred map and differs from the
    one that pools V before the blur (the two means differ for a
    non-constant image)."""
    x = rand(1, 5, 5, 16)
    p = params(16, 2, 4, 16)
    y = oracle.mbconv_s2_forward(x, p)
    np.testing.assert_allclose(y, torch_mbconv_s2(x, p), rtol=0, atol=1e-11)
    assert np.abs(y - torch_mbconv_s2(x, p, pool_before_blur=True)).max() > 1e-6
