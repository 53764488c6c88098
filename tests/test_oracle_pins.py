"""Pins for the fp64 oracle against things other than itself: brute force on
tiny inputs, library routines (torch float64), closed forms, invariants and
textbook values.  Shapes are deliberately asymmetric (H != W, E*C != C,
non-symmetric kernels) so that a transposed operand or a swapped index fails.
CPU only."""
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))
RNG = np.random.default_rng(1234)


def rand(*shape):
    return RNG.standard_normal(shape)


# ---------------------------------------------------------------- depth-wise
def brute_depthwise(x, w, s, b):
    """Direct sum over taps with explicit zero padding, pure Python loops."""
    N, H, W, C = x.shape
    k = w.shape[0]
    pad = k // 2
    xp = np.zeros((N, H + 2 * pad, W + 2 * pad, C))
    xp[:, pad:pad + H, pad:pad + W, :] = x
    out = np.zeros_like(x)
    for n in range(N):
        for h in range(H):
            for ww in range(W):
                for c in range(C):
                    acc = 0.0
                    for i in range(k):
                        for j in range(k):
                            acc += w[i, j, c] * xp[n, h + i, ww + j, c]
                    out[n, h, ww, c] = s[c] * acc + b[c]
    return out


@pytest.mark.parametrize("k", [1, 3, 5, 7])
@pytest.mark.parametrize("H,W", [(1, 1), (2, 5), (5, 3), (6, 7)])
def test_depthwise_brute_force(k, H, W):
    N, C = 2, 3
    x, w, s, b = rand(N, H, W, C), rand(k, k, C), rand(C), rand(C)
    got = oracle.depthwise(x, w, s, b)
    np.testing.assert_allclose(got, brute_depthwise(x, w, s, b), rtol=0, atol=1e-12)


@pytest.mark.parametrize("k", [1, 3, 5, 7])
def test_depthwise_matches_torch_conv2d_groups(k):
    N, H, W, C = 2, 9, 6, 5
    x, w = rand(N, H, W, C), rand(k, k, C)
    ref = F.conv2d(torch.from_numpy(x).permute(0, 3, 1, 2),
                   torch.from_numpy(w).permute(2, 0, 1).unsqueeze(1),
                   padding=k // 2, groups=C).permute(0, 2, 3, 1).numpy()
    np.testing.assert_allclose(oracle.depthwise(x, w), ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("k", [1, 3, 5, 7])
def test_depthwise_delta_kernel_is_identity(k):
    x = rand(1, 4, 9, 6)
    w = np.zeros((k, k, 6))
    w[k // 2, k // 2, :] = 1.0
    assert np.array_equal(oracle.depthwise(x, w), x)


@pytest.mark.parametrize("k", [3, 5, 7])
def test_depthwise_constant_input_closed_form(k):
    """x == a, all-ones taps: D = a * (#in-image rows) * (#in-image cols)."""
    H, W, C, a = 5, 8, 2, 1.75
    x = np.full((1, H, W, C), a)
    d = oracle.depthwise(x, np.ones((k, k, C)))
    pad = k // 2
    for h in range(H):
        rows = min(h + pad, H - 1) - max(h - pad, 0) + 1
        for ww in range(W):
            cols = min(ww + pad, W - 1) - max(ww - pad, 0) + 1
            assert d[0, h, ww, 0] == pytest.approx(a * rows * cols, abs=1e-12)


def test_depthwise_translation_equivariance_interior():
    k, pad = 3, 1
    x = rand(1, 10, 12, 4)
    w = rand(k, k, 4)
    xs = np.roll(x, shift=(1, 2), axis=(1, 2))
    d, ds = oracle.depthwise(x, w), oracle.depthwise(xs, w)
    # interior of the shifted output, away from both the padding and the wrap
    np.testing.assert_allclose(ds[:, 1 + 1 + pad:-pad, 2 + 1 + pad:-pad],
                               d[:, 1 + pad:-pad - 1, 1 + pad:-pad - 2], atol=1e-12)


# ---------------------------------------------------------------- point-wise
def test_pointwise_is_matmul():
    x, a, s, b = rand(3, 4, 5, 6), rand(10, 6), rand(10), rand(10)
    got = oracle.pointwise(x, a, s, b)
    ref = (x.reshape(-1, 6) @ a.T) * s + b
    np.testing.assert_allclose(got.reshape(-1, 10), ref, rtol=1e-13, atol=1e-12)


def test_pointwise_matches_torch_conv1x1():
    x, a = rand(2, 3, 7, 8), rand(5, 8)
    ref = F.conv2d(torch.from_numpy(x).permute(0, 3, 1, 2),
                   torch.from_numpy(a)[:, :, None, None]).permute(0, 2, 3, 1).numpy()
    np.testing.assert_allclose(oracle.pointwise(x, a), ref, atol=1e-12)


# ---------------------------------------------------------------- activation
def _golden_cdf():
    rows = []
    with open(os.path.join(HERE, "golden", "normal_cdf.txt")) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                xv, pv = line.split()
                rows.append((float(xv), float(pv)))
    return rows


@pytest.mark.parametrize("xv,phi", _golden_cdf())
def test_gelu_equals_x_times_normal_cdf_table(xv, phi):
    assert oracle.act(xv, "gelu") == pytest.approx(xv * phi, abs=abs(xv) * 6e-10)


def test_gelu_identities():
    assert oracle.act(0.0, "gelu") == 0.0
    for u in np.linspace(-7, 7, 57):
        # odd part of u*Phi(u) is u/2: GELU(u) - GELU(-u) = u
        assert oracle.act(u, "gelu") - oracle.act(-u, "gelu") == pytest.approx(u, abs=1e-14)
    assert oracle.act(9.0, "gelu") == pytest.approx(9.0, abs=1e-15)
    assert abs(oracle.act(-9.0, "gelu")) < 1e-15


def test_gelu_matches_torch_exact_gelu():
    u = np.linspace(-8, 8, 401)
    ref = F.gelu(torch.from_numpy(u), approximate="none").numpy()
    got = np.array([oracle.act(v, "gelu") for v in u])
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-15)


def test_relu_and_identity():
    for u in (-2.5, -0.0, 0.0, 3.25):
        assert oracle.act(u, "relu") == max(u, 0.0)
        assert oracle.act(u, "none") == u


# ---------------------------------------------------------------- whole block
def _params(C, E, k, scales=True):
    EC = E * C
    p = {"dw_w": rand(k, k, C), "w1": rand(EC, C) / math.sqrt(C), "w2": rand(C, EC) / math.sqrt(EC),
         "b0": rand(C), "b1": rand(EC), "b2": rand(C)}
    if scales:
        p.update(s0=RNG.uniform(0.5, 1.5, C), s1=RNG.uniform(0.5, 1.5, EC),
                 s2=RNG.uniform(0.5, 1.5, C))
    return p


def torch_block(x, p, act):
    """The block composed from torch float64 library ops."""
    C = x.shape[-1]
    k = p["dw_w"].shape[0]
    t = lambda a: torch.from_numpy(np.asarray(a, dtype=np.float64))
    ones = lambda n: torch.ones(n, dtype=torch.float64)
    xt = t(x).permute(0, 3, 1, 2)
    d = F.conv2d(xt, t(p["dw_w"]).permute(2, 0, 1).unsqueeze(1), padding=k // 2, groups=C)
    d = d.permute(0, 2, 3, 1) * (t(p["s0"]) if "s0" in p else ones(C)) + t(p["b0"])
    EC = p["w1"].shape[0]
    u = F.linear(d, t(p["w1"])) * (t(p["s1"]) if "s1" in p else ones(EC)) + t(p["b1"])
    g = {"gelu": lambda v: F.gelu(v, approximate="none"), "relu": F.relu, "none": lambda v: v}[act](u)
    z = F.linear(g, t(p["w2"])) * (t(p["s2"]) if "s2" in p else ones(C)) + t(p["b2"])
    return (t(x) + z).numpy()


@pytest.mark.parametrize("act", ["gelu", "relu", "none"])
@pytest.mark.parametrize("C,E,k,H,W", [(4, 3, 3, 5, 7), (6, 2, 5, 4, 3), (3, 4, 7, 6, 2), (5, 1, 1, 3, 4)])
def test_block_matches_torch_composition(act, C, E, k, H, W):
    x = rand(2, H, W, C)
    p = _params(C, E, k)
    np.testing.assert_allclose(oracle.block_forward(x, p, act), torch_block(x, p, act),
                               rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("act", ["gelu", "relu", "none"])
def test_loop_fused_order_equals_layer_by_layer(act):
    """eq. e:ffn-eff (one hidden channel at a time) == eq. e:ffn."""
    x = rand(2, 6, 5, 8)
    p = _params(8, 4, 3)
    a = oracle.block_forward(x, p, act)
    b = oracle.block_forward(x, p, act, loopfused=True)
    np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-12)


def test_zero_project_weights_pass_the_residual():
    x = rand(1, 5, 6, 4)
    p = _params(4, 4, 3)
    p["w2"] = np.zeros_like(p["w2"])
    p["b2"] = np.zeros(4)
    assert np.array_equal(oracle.block_forward(x, p, "gelu"), x)
    p["b2"] = rand(4)
    np.testing.assert_array_equal(oracle.block_forward(x, p, "gelu"), x + p["b2"])


def test_identity_activation_block_is_affine():
    x1, x2 = rand(1, 5, 4, 3), rand(1, 5, 4, 3)
    p = _params(3, 2, 3)
    f = lambda v: oracle.block_forward(v, p, "none")
    al, be = 0.7, -1.3
    lhs = f(al * x1 + be * x2)
    rhs = al * f(x1) + be * f(x2) + (1 - al - be) * f(np.zeros_like(x1))
    np.testing.assert_allclose(lhs, rhs, atol=1e-11)


def test_batch_independence():
    x = rand(3, 5, 6, 4)
    p = _params(4, 3, 3)
    whole = oracle.block_forward(x, p, "gelu")
    for n in range(3):
        np.testing.assert_array_equal(whole[n:n + 1], oracle.block_forward(x[n:n + 1], p, "gelu"))


def test_threads_do_not_change_the_result():
    x = rand(2, 7, 5, 4)
    p = _params(4, 2, 5)
    a = oracle.block_forward(x, p, "gelu", nthreads=1)
    b = oracle.block_forward(x, p, "gelu", nthreads=5)
    assert np.array_equal(a, b)


def test_missing_scales_mean_one():
    x = rand(1, 4, 4, 4)
    p = _params(4, 2, 3, scales=False)
    q = dict(p, s0=np.ones(4), s1=np.ones(8), s2=np.ones(4))
    assert np.array_equal(oracle.block_forward(x, p), oracle.block_forward(x, q))


# ---------------------------------------------------------------- down-sampling
def test_downsample_matches_torch_strided_conv():
    x, wd, s, b = rand(2, 6, 8, 5), rand(7, 2, 2, 5), rand(7), rand(7)
    ref = F.conv2d(torch.from_numpy(x).permute(0, 3, 1, 2),
                   torch.from_numpy(wd).permute(0, 3, 1, 2), stride=2)
    ref = (ref.permute(0, 2, 3, 1) * torch.from_numpy(s) + torch.from_numpy(b)).numpy()
    np.testing.assert_allclose(oracle.downsample(x, wd, s, b), ref, atol=1e-12)


def test_downsample_is_space_to_depth_then_matmul():
    N, H, W, Cin, Cout = 1, 4, 6, 3, 4
    x, wd = rand(N, H, W, Cin), rand(Cout, 2, 2, Cin)
    s2d = x.reshape(N, H // 2, 2, W // 2, 2, Cin).transpose(0, 1, 3, 2, 4, 5).reshape(N, H // 2, W // 2, 4 * Cin)
    ref = s2d @ wd.reshape(Cout, 4 * Cin).T
    np.testing.assert_allclose(oracle.downsample(x, wd), ref, atol=1e-12)
