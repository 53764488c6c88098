"""Pins for the oracle's grouped-conv block (the paper's own ConvFirst block,
Sec. 5.3: grouped k x k conv of group width 8, FFN, residual) and for the
oracle's stack composition.  Everything is checked against something other
than the function under test: brute-force loops, the grouped conv written in
the paper's index order (eq. f:grouped-conv2d), torch float64 library
routines, and the degenerate cases that reduce to other pinned functions
(group width 1 = depth-wise, one group = dense conv).  CPU only."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle

RNG = np.random.default_rng(4321)


def rand(*shape):
    return RNG.standard_normal(shape)


def brute_gconv(x, a, s, b):
    """x [N,H,W,C], a [k,k,C,gw]: direct sum with explicit zero padding."""
    N, H, W, C = x.shape
    k, _, _, gw = a.shape
    pad = k // 2
    xp = np.zeros((N, H + 2 * pad, W + 2 * pad, C))
    xp[:, pad:pad + H, pad:pad + W] = x
    out = np.zeros_like(x)
    for n in range(N):
        for h in range(H):
            for w in range(W):
                for c in range(C):
                    g0 = (c // gw) * gw
                    acc = 0.0
                    for i in range(k):
                        for j in range(k):
                            for t in range(gw):
                                acc += a[i, j, c, t] * xp[n, h + i, w + j, g0 + t]
                    out[n, h, w, c] = s[c] * acc + b[c]
    return out


def torch_gconv(x, a):
    """torch conv2d(groups = C / gw) in float64; a [k,k,C,gw] -> torch [C,gw,k,k]."""
    k, _, C, gw = a.shape
    wt = torch.from_numpy(np.ascontiguousarray(a.transpose(2, 3, 0, 1)))
    return F.conv2d(torch.from_numpy(x).permute(0, 3, 1, 2), wt, padding=k // 2,
                    groups=C // gw).permute(0, 2, 3, 1).numpy()


@pytest.mark.parametrize("k,gw,C", [(1, 8, 16), (3, 8, 16), (3, 2, 6), (5, 4, 8), (3, 1, 3)])
@pytest.mark.parametrize("H,W", [(1, 1), (2, 5), (4, 3)])
def test_gconv_brute_force(k, gw, C, H, W):
    x, a, s, b = rand(2, H, W, C), rand(k, k, C, gw), rand(C), rand(C)
    np.testing.assert_allclose(oracle.gconv(x, a, s, b), brute_gconv(x, a, s, b), rtol=0, atol=1e-12)


@pytest.mark.parametrize("k,gw,C", [(3, 8, 16), (3, 8, 48), (5, 8, 32), (7, 4, 12), (1, 8, 24)])
def test_gconv_matches_torch_grouped_conv2d(k, gw, C):
    x, a = rand(2, 9, 7, C), rand(k, k, C, gw)
    np.testing.assert_allclose(oracle.gconv(x, a), torch_gconv(x, a), rtol=0, atol=1e-11)


@pytest.mark.parametrize("gw,C", [(8, 16), (8, 32), (4, 12), (1, 5)])
def test_gconv_equals_the_papers_grouped_conv_equation(gw, C):
    """The block layer against eq. f:grouped-conv2d written in the paper's
    [K][R][S][T] index order with g(k) = floor(kC / (KT)), K = C."""
    x, a = rand(2, 6, 8, C), rand(3, 3, C, gw)
    paper = oracle.grouped_conv(x, a.transpose(2, 0, 1, 3), groups=C // gw, stride=1, pad=1)
    np.testing.assert_allclose(oracle.gconv(x, a), paper, rtol=0, atol=1e-12)


def test_papers_grouped_conv_equation_matches_torch_with_stride_and_more_outputs():
    """The generic form itself, with K != C (g(k) = floor(kC/(KT))), stride 2."""
    C, K, T = 8, 16, 4
    x, a = rand(2, 7, 9, C), rand(K, 3, 3, T)
    got = oracle.grouped_conv(x, a, groups=C // T, stride=2, pad=1)
    ref = F.conv2d(torch.from_numpy(x).permute(0, 3, 1, 2),
                   torch.from_numpy(np.ascontiguousarray(a.transpose(0, 3, 1, 2))), stride=2, padding=1,
                   groups=C // T).permute(0, 2, 3, 1).numpy()
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


def test_gconv_group_width_one_is_the_depthwise_layer():
    x, a, s, b = rand(2, 5, 6, 7), rand(3, 3, 7, 1), rand(7), rand(7)
    assert np.array_equal(oracle.gconv(x, a, s, b), oracle.depthwise(x, a[..., 0], s, b))


def test_gconv_one_group_is_a_dense_conv():
    C = 6
    x, a = rand(1, 5, 4, C), rand(3, 3, C, C)
    wt = torch.from_numpy(np.ascontiguousarray(a.transpose(2, 3, 0, 1)))
    ref = F.conv2d(torch.from_numpy(x).permute(0, 3, 1, 2), wt, padding=1).permute(0, 2, 3, 1).numpy()
    np.testing.assert_allclose(oracle.gconv(x, a), ref, rtol=0, atol=1e-11)


@pytest.mark.parametrize("k", [1, 3, 5])
def test_gconv_delta_kernel_is_identity(k):
    C, gw = 16, 8
    x = rand(2, 4, 5, C)
    a = np.zeros((k, k, C, gw))
    for c in range(C):
        a[k // 2, k // 2, c, c % gw] = 1.0
    assert np.array_equal(oracle.gconv(x, a), x)


def test_gconv_reads_only_its_own_group():
    """Changing the input channels of group 1 leaves group 0's outputs alone."""
    C, gw = 16, 8
    x, a = rand(1, 5, 5, C), rand(3, 3, C, gw)
    x2 = x.copy()
    x2[..., 8:] = rand(1, 5, 5, 8)
    d, d2 = oracle.gconv(x, a), oracle.gconv(x2, a)
    assert np.array_equal(d[..., :8], d2[..., :8])
    assert not np.allclose(d[..., 8:], d2[..., 8:])


# ---------------------------------------------------------------- grouped block
def params(C, E, k, gw, scales=True):
    p = {"gw_w": rand(k, k, C, gw) / np.sqrt(k * k * gw), "w1": rand(E * C, C) / np.sqrt(C),
         "w2": rand(C, E * C) / np.sqrt(E * C), "b0": rand(C), "b1": rand(E * C), "b2": rand(C)}
    if scales:
        p.update(s0=RNG.uniform(0.5, 1.5, C), s1=RNG.uniform(0.5, 1.5, E * C), s2=RNG.uniform(0.5, 1.5, C))
    return p


def torch_gblock(x, p, act):
    t = lambda a: None if a is None else torch.from_numpy(np.asarray(a))
    xt = torch.from_numpy(x)
    a = p["gw_w"]
    k, _, C, gw = a.shape
    d = torch.from_numpy(torch_gconv(x, a))
    if p.get("s0") is not None:
        d = d * t(p["s0"])
    d = d + t(p["b0"])
    u = F.linear(d, t(p["w1"]))
    if p.get("s1") is not None:
        u = u * t(p["s1"])
    u = u + t(p["b1"])
    g = {"relu": F.relu, "gelu": lambda v: F.gelu(v, approximate="none"), "none": lambda v: v}[act](u)
    z = F.linear(g, t(p["w2"]))
    if p.get("s2") is not None:
        z = z * t(p["s2"])
    return (xt + z + t(p["b2"])).numpy()


@pytest.mark.parametrize("act", ["relu", "gelu", "none"])
@pytest.mark.parametrize("C,E,k,H,W", [(16, 3, 3, 5, 7), (32, 6, 3, 4, 4), (24, 2, 5, 3, 6), (8, 1, 1, 2, 3)])
def test_gblock_matches_torch_composition(act, C, E, k, H, W):
    x = rand(2, H, W, C)
    p = params(C, E, k, 8)
    np.testing.assert_allclose(oracle.gblock_forward(x, p, act=act), torch_gblock(x, p, act), rtol=0,
                               atol=1e-11)


def test_gblock_group_width_one_is_the_depthwise_block():
    C, E = 8, 3
    x = rand(2, 5, 4, C)
    p = params(C, E, 3, 1)
    q = {kk: v for kk, v in p.items() if kk != "gw_w"}
    q["dw_w"] = p["gw_w"][..., 0]
    for act in ("relu", "gelu"):
        assert np.array_equal(oracle.gblock_forward(x, p, act=act), oracle.block_forward(x, q, act=act))


def test_gblock_zero_project_weights_pass_the_residual():
    x = rand(2, 4, 6, 16)
    p = params(16, 3, 3, 8)
    p["w2"] = np.zeros_like(p["w2"])
    p["b2"] = np.zeros(16)
    assert np.array_equal(oracle.gblock_forward(x, p), x)


def test_gblock_identity_activation_is_affine():
    """With phi = identity the block is affine in x: f(a x1 + b x2) - f(0)
    = a (f(x1) - f(0)) + b (f(x2) - f(0))."""
    p = params(16, 2, 3, 8)
    x1, x2 = rand(1, 4, 5, 16), rand(1, 4, 5, 16)
    f = lambda x: oracle.gblock_forward(x, p, act="none")
    f0 = f(np.zeros_like(x1))
    lhs = f(0.7 * x1 - 1.3 * x2) - f0
    rhs = 0.7 * (f(x1) - f0) - 1.3 * (f(x2) - f0)
    np.testing.assert_allclose(lhs, rhs, atol=1e-11)


def test_gblock_batch_independence():
    p = params(16, 3, 3, 8)
    x = rand(3, 5, 5, 16)
    y = oracle.gblock_forward(x, p)
    for n in range(3):
        assert np.array_equal(y[n:n + 1], oracle.gblock_forward(x[n:n + 1], p))


# ---------------------------------------------------------------- stack
def torch_block(xt, p, act):
    t = lambda a: None if a is None else torch.from_numpy(np.asarray(a))
    k, _, C = p["dw_w"].shape
    d = F.conv2d(xt.permute(0, 3, 1, 2), t(p["dw_w"]).permute(2, 0, 1).unsqueeze(1), padding=k // 2,
                 groups=C).permute(0, 2, 3, 1)
    d = d * t(p["s0"]) + t(p["b0"])
    u = F.linear(d, t(p["w1"])) * t(p["s1"]) + t(p["b1"])
    g = {"relu": F.relu, "gelu": lambda v: F.gelu(v, approximate="none")}[act](u)
    return xt + F.linear(g, t(p["w2"])) * t(p["s2"]) + t(p["b2"])


def torch_down(xt, p):
    t = lambda a: torch.from_numpy(np.asarray(a))
    y = F.conv2d(xt.permute(0, 3, 1, 2), t(p["wd"]).permute(0, 3, 1, 2), stride=2).permute(0, 2, 3, 1)
    return y * t(p["sd"]) + t(p["bd"])


@pytest.mark.parametrize("act", ["gelu", "relu"])
def test_stack_matches_torch_composition(act):
    """oracle.stack_forward against blocks (depth-wise conv2d, linear, phi,
    linear, residual) and 2x2 stride-2 convs composed in torch float64,
    with an odd layer order (block, down, block, block, down)."""
    def blk(C, E=2, k=3):
        return ("block", {"dw_w": rand(k, k, C) / k, "s0": RNG.uniform(0.5, 1.5, C), "b0": rand(C),
                          "w1": rand(E * C, C) / np.sqrt(C), "s1": RNG.uniform(0.5, 1.5, E * C),
                          "b1": rand(E * C), "w2": rand(C, E * C) / np.sqrt(E * C),
                          "s2": RNG.uniform(0.5, 1.5, C), "b2": rand(C)})

    def down(ci, co):
        return ("down", {"wd": rand(co, 2, 2, ci) / np.sqrt(4 * ci), "sd": RNG.uniform(0.5, 1.5, co),
                         "bd": rand(co)})

    layers = [blk(4), down(4, 6), blk(6, k=5), blk(6, E=3), down(6, 8)]
    x = rand(2, 8, 12, 4)
    xt = torch.from_numpy(x)
    for kind, p in layers:
        xt = torch_block(xt, p, act) if kind == "block" else torch_down(xt, p)
    got = oracle.stack_forward(x, layers, act=act)
    assert got.shape == (2, 2, 3, 8)
    np.testing.assert_allclose(got, xt.numpy(), rtol=0, atol=1e-11)
