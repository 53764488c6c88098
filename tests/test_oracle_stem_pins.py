"""Pins for the oracle's stem (a 3 x 3 stride-2 convolution from 3 channels,
folded batch norm, ReLU; App. A and the ConvFirstNet figure caption) and for
the stem followed by the first ConvFirst block.  Checked against torch
float64 library routines and special cases that fix the stride, the
padding and the channel order.  CPU only."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle

RNG = np.random.default_rng(2024)


def torch_stem(x, w, s=None, b=None):
    u = F.conv2d(torch.from_numpy(x).permute(0, 3, 1, 2), torch.from_numpy(w).permute(0, 3, 1, 2).contiguous(),
                 stride=2, padding=1)
    if s is not None:
        u = u * torch.from_numpy(s)[:, None, None]
    if b is not None:
        u = u + torch.from_numpy(b)[:, None, None]
    return F.relu(u).permute(0, 2, 3, 1).numpy()


@pytest.mark.parametrize("H,W,C", [(8, 8, 16), (7, 9, 16), (1, 1, 32), (2, 5, 16), (13, 6, 32), (11, 10, 24)])
def test_stem_matches_torch(H, W, C):
    x = RNG.standard_normal((2, H, W, 3))
    w = RNG.standard_normal((C, 3, 3, 3)) / 5.0           # [K][R][S][T]
    s, b = RNG.uniform(0.5, 1.5, C), RNG.standard_normal(C) * 0.5
    y = oracle.stem_forward(x, w, s, b)
    assert y.shape == (2, (H + 1) // 2, (W + 1) // 2, C)
    np.testing.assert_allclose(y, torch_stem(x, w, s, b), rtol=0, atol=1e-12)
    np.testing.assert_allclose(oracle.stem_forward(x, w), torch_stem(x, w), rtol=0, atol=1e-12)


def test_stem_centre_tap_samples_even_pixels():
    """A kernel that is 1 at the centre tap of input channel t copies
    x[2r, 2c, t] (stride 2, one pixel of padding); ReLU clips the negatives."""
    x = RNG.standard_normal((1, 9, 10, 3))
    w = np.zeros((16, 3, 3, 3))
    for k in range(16):
        w[k, 1, 1, k % 3] = 1.0
    y = oracle.stem_forward(x, w)
    want = np.maximum(x[:, 0::2, 0::2, :][..., [k % 3 for k in range(16)]], 0.0)
    assert np.array_equal(y, want)


def test_stem_corner_taps_see_the_padding():
    """The top-left tap reads row 2r-1, column 2c-1: zero for the first output
    row and column, x[2r-1, 2c-1] elsewhere."""
    x = np.abs(RNG.standard_normal((1, 6, 6, 3))) + 0.1
    w = np.zeros((16, 3, 3, 3))
    w[:, 0, 0, 1] = 1.0
    y = oracle.stem_forward(x, w)
    assert np.all(y[0, 0, :, :] == 0.0) and np.all(y[0, :, 0, :] == 0.0)
    np.testing.assert_array_equal(y[0, 1:, 1:, 0], x[0, 1:5:2, 1:5:2, 1])


def test_stem_block_composition_matches_torch():
    """Stem, then grouped conv (group width 8) + FFN + ReLU + residual, composed
    in torch float64."""
    N, H, W, C, E = 2, 10, 12, 16, 3
    x = RNG.standard_normal((N, H, W, 3))
    sw = RNG.standard_normal((C, 3, 3, 3)) / 5.0
    ss, sb = RNG.uniform(0.5, 1.5, C), RNG.standard_normal(C) * 0.3
    p = {"gw_w": RNG.standard_normal((3, 3, C, 8)) / 8.0, "w1": RNG.standard_normal((E * C, C)) / 4.0,
         "w2": RNG.standard_normal((C, E * C)) / 7.0, "s0": RNG.uniform(0.5, 1.5, C),
         "b0": RNG.standard_normal(C) * 0.3, "b1": RNG.standard_normal(E * C) * 0.3, "b2": RNG.standard_normal(C) * 0.3}
    y = oracle.stem_gblock_forward(x, {"sw": sw, "ss": ss, "sb": sb}, p)
    t = lambda a: torch.from_numpy(a)
    u = t(torch_stem(x, sw, ss, sb))                                       # [N, H/2, W/2, C]
    d = F.conv2d(u.permute(0, 3, 1, 2), t(p["gw_w"]).permute(2, 3, 0, 1).contiguous(), padding=1, groups=C // 8)
    d = (d * t(p["s0"])[:, None, None] + t(p["b0"])[:, None, None]).permute(0, 2, 3, 1)
    h = F.relu(F.linear(d, t(p["w1"]), t(p["b1"])))
    ref = (u + F.linear(h, t(p["w2"]), t(p["b2"]))).numpy()
    np.testing.assert_allclose(y, ref, rtol=0, atol=1e-11)
