"""Parity of the block for a handful of pixels (N*H*W <= 64, C = 128, 256,
512) with the fp64 oracle.  cf_block_forward runs these shapes by default on
one workgroup per 32 output channels, each recomputing the expand and summing
its waves' projections in LDS (no workspace).

Gate: max |gpu - oracle| <= 2e-2 * max |oracle| over the whole output; fp16
cases also meet DIAG_F16.  Covers one and two 32-pixel blocks (P = 1, 32, 33,
45, 49, 64), k = 1 to 7 with taps crossing the image border, E = 1 to 4, the
three activations, both dtypes, null scales and biases, image independence
and determinism."""
import sys

import pytest
import torch

import paper_2404_03617_amd as cf

from _util import DIAG_F16, assert_close, make_block, oracle_block, to_dev

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


SHAPES = [
    # C, E, k, N, H, W
    (128, 4, 3, 1, 7, 7),
    (128, 1, 5, 2, 4, 8),     # 64 pixels, two images
    (128, 2, 7, 1, 1, 1),     # one pixel: every tap but the centre is padding
    (256, 4, 3, 4, 4, 4),     # four images of 4 x 4
    (256, 2, 1, 1, 1, 33),    # 33 pixels: the second block holds one
    (256, 4, 7, 1, 8, 8),
    (512, 4, 3, 1, 7, 7),     # the N = 1 latency workload's shape
    (512, 1, 5, 3, 3, 5),     # 45 pixels over three images
    (512, 2, 7, 1, 2, 32),    # 64 pixels, rows shorter than the taps are tall
    (512, 4, 3, 1, 1, 32),    # exactly one block
]


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("case", SHAPES, ids=lambda c: "C%d_E%d_k%d_N%d_%dx%d" % c)
def test_slice_block_matches_oracle(case, dtype):
    C, E, k, N, H, W = case
    say("slice", case, dtype)
    x, p = make_block(71, N, H, W, C, E, k, dtype)
    xd, pd = x.cuda(), to_dev(p)
    for act in ("gelu", "relu", "none"):
        y = cf.block_forward(xd, pd, act=act)
        torch.cuda.synchronize()
        assert_close(y, oracle_block(x, p, act), what="slice %s %s %s" % (case, dtype, act),
                     diag=DIAG_F16 if dtype == "f16" else None)


def test_slice_null_scales_and_biases():
    x, p = make_block(72, 1, 7, 7, 512, 4, 3, "bf16", scales="none", bias_std=None)
    assert all(p[k] is None for k in ("s0", "b0", "s1", "b1", "s2", "b2"))
    y = cf.block_forward(x.cuda(), to_dev(p))
    assert_close(y, oracle_block(x, p), what="slice null scale/bias")


def test_slice_zero_project_weights_pass_the_residual_exactly():
    x, p = make_block(73, 2, 4, 5, 256, 4, 3, "f16")
    p["w2"] = torch.zeros_like(p["w2"])
    p["b2"] = None
    y = cf.block_forward(x.cuda(), to_dev(p))
    assert torch.equal(y.cpu(), x)


def test_slice_images_are_independent_and_deterministic():
    N, H, W, C, E, k = 4, 4, 4, 256, 4, 3
    x, p = make_block(74, N, H, W, C, E, k, "bf16")
    xd, pd = x.cuda(), to_dev(p)
    y = cf.block_forward(xd, pd)
    assert torch.equal(y, cf.block_forward(xd, pd))
    x2 = xd.clone()
    x2[1] = make_block(75, 1, H, W, C, E, k, "bf16")[0][0].cuda()
    y2 = cf.block_forward(x2, pd)
    torch.cuda.synchronize()
    assert torch.equal(y[0], y2[0]) and torch.equal(y[2:], y2[2:])
    assert not torch.equal(y[1], y2[1])
