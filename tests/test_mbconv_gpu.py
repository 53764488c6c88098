"""Parity of the fused MBConv + Squeeze & Excitation kernel (Sec. 5.4, 5.4.1)
on the GPU with the fp64 oracle.

Gate: max |gpu - oracle| <= 2e-2 * max |oracle| over the whole output (the
sampled images at batch 128); fp16 cases also meet the diagnostic bound
DIAG_F16.  Covers one to sixteen hidden groups per image, C not a multiple of
32 or 64 (half K steps, partial output-channel blocks), every image size
class (one pixel, one row, one column, odd sizes, 16 x 16), R from 1 to 256,
both I/O dtypes, null scales and biases, evaluation in place, a workspace
for a single image in flight, independence of the images, determinism, and
the ten shapes of the paper's MBConv benchmark table at batch 128."""
import sys

import pytest
import torch

import oracle
import paper_2404_03617_amd as cf
from paper_2404_03617_amd import synth
from paper_2404_03617_amd.workloads import MBCONV_WORKLOADS

from _util import DIAG_F16, assert_close, to_dev

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def make(seed, N, H, W, C, E, R, dtype="f16", scales="uniform", bias_std=0.5):
    x = synth.activations(seed, N, H, W, C, dtype)
    p = synth.mbconv_params(seed, 0, C, E, R, dtype, scales=scales, bias_std=bias_std)
    return x, p


def ref(x, p):
    return oracle.mbconv_forward(synth.to_f64(x), synth.params_f64(p))


def run(x, p, **kw):
    """The kernel on x (CPU tensor) with its own workspace; returns (y, ws)."""
    N, H, W, C = x.shape
    EC, R = p["w1"].shape[0], p["wr"].shape[0]
    xd = x.cuda()
    ws = torch.zeros(max(1, cf.mbconv_workspace_bytes(N, H, W, C, EC // C, R, x.dtype)), dtype=torch.uint8,
                     device="cuda")
    y = cf.mbconv_forward(xd, to_dev(p), ws=ws, **kw)
    torch.cuda.synchronize()
    return y, ws


def barrier_flag(ws):
    return int(ws[:4].view(torch.int32).item())


SWEEP = [
    # C, E, R, N, H, W
    (16, 4, 4, 2, 5, 6),       # one hidden group: the barriers meet at once
    (32, 2, 8, 3, 7, 9),
    (48, 4, 12, 2, 16, 16),    # C % 32 == 16: the last expand K step is half padding
    (64, 4, 16, 3, 11, 13),    # P = 143: the 8-wave kernel with a ragged tile
    (128, 4, 32, 4, 8, 8),     # the paper's 8 x 8 shape, 4-wave kernel, one tile per wave
    (144, 4, 36, 2, 16, 16),   # C % 64 == 16: a partial block of output channels
    (160, 4, 40, 2, 8, 8),
    (64, 1, 256, 2, 1, 1),     # one pixel, the largest R
    (80, 4, 1, 2, 3, 16),      # R = 1, full-width rows
    (96, 2, 24, 2, 16, 1),     # one column
    (128, 6, 32, 1, 12, 10),   # P = 120: 4 waves, two tiles each
    (256, 4, 64, 2, 5, 7),     # sixteen hidden groups
]


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("case", SWEEP, ids=lambda c: "C%d_E%d_R%d_N%d_%dx%d" % c)
def test_mbconv_matches_oracle(case, dtype):
    C, E, R, N, H, W = case
    say("mbconv", case, dtype)
    x, p = make(81, N, H, W, C, E, R, dtype)
    y, ws = run(x, p)
    assert barrier_flag(ws) == 0
    assert_close(y, ref(x, p), what="mbconv %s %s" % (case, dtype), diag=DIAG_F16 if dtype == "f16" else None)
    # the ordinary launch of the same grid gives the same bits
    ye, wse = run(x, p, launch="exclusive")
    assert barrier_flag(wse) == 0
    assert torch.equal(ye, y)


def test_mbconv_null_scales_and_biases():
    x, p = make(82, 2, 9, 9, 64, 4, 16, scales="none", bias_std=None)
    assert all(p[k] is None for k in ("s1", "b1", "s2", "b2", "br", "be", "s3", "b3"))
    y, _ = run(x, p)
    assert_close(y, ref(x, p), what="mbconv null scale/bias", diag=DIAG_F16)


def test_mbconv_zero_project_weights_pass_the_residual_exactly():
    x, p = make(83, 3, 8, 8, 64, 4, 16)
    p["w2"] = torch.zeros_like(p["w2"])
    p["b3"] = None
    y, _ = run(x, p)
    assert torch.equal(y.cpu(), x)


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_mbconv_in_place_and_small_workspace_match_bitwise(dtype):
    """y = x in place, and a workspace for one image in flight (the images
    then run one after another), give the same bits as the default call."""
    N, H, W, C, E, R = 6, 16, 16, 128, 4, 32
    x, p = make(84, N, H, W, C, E, R, dtype)
    y, _ = run(x, p)
    xd, pd = x.cuda(), to_dev(p)
    cf.mbconv_forward(xd, pd, out=xd)
    torch.cuda.synchronize()
    assert torch.equal(xd, y)
    lib = cf.lib()
    full = lib.cf_mbconv_workspace_bytes(N, H, W, C, E, R, cf.DTYPES[x.dtype])
    # the workspace for one image in flight: flag and barrier lines, squeeze
    # shares, the two halves of one image's exchange buffer
    G = E * C // 64
    one_slot = 256 + 2048 * 128 + ((N * G * R * 4 + 255) // 256) * 256 + 2 * H * W * E * C * 2
    assert one_slot <= full
    ws = torch.zeros(one_slot, dtype=torch.uint8, device="cuda")
    y1 = cf.mbconv_forward(x.cuda(), pd, ws=ws)
    torch.cuda.synchronize()
    assert barrier_flag(ws) == 0
    assert torch.equal(y1, y)
    small = torch.empty(one_slot - 256, dtype=torch.uint8, device="cuda")
    with pytest.raises(cf.CFError) as ei:
        cf.mbconv_forward(x.cuda(), pd, ws=small)
    assert ei.value.status == cf.CF_ERR_WORKSPACE


def test_mbconv_images_are_independent_and_deterministic():
    """The squeeze couples the pixels of one image and no others: changing
    image 0 leaves the bits of every other image unchanged."""
    N, H, W, C, E, R = 9, 8, 8, 128, 4, 32
    x, p = make(85, N, H, W, C, E, R)
    xd, pd = x.cuda(), to_dev(p)
    y = cf.mbconv_forward(xd, pd)
    assert torch.equal(y, cf.mbconv_forward(xd, pd))
    x2 = xd.clone()
    x2[0] = synth.activations(86, 1, H, W, C)[0].cuda()
    y2 = cf.mbconv_forward(x2, pd)
    torch.cuda.synchronize()
    assert torch.equal(y[1:], y2[1:])
    assert not torch.equal(y[0], y2[0])


SAMPLE = [0, 37, 90, 127]


@pytest.mark.parametrize("name", list(MBCONV_WORKLOADS))
def test_mbconv_paper_table_shapes(name):
    """The ten shapes of the paper's MBConv table at batch 128 (the benchmark's
    own inputs); the oracle checks four images spread over the batch (the
    images are independent, pinned above and in the oracle's tests)."""
    w = MBCONV_WORKLOADS[name]
    say("mbconv workload", name)
    x = synth.activations(w["seed"], w["N"], w["H"], w["W"], w["C"], w["dtype"])
    p = synth.mbconv_params(w["seed"], 0, w["C"], w["E"], w["R"], w["dtype"])
    y, ws = run(x, p)
    assert barrier_flag(ws) == 0
    assert torch.isfinite(y.float()).all()
    assert_close(y.cpu()[SAMPLE], ref(x[SAMPLE], p), what=name, diag=DIAG_F16)


def test_mbconv_workspace_reused_across_calls():
    """One zeroed workspace serves a sequence of calls of different shapes
    and batch sizes (every call leaves the barrier lines at zero): each output
    equals, bit for bit, the output with a fresh workspace."""
    shapes = [(128, 4, 32, 6, 16, 16), (128, 4, 32, 9, 8, 8), (256, 4, 64, 3, 5, 7), (64, 2, 16, 20, 4, 4),
              (128, 4, 32, 6, 16, 16)]
    need = max(cf.mbconv_workspace_bytes(N, H, W, C, E, R) for C, E, R, N, H, W in shapes)
    ws = torch.zeros(need, dtype=torch.uint8, device="cuda")
    for i, (C, E, R, N, H, W) in enumerate(shapes):
        x, p = make(90 + i, N, H, W, C, E, R)
        xd, pd = x.cuda(), to_dev(p)
        for _ in range(2):
            y = cf.mbconv_forward(xd, pd, ws=ws)
            torch.cuda.synchronize()
            assert barrier_flag(ws) == 0
            assert torch.equal(y, cf.mbconv_forward(xd, pd))
