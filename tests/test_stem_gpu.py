"""Parity of the network stem (3x3 stride-2 conv from 3 channels, folded
norm, ReLU; App. A) and of the stem fused into the first ConvFirst block
(the grouped-conv block, Sec. 5.3) with the fp64 oracle.

Gate: max |gpu - oracle| <= 2e-2 * max |oracle| over the whole output (the
sampled images at batch 128); fp16 cases also meet DIAG_F16.  The fused
kernel must equal, bit for bit, the stem kernel followed by the grouped
block kernel: both round the stem output to the I/O dtype the same way, so
any difference is an error of the halo computed from the image."""
import sys

import pytest
import torch

import oracle
import paper_2404_03617_amd as cf
from paper_2404_03617_amd import synth
from paper_2404_03617_amd.workloads import STEM_WORKLOADS

from _util import DIAG_F16, assert_close, to_dev

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def make(seed, N, Hin, Win, C, E, dtype="f16", scales="uniform", bias_std=0.5):
    x = synth.activations(seed, N, Hin, Win, 3, dtype)
    st = synth.stem_params(seed, 0, C, dtype, scales=scales, bias_std=bias_std)
    p = synth.gblock_params(seed, 1, C, E, 3, dtype, scales=scales, bias_std=bias_std)
    return x, st, p


def ref_stem(x, st):
    return oracle.stem_forward(synth.to_f64(x), synth.to_f64(st["sw"]), synth.to_f64(st.get("ss")),
                               synth.to_f64(st.get("sb")))


def ref_fused(x, st, p, act="relu"):
    return oracle.stem_gblock_forward(synth.to_f64(x), synth.params_f64(st), synth.params_f64(p), act=act)


SHAPES = [
    # N, Hin, Win
    (2, 16, 16),
    (1, 9, 13),     # odd sizes: the last stem row and column see the padding
    (3, 1, 1),      # one stem pixel
    (2, 37, 70),    # several 16-column segments, a ragged row band
    (1, 64, 34),
]


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("C", [16, 32])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "N%d_%dx%d" % s)
def test_stem_and_fused_block_match_oracle(shape, C, dtype):
    N, Hin, Win = shape
    say("stem", shape, C, dtype)
    x, st, p = make(31, N, Hin, Win, C, 3, dtype)
    xd, sd, pd = x.cuda(), to_dev(st), to_dev(p)
    s = cf.stem_forward(xd, sd)
    torch.cuda.synchronize()
    diag = DIAG_F16 if dtype == "f16" else None
    assert_close(s, ref_stem(x, st), what="stem %s C%d %s" % (shape, C, dtype), diag=diag)
    for act in ("relu", "gelu", "none"):
        y = cf.stem_gblock_forward(xd, sd, pd, act=act)
        torch.cuda.synchronize()
        assert torch.equal(y, cf.gblock_forward(s, pd, act=act)), "fused != stem kernel + block kernel"
        assert_close(y, ref_fused(x, st, p, act), what="stem+block %s C%d %s %s" % (shape, C, dtype, act), diag=diag)


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "N%d_%dx%d" % s)
def test_stem_c24_matches_oracle(shape, dtype):
    """The paper's third stem width: two channel tiles, the second half used."""
    N, Hin, Win = shape
    say("stem C24", shape, dtype)
    x = synth.activations(35, N, Hin, Win, 3, dtype)
    st = synth.stem_params(35, 0, 24, dtype, scales="uniform", bias_std=0.5)
    xd = x.cuda()
    y = torch.full((N, (Hin + 1) // 2, (Win + 1) // 2, 24), 7.0, dtype=xd.dtype, device="cuda")
    cf.stem_forward(xd, to_dev(st), out=y)
    torch.cuda.synchronize()
    assert_close(y, ref_stem(x, st), what="stem C24 %s %s" % (shape, dtype),
                 diag=DIAG_F16 if dtype == "f16" else None)


def test_fused_null_scales_and_biases():
    x, st, p = make(32, 2, 20, 18, 16, 3, scales="none", bias_std=None)
    y = cf.stem_gblock_forward(x.cuda(), to_dev(st), to_dev(p))
    assert_close(y, ref_fused(x, st, p), what="stem+block null scale/bias", diag=DIAG_F16)


def test_fused_images_are_independent():
    N, Hin, Win, C = 5, 30, 40, 32
    x, st, p = make(33, N, Hin, Win, C, 3)
    xd, sd, pd = x.cuda(), to_dev(st), to_dev(p)
    y = cf.stem_gblock_forward(xd, sd, pd)
    assert torch.equal(y, cf.stem_gblock_forward(xd, sd, pd))
    x2 = xd.clone()
    x2[2] = synth.activations(34, 1, Hin, Win, 3)[0].cuda()
    y2 = cf.stem_gblock_forward(x2, sd, pd)
    torch.cuda.synchronize()
    assert torch.equal(y[:2], y2[:2]) and torch.equal(y[3:], y2[3:])
    assert not torch.equal(y[2], y2[2])


SAMPLE = [0, 45, 127]


@pytest.mark.parametrize("name", list(STEM_WORKLOADS))
def test_stem_workloads(name):
    """The two stem + first-block shapes at batch 128 (the benchmark's own
    inputs): the fused kernel equals the unfused pair on the whole tensor;
    the oracle checks three images spread over the batch."""
    w = STEM_WORKLOADS[name]
    say("stem workload", name)
    x = synth.activations(w["seed"], w["N"], w["Hin"], w["Win"], 3, w["dtype"])
    st = synth.stem_params(w["seed"], 0, w["C"], w["dtype"])
    p = synth.gblock_params(w["seed"], 1, w["C"], w["E"], w["k"], w["dtype"])
    xd, sd, pd = x.cuda(), to_dev(st), to_dev(p)
    y = cf.stem_gblock_forward(xd, sd, pd, act=w["act"])
    torch.cuda.synchronize()
    assert torch.equal(y, cf.gblock_forward(cf.stem_forward(xd, sd), pd, act=w["act"]))
    assert_close(y.cpu()[SAMPLE], ref_fused(x[SAMPLE], st, p, w["act"]), what=name, diag=DIAG_F16)
