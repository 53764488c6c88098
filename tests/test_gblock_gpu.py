"""Parity of the paper's own ConvFirst block (3 x 3 grouped conv of group
width 8, FFN, residual; Sec. 5.3) on the GPU with the fp64 oracle.

Gate: max |gpu - oracle| <= 2e-2 * max |oracle| over the whole output; the
fp16 cases also meet the diagnostic bound DIAG_F16.  Covers every supported
channel count, expansions whose hidden width is not a multiple of 32, edge
shapes (single pixel, widths below and not a multiple of the 16-column block,
odd heights), both I/O dtypes, the three activations, and the eight shapes of
the paper's kernel benchmark table at batch 128."""
import sys

import pytest
import torch

import oracle
import paper_2404_03617_amd as cf
from paper_2404_03617_amd import synth
from paper_2404_03617_amd.workloads import GBLOCK_WORKLOADS

from _util import DIAG_F16, assert_close, to_dev

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def make(seed, N, H, W, C, E, dtype="f16", scales="uniform", bias_std=1.0):
    x = synth.activations(seed, N, H, W, C, dtype)
    p = synth.gblock_params(seed, 0, C, E, 3, dtype, scales=scales, bias_std=bias_std)
    return x, p


def ref(x, p, act="relu"):
    return oracle.gblock_forward(synth.to_f64(x), synth.params_f64(p), act=act)


SWEEP = [
    # C, E, N, H, W
    (16, 3, 2, 9, 13),      # E*C = 48: the last hidden chunk is half padding
    (16, 1, 1, 1, 1),       # a single pixel
    (32, 3, 2, 5, 37),      # width not a multiple of 16, odd height
    (32, 6, 1, 16, 16),
    (48, 6, 3, 7, 7),       # C = 48: the second expand K step is half padding
    (48, 2, 1, 2, 40),
    (64, 6, 2, 11, 20),
    (64, 1, 1, 33, 3),      # tall, narrow
    (80, 3, 2, 6, 17),
    (96, 6, 1, 12, 12),
    (112, 2, 2, 5, 9),
    (96, 1, 1, 4, 33),      # one row band, three segments
    (112, 4, 1, 9, 18),
]


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("case", SWEEP, ids=lambda c: "C%d_E%d_N%d_%dx%d" % c)
def test_gblock_matches_oracle(case, dtype):
    C, E, N, H, W = case
    say("gblock", case, dtype)
    x, p = make(71, N, H, W, C, E, dtype)
    xd, pd = x.cuda(), to_dev(p)
    for act in ("relu", "gelu", "none"):
        y = cf.gblock_forward(xd, pd, act=act)
        torch.cuda.synchronize()
        assert_close(y, ref(x, p, act), what="gblock %s %s %s" % (case, dtype, act),
                     diag=DIAG_F16 if dtype == "f16" else None)


def test_gblock_null_scales_and_biases():
    x, p = make(72, 2, 6, 18, 32, 3, scales="none", bias_std=None)
    y = cf.gblock_forward(x.cuda(), to_dev(p))
    assert_close(y, ref(x, p), what="gblock null scale/bias", diag=DIAG_F16)


def test_gblock_zero_project_weights_pass_the_residual_exactly():
    x, p = make(73, 2, 7, 21, 48, 6)
    p["w2"] = torch.zeros_like(p["w2"])
    p["b2"] = None
    y = cf.gblock_forward(x.cuda(), to_dev(p))
    assert torch.equal(y.cpu(), x)


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_gblock_images_are_independent_and_deterministic(dtype):
    N, H, W, C, E = 9, 10, 20, 64, 6
    x, p = make(74, N, H, W, C, E, dtype)
    xd, pd = x.cuda(), to_dev(p)
    y = cf.gblock_forward(xd, pd)
    assert torch.equal(y, cf.gblock_forward(xd, pd))
    x2 = xd.clone()
    x2[0] = synth.activations(75, 1, H, W, C, dtype)[0].cuda()
    y2 = cf.gblock_forward(x2, pd)
    torch.cuda.synchronize()
    assert torch.equal(y[1:], y2[1:])
    assert not torch.equal(y[0], y2[0])


@pytest.mark.parametrize("name", list(GBLOCK_WORKLOADS))
def test_gblock_paper_table_shapes(name):
    """The eight shapes of the paper's kernel benchmark table at batch 128,
    whole output against the oracle (the benchmark's own inputs)."""
    w = GBLOCK_WORKLOADS[name]
    say("gblock workload", name)
    x = synth.activations(w["seed"], w["N"], w["H"], w["W"], w["C"], w["dtype"])
    p = synth.gblock_params(w["seed"], 0, w["C"], w["E"], w["k"], w["dtype"])
    y = cf.gblock_forward(x.cuda(), to_dev(p), act=w["act"])
    torch.cuda.synchronize()
    assert_close(y.cpu(), ref(x, p, w["act"]), what=name, diag=DIAG_F16)
