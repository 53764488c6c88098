"""The micro-batched stage schedule (Sec. 5.5.2) on the GPU: every block of
the stage over a micro-batch of images before the next micro-batch.  Its
output is the same function of the input as the plain stage: compared with
the fp64 oracle over the whole output, and bit for bit with cf_stage_forward
where both run the same kernels (no hidden split)."""
import sys

import pytest
import torch

import oracle
import paper_2404_03617_amd as cf
from paper_2404_03617_amd import synth

from _util import assert_close, to_dev

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def stage(seed, depth, N, H, W, C, E, k, dtype="f16"):
    x = synth.activations(seed, N, H, W, C, dtype)
    blocks = [synth.block_params(seed, i, C, E, k, dtype, scales="uniform", bias_std=0.5) for i in range(depth)]
    return x, blocks


def oracle_stage(x, blocks, act="gelu"):
    return oracle.stack_forward(synth.to_f64(x), [("block", synth.params_f64(b)) for b in blocks], act=act)


@pytest.mark.parametrize("case", [
    # depth, N, H, W, C, E, k, micro_batch, dtype
    (2, 10, 9, 13, 64, 4, 3, 3, "f16"),    # micro-batches 3, 3, 3, 1
    (3, 5, 7, 9, 128, 2, 5, 2, "f16"),     # three blocks: both ping-pong buffers
    (2, 4, 14, 14, 256, 4, 7, 0, "f16"),   # default micro-batch size
    (2, 3, 7, 7, 512, 4, 3, 2, "f16"),
    (4, 6, 6, 10, 64, 4, 3, 1, "bf16"),    # one image at a time
    (1, 5, 8, 8, 128, 4, 3, 2, "f16"),     # a single block needs no workspace
    (2, 3, 5, 5, 64, 4, 3, 8, "f16"),      # micro-batch larger than the batch
], ids=lambda c: "D%d_N%d_%dx%d_C%d_E%d_k%d_m%d_%s" % c)
def test_microbatch_stage_matches_oracle_and_plain_stage(case):
    depth, N, H, W, C, E, k, m, dtype = case
    say("microbatch stage", case)
    x, blocks = stage(81, depth, N, H, W, C, E, k, dtype)
    xd, bd = x.cuda(), [to_dev(b) for b in blocks]
    y = cf.stage_forward_microbatch(xd, bd, micro_batch=m)
    torch.cuda.synchronize()
    assert_close(y.cpu(), oracle_stage(x, blocks), what="microbatch stage %s" % (case,))
    if C != 512:  # (a plain C = 512 fp16 stage may split its hidden layer: other summation order)
        assert torch.equal(y, cf.stage_forward(xd, bd))


def test_microbatch_stage_full_size_first_stage_of_the_stack():
    """Stage 1 of the four-stage stack (two C = 64 blocks at 56 x 56, N = 128)
    with the default micro-batch, whole output against the oracle."""
    name = "stack_n128_56x56_d2262_c64to512_e4_k3_f16"
    from paper_2404_03617_amd.workloads import WORKLOADS
    w = WORKLOADS[name]
    x = synth.activations(w["seed"], w["N"], w["H"], w["W"], w["widths"][0], w["dtype"])
    layers = synth.stack_layers(w["seed"], w["depths"], w["widths"], w["E"], w["k"], w["dtype"])
    blocks = [p for _, p in layers[:w["depths"][0]]]
    say("microbatch stage 1 of", name)
    y = cf.stage_forward_microbatch(x.cuda(), [to_dev(b) for b in blocks])
    torch.cuda.synchronize()
    assert_close(y.cpu(), oracle_stage(x, blocks), what="stage 1 micro-batched")
