"""The C = 512 stage run layer by layer (depth-wise kernel, two hipBLASLt
GEMMs, two elementwise kernels), which cf_stage_forward takes for fp16
C = 512 stages over at least 4096 pixels when its workspace has the room
(the block of Sec. 5.2 evaluated in the unfused schedule).  Compared with
the fp64 oracle on images spread over the batch (images are independent:
every GEMM row is one pixel), with null scales and biases, and as graph
replays."""
import sys

import pytest
import torch

import oracle
import paper_2404_03617_amd as cf
from paper_2404_03617_amd import synth

from _util import DIAG_F16, assert_close, to_dev

pytestmark = pytest.mark.gpu

N, H, W, C, E, K3 = 96, 7, 7, 512, 4, 3  # 4704 pixels
SAMPLE = [0, 41, 95]


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def stage(seed, depth, scales="uniform", bias_std=0.5):
    x = synth.activations(seed, N, H, W, C, "f16")
    blocks = [synth.block_params(seed, i, C, E, K3, "f16", scales=scales, bias_std=bias_std) for i in range(depth)]
    return x, blocks


def ref(x, blocks, act):
    return oracle.stack_forward(synth.to_f64(x[SAMPLE]), [("block", synth.params_f64(b)) for b in blocks], act=act)


@pytest.mark.parametrize("act", ["gelu", "relu", "none"])
def test_c512_layer_by_layer_stage_matches_oracle(act):
    say("c512 layer-by-layer stage", act)
    x, blocks = stage(301, 2)
    xd, bd = x.cuda(), [to_dev(b) for b in blocks]
    y = cf.stage_forward(xd, bd, act=act)
    torch.cuda.synchronize()
    assert_close(y.cpu()[SAMPLE], ref(x, blocks, act), what="c512 stage %s" % act, diag=DIAG_F16)
    assert torch.equal(y, cf.stage_forward(xd, bd, act=act))  # deterministic


def test_c512_layer_by_layer_null_scales_and_biases():
    x, blocks = stage(303, 2, scales="none", bias_std=None)
    assert all(b[k] is None for b in blocks for k in ("s0", "b0", "s1", "b1", "s2", "b2"))
    xd, bd = x.cuda(), [to_dev(b) for b in blocks]
    y = cf.stage_forward(xd, bd)
    torch.cuda.synchronize()
    assert_close(y.cpu()[SAMPLE], ref(x, blocks, "gelu"), what="c512 null vectors", diag=DIAG_F16)


def test_c512_layer_by_layer_graph_replays_match_eager():
    """The stage captured after an eager call (the library plans exist) and
    replayed three times with eager work in between: every replay equals the
    eager output bit for bit."""
    x, blocks = stage(305, 2)
    xd, bd = x.cuda(), [to_dev(b) for b in blocks]
    need = cf.lib().cf_stage_workspace_bytes(2, N, H, W, C, cf.DTYPES[torch.float16])
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    y_eager = cf.stage_forward(xd, bd, ws=ws).clone()
    out = torch.empty_like(xd)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        cf.stage_forward(xd, bd, ws=ws, out=out)
    for i in range(3):
        out.zero_()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, y_eager), "replay %d" % i
        cf.stage_forward(xd, bd)  # eager work between replays
        torch.cuda.synchronize()
