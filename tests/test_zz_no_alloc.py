"""The allocation-free split entry point (cf_block_forward_split_noalloc)
against the workspace one (cf_block_forward_split): same kernels, partials in
the library's static device scratch instead of the caller's workspace.

Two calls in a row, the second on a smaller input (the scratch keeps the first
call's contents), each checked bit for bit against the workspace entry point
and against the fp64 oracle; a call whose partials exceed the scratch is
rejected before any launch; with a preallocated output the call makes no
allocation through torch."""
import ctypes

import pytest
import torch

import paper_2404_03617_amd as cf

from _util import assert_close, make_block, oracle_block, to_dev

pytestmark = pytest.mark.gpu

# (C, E, k, N, H, W, groups, dtype): the first is the N = 1, 7x7, C = 512 bf16
# latency workload with 64 hidden groups (6.4 MB of partials), the second a
# smaller one (0.4 MB), so the second call reads a scratch the first filled.
CALLS = [(512, 4, 3, 1, 7, 7, 64, "bf16"), (64, 4, 3, 1, 14, 14, 8, "f16")]


def test_noalloc_matches_the_workspace_entry_point_on_two_calls():
    for i, (C, E, k, N, H, W, groups, dtype) in enumerate(CALLS):
        print("noalloc call", i, (C, E, k, N, H, W, groups, dtype), flush=True)
        x, p = make_block(61 + i, N, H, W, C, E, k, dtype)
        xd, pd = x.cuda(), to_dev(p)
        ref_ws = cf.block_forward_split(xd, pd, groups=groups)
        out = torch.empty_like(xd)
        torch.cuda.synchronize()
        before = torch.cuda.memory_stats().get("allocation.all.allocated", 0)
        y = cf.block_forward_split_noalloc(xd, pd, groups=groups, out=out)
        after = torch.cuda.memory_stats().get("allocation.all.allocated", 0)
        torch.cuda.synchronize()
        assert after == before, "the call allocated through torch"
        assert y.data_ptr() == out.data_ptr()
        assert torch.equal(y, ref_ws), "call %d differs from cf_block_forward_split" % i
        assert_close(y.cpu(), oracle_block(x, p), what="noalloc call %d" % i)


def test_noalloc_rejects_partials_beyond_the_scratch():
    # N = 3, 14x14, C = 256, 32 groups: 19.3 MB of partials > 16 MiB
    x, p = make_block(63, 3, 14, 14, 256, 4, 3, "f16")
    xd, pd = x.cuda(), to_dev(p)
    y = torch.full_like(xd, 7.0)
    with pytest.raises(cf.CFError) as ei:
        cf.block_forward_split_noalloc(xd, pd, groups=32, out=y)
    assert ei.value.status == cf.CF_ERR_WORKSPACE
    assert "scratch" in str(ei.value)
    torch.cuda.synchronize()
    assert bool((y == 7.0).all()), "a rejected call must not touch y"
