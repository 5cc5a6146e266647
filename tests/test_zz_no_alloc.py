"""emu_reshard_noalloc, the reshard for callers that cannot allocate device memory: its plan tables live
in the library's static per-device array instead of a caller workspace. Its output must equal
emu_reshard's (which the other GPU tests check against the oracle) byte for byte, with the same write
footprint, over consecutive calls that switch plans (the second smaller than the first), come back to
an earlier plan, and repeat a plan whose tables are already resident; and replays of a HIP graph that
captured it must match the eager result.

Workloads: the 1B decoder bf16 TP4 PP1 -> TP2 PP1 (3.0 GB of destination shards), then the tiny decoder
TP1 PP1 -> TP2 PP1 (3.95 MB).
"""
import pytest

import oracle
from paper_2609_34645_amd import emu
from tests.gpu_util import Guard, check_reshard, fill_device, full_model, o_layout, say, upload_shards
from tests.shapes import ONE_B, TINY

pytestmark = pytest.mark.gpu
GUARD = 256


def _pair(plan, S, label):
    """emu_reshard into one prefilled set, emu_reshard_noalloc into another; equal bytes, both guarded."""
    import torch

    ws = plan.workspace()
    ref, got = plan.alloc(1, fill=0xA5, guard=GUARD), plan.alloc(1, fill=0xA5, guard=GUARD)
    g = Guard(keep=S.tensors, fills=[(ref.tensors, 0xA5)], label=f"{label}: emu_reshard")
    plan.reshard(ws, S.ptrs, ref.ptrs)
    torch.cuda.synchronize()
    g.check()
    g = Guard(keep=S.tensors, fills=[(got.tensors, 0xA5)], label=f"{label}: emu_reshard_noalloc")
    plan.reshard_noalloc(S.ptrs, got.ptrs)
    torch.cuda.synchronize()
    g.check()
    for i, (a, b) in enumerate(zip(ref.bufs, got.bufs)):
        assert torch.equal(a, b), f"{label}: rank buffer {i} differs from emu_reshard's"
    say(f"  {label}: emu_reshard_noalloc == emu_reshard ({plan.info['bytes_written']} bytes)")
    return got


def test_noalloc_matches_reshard(gpu_lib):
    import torch

    big = emu.Plan(emu.Layout(emu.Model(*ONE_B), 4, 1), emu.Layout(emu.Model(*ONE_B), 2, 1))
    tm = emu.Model(*TINY)
    small = emu.Plan(emu.Layout(tm, 1, 1), emu.Layout(tm, 2, 1))
    SB = big.alloc(0, fill=0x5A, guard=GUARD)
    fill_device(big, 0, SB, seed=31)
    SS = small.alloc(0, fill=0x5A, guard=GUARD)
    os_ = o_layout(small.src)
    upload_shards(oracle.shard(full_model(os_.model, 32), os_), SS)
    torch.cuda.synchronize()
    _pair(big, SB, "1B, first call (tables copied in)")
    D = _pair(small, SS, "tiny, second call with a smaller plan")
    check_reshard(small, SS, D, label="tiny via emu_reshard_noalloc")
    _pair(big, SB, "1B again, after the tiny plan replaced its tables")
    _pair(big, SB, "1B repeated, tables resident")


def test_noalloc_in_a_hip_graph(gpu_lib):
    """Tables made resident by an eager call, then the call captured in a HIP graph; every replay, on new
    source contents written eagerly between replays, equals emu_reshard's eager result."""
    import torch

    tm = emu.Model(*TINY)
    plan = emu.Plan(emu.Layout(tm, 1, 1), emu.Layout(tm, 2, 1))
    ws = plan.workspace()
    S = plan.alloc(0, fill=0x5A, guard=GUARD)
    D, ref = plan.alloc(1, fill=0xA5, guard=GUARD), plan.alloc(1, fill=0xA5, guard=GUARD)
    plan.reshard_noalloc(S.ptrs, D.ptrs)
    torch.cuda.synchronize()
    stream = torch.cuda.Stream()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        plan.reshard_noalloc(S.ptrs, D.ptrs)
    os_ = o_layout(plan.src)
    for replay, seed in enumerate((41, 42, 43)):
        upload_shards(oracle.shard(full_model(os_.model, seed), os_), S)
        for t in D.tensors:
            t.fill_(replay + 1)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        plan.reshard(ws, S.ptrs, ref.ptrs)
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(zip(ref.bufs, D.bufs)):
            assert torch.equal(a, b), f"graph replay {replay}: rank buffer {i} differs"
    check_reshard(plan, S, D, label="tiny, last graph replay")
    del graph
