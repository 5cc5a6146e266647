"""GPU parity on provenance tags: every source element carries its own logical id + 1, so any misrouted,
duplicated, dropped or replica-sourced element shows in the output, which random weights (where equal
values are common in bf16) could hide.

* source tags: id + 1 of the element's logical coordinate; a replica of an element already held by an
  earlier rank (norms on TP ranks > 0, KV heads replicated past their first rank) carries the tag with its
  top bit set, and source pad rows carry an all-ones sentinel: neither may ever reach the output;
* expected destination: id + 1 everywhere, zero in destination pad rows;
* buckets: each destination rank's tags concatenated and cut every B bytes, from pack and from the fused
  source -> bucket plan; unpack restores the destination tensors;
* every call leaves its inputs' allocations byte-identical and the bytes around its outputs' views
  (alignment gaps, guard bands, short buckets' tails) at their prefill.

Micro-model layouts, in bf16 (16-bit tags; the models have fewer than 2^15 elements) and fp32 (32-bit tags).
"""
import itertools
import random

import numpy as np
import pytest

import oracle
from oracle import coords
from paper_2609_34645_amd import emu
from tests.gpu_util import Guard, o_layout, say, upload_shards
from tests.shapes import MICRO, MICRO_KV

pytestmark = pytest.mark.gpu

GUARD = 48  # bytes of prefilled guard band around every tensor and bucket view
FORMATS = [("interleaved", "block"), ("separate", "separate"), ("interleaved", "separate"), ("separate", "block")]
TAG = {"bf16": (np.uint16, 0x8000, 0xFFFF), "fp32": (np.uint32, 0x8000_0000, 0xFFFF_FFFF)}
_CACHE = {}


def tags(lay, source):
    """Per rank, per tensor: the tag array of layout `lay` (an emu.Layout), as a source or as the
    expected destination."""
    key = (lay, source)
    if key not in _CACHE:
        ol = o_layout(lay)
        dt, rep_bit, sentinel = TAG[lay.dtype]
        seen, out = set(), []
        for specs, per in zip(oracle.rank_inventory(ol), coords.element_ids(ol)):
            rank = []
            for s, ids in zip(specs, per):
                a = np.array(ids, dtype=np.int64)
                assert a.max() + 1 < rep_bit
                if source:
                    t = np.where(a < 0, sentinel, a + 1)
                    rep = np.array([x >= 0 and x in seen for x in ids], dtype=bool)
                    t = np.where(rep, t | rep_bit, t)
                    seen.update(x for x in ids if x >= 0)
                else:
                    t = np.where(a < 0, 0, a + 1)
                rank.append(t.astype(dt).reshape(s.shape))
            out.append(rank)
        _CACHE[key] = out
    return _CACHE[key]


def host_bytes(t):
    return t.cpu().numpy().view(np.uint8)


def run_tagged(src, dst, B):
    import torch

    plan = emu.Plan(src, dst)
    ws = plan.workspace()
    S, D = plan.alloc(0, fill=0x5A, guard=GUARD), plan.alloc(1, fill=0xA5, guard=GUARD)
    upload_shards(tags(src, True), S, tweak_replicas=False)
    label = f"{src} -> {dst}"

    def guarded(call, keep, fills, what):
        g = Guard(keep=keep, fills=fills, label=f"{label}: {what}")
        call()
        torch.cuda.synchronize()
        g.check()

    guarded(lambda: plan.reshard(ws, S.ptrs, D.ptrs), S.tensors, [(D.tensors, 0xA5)], "reshard")
    want = tags(dst, False)
    flat = [a for rank in want for a in rank]
    for i, (t, w) in enumerate(zip(D.tensors, flat)):
        assert np.array_equal(host_bytes(t), w.reshape(-1).view(np.uint8)), f"{label}: destination tensor {i}"
    # buckets: each rank's stream cut every B bytes, from pack and from the fused plan
    streams = [np.concatenate([a.reshape(-1).view(np.uint8) for a in rank]) for rank in want]
    expect = [s[k:k + B] for s in streams for k in range(0, len(s), B)]
    bufs, bptrs = plan.alloc_buckets(1, B, fill=0x77, guard=GUARD)
    guarded(lambda: plan.pack(ws, 1, B, D.ptrs, bptrs), D.tensors, [(bufs, 0x77)], f"pack B={B}")
    R = plan.alloc(1, fill=0x11, guard=GUARD)
    guarded(lambda: plan.unpack(ws, 1, B, bptrs, R.ptrs), bufs, [(R.tensors, 0x11)], f"unpack B={B}")
    fused = emu.Plan(src, dst, bucket_bytes=B)
    fws = fused.workspace()
    fbufs, fbptrs = plan.alloc_buckets(1, B, fill=0x33, guard=GUARD)
    guarded(lambda: fused.reshard(fws, S.ptrs, fbptrs), S.tensors, [(fbufs, 0x33)], f"fused B={B}")
    assert len(bufs) == len(expect) == len(fbufs)
    for k, (b, f, e) in enumerate(zip(bufs, fbufs, expect)):
        assert np.array_equal(host_bytes(b), e), f"{label}: bucket {k} (B={B})"
        assert np.array_equal(host_bytes(f), e), f"{label}: fused bucket {k} (B={B})"
    for i, (x, y) in enumerate(zip(D.tensors, R.tensors)):
        assert torch.equal(x, y), f"{label}: unpacked tensor {i}"


def layouts(shape, dtype, tps, pps, pads):
    m = emu.Model(*shape)
    return [emu.Layout(m, tp, pp, pad, dtype, q, g)
            for tp, pp, pad, (q, g) in itertools.product(tps, pps, pads, FORMATS)
            if emu.layout_check(emu.Layout(m, tp, pp, pad, dtype, q, g)) == 0]


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_provenance_tags_micro(gpu_lib, dtype):
    """Every micro layout (TP 1/2/4 x PP 1/2/4 x pad 0/2 x four format pairs) as a source, each with three
    destinations, with a bucket size that is a random multiple of the element size."""
    rng = random.Random(3 if dtype == "bf16" else 4)
    lays = layouts(MICRO, dtype, (1, 2, 4), (1, 2, 4), (0, 2))
    es = 2 if dtype == "bf16" else 4
    n = 0
    for i, src in enumerate(lays):
        for dst in (lays[(i * 7 + 1) % len(lays)], lays[(i * 13 + 5) % len(lays)], rng.choice(lays)):
            run_tagged(src, dst, es * rng.randint(1, 300))
            n += 1
    say(f"  {n} tagged {dtype} layout pairs exact")


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_provenance_tags_kv_replication_uneven_pp(gpu_lib, dtype):
    """TP up to 8 over 2 KV heads (KV heads replicated), PP 1/2/3 over 3 layers (uneven stages): replicas
    and pad rows must never reach the output."""
    rng = random.Random(5 if dtype == "bf16" else 6)
    lays = layouts(MICRO_KV, dtype, (1, 2, 4, 8), (1, 2, 3), (0, 2))
    es = 2 if dtype == "bf16" else 4
    n = 0
    for i, src in enumerate(lays):
        for dst in (lays[(i * 5 + 3) % len(lays)], rng.choice(lays)):
            run_tagged(src, dst, es * rng.randint(1, 300))
            n += 1
    say(f"  {n} tagged {dtype} KV-replication / uneven-PP pairs exact")
