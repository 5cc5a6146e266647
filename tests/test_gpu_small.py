"""GPU parity on small models: every output byte compared with the oracle on the same seeded inputs.

Covers the micro models (which also exercise the byte-granular path: 8-byte o/down runs at TP4), the
tiny 2-layer decoder's Split TP1 PP1 -> TP2 PP1 and Merge back, the tiny transition captured in a HIP
graph and replayed, format changes, padded vocabularies with zero-filled destination pad rows, every
launch option, and bucket pack/unpack at awkward bucket sizes (including sizes that put source and
bucket bytes at different 16-byte phases).
"""
import ctypes
import itertools

import numpy as np
import pytest

import oracle
from paper_2609_34645_amd import emu
from tests.gpu_util import (Guard, check_buckets, check_reshard, check_upload, fill_device, full_model, host_view,
                             o_layout, say, upload_shards)
from tests.shapes import MICRO, MICRO8, MICRO_KV, TINY

pytestmark = pytest.mark.gpu

FORMATS = [("interleaved", "block"), ("separate", "separate"), ("interleaved", "separate")]


GUARD = 48  # bytes of prefilled guard band around every tensor and bucket view


def run_pair(src, dst, seed=5, options=None, bucket_sizes=(), fused=False, receiver_bucket=0):
    """Reshard (and pack / unpack / fused plan / receiver plan) one layout pair on seeded oracle shards;
    every output byte against the oracle, and every call's write footprint checked (Guard). With
    receiver_bucket, the source set is packed into buckets of that size and the receiver plan
    (emu_plan_from_buckets) must rebuild the destination set from them."""
    import torch

    for k, v in (options or {}).items():
        emu.set_option(k, v)
    plan = emu.Plan(src, dst)
    os_ = o_layout(src)
    ws = plan.workspace()
    S = plan.alloc(0, fill=0x5A, guard=GUARD)
    D = plan.alloc(1, fill=0xA5, guard=GUARD)
    plan.check_tables(S.ptrs, D.ptrs)
    upload_shards(oracle.shard(full_model(os_.model, seed, src.dtype), os_), S, tp=src.tp)
    label = f"{src.tp}x{src.pp}->{dst.tp}x{dst.pp}"
    g = Guard(keep=S.tensors, fills=[(D.tensors, 0xA5)], label=f"reshard {label}")
    plan.reshard(ws, S.ptrs, D.ptrs)
    torch.cuda.synchronize()
    g.check()
    check_reshard(plan, S, D, label=label)
    for B in bucket_sizes:
        bufs, bptrs = plan.alloc_buckets(1, B, fill=0x77, guard=GUARD)
        plan.check_bucket_tables(1, B, D.ptrs, bptrs)
        g = Guard(keep=D.tensors, fills=[(bufs, 0x77)], label=f"pack B={B} {label}")
        plan.pack(ws, 1, B, D.ptrs, bptrs)
        torch.cuda.synchronize()
        g.check()
        R = plan.alloc(1, fill=0x11, guard=GUARD)
        g = Guard(keep=bufs, fills=[(R.tensors, 0x11)], label=f"unpack B={B} {label}")
        plan.unpack(ws, 1, B, bptrs, R.ptrs)
        torch.cuda.synchronize()
        g.check()
        dd = plan.tensors(1)
        ranks = {}
        for i, d in enumerate(dd):
            ranks.setdefault(d["rank"], []).append(host_view(D.tensors[i], d, dst.dtype))
        check_buckets(plan, 1, B, [ranks[r] for r in sorted(ranks)], bufs, label=f"B={B}")
        for a, b in zip(D.tensors, R.tensors):
            assert torch.equal(a, b)
        if fused:  # source shards straight into buckets: the same buckets as reshard + pack
            fp = emu.Plan(src, dst, bucket_bytes=B)
            fws = fp.workspace()
            fbufs, fbptrs = plan.alloc_buckets(1, B, fill=0x33, guard=GUARD)
            fp.check_tables(S.ptrs, fbptrs)
            g = Guard(keep=S.tensors, fills=[(fbufs, 0x33)], label=f"fused B={B} {label}")
            fp.reshard(fws, S.ptrs, fbptrs)
            torch.cuda.synchronize()
            g.check()
            for k, (a, b) in enumerate(zip(bufs, fbufs)):
                assert torch.equal(a, b), f"fused bucket {k} differs (B={B})"
    if receiver_bucket:
        Bs = receiver_bucket
        sbufs, sbptrs = plan.alloc_buckets(0, Bs, fill=0x44, guard=GUARD)
        g = Guard(keep=S.tensors, fills=[(sbufs, 0x44)], label=f"pack source Bs={Bs} {label}")
        plan.pack(ws, 0, Bs, S.ptrs, sbptrs)
        torch.cuda.synchronize()
        g.check()
        rp = emu.Plan(src, dst, src_bucket_bytes=Bs)
        rws = rp.workspace()
        R2 = rp.alloc(1, fill=0x66, guard=GUARD)
        rp.check_tables(sbptrs, R2.ptrs)
        g = Guard(keep=sbufs, fills=[(R2.tensors, 0x66)], label=f"receiver Bs={Bs} {label}")
        rp.reshard(rws, sbptrs, R2.ptrs)
        torch.cuda.synchronize()
        g.check()
        for i, (a, b) in enumerate(zip(D.tensors, R2.tensors)):
            assert torch.equal(a, b), f"receiver plan (Bs={Bs}): tensor {i} differs"
    return plan


def micro_pairs(shape, dtype):
    m = emu.Model(*shape)
    lays = [emu.Layout(m, tp, pp, pad, dtype, q, g) for tp, pp, pad, (q, g) in
            itertools.product((1, 2, 4), (1, 2, 4), (0, 2), FORMATS)]
    return lays


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_micro_pairs(gpu_lib, dtype):
    lays = micro_pairs(MICRO, dtype)
    n = 0
    for i, src in enumerate(lays):
        for dst in lays[i % 5::5]:
            run_pair(src, dst, seed=i)
            n += 1
    say(f"  {n} micro layout pairs bit-exact ({dtype})")


def random_valid_layout(rng, model, dtype):
    while True:
        L = model.num_layers
        lay = emu.Layout(model, rng.choice([1, 1, 2, 2, 3, 4, 8]), rng.randint(1, L), rng.choice([0, 0, 1, 2, 3]),
                         dtype, rng.choice(["interleaved", "separate"]), rng.choice(["block", "separate"]))
        if emu.layout_check(lay) == 0:
            return lay


@pytest.mark.parametrize("row_wrap", [1, 0], ids=["row_wrap", "whole_rows"])
def test_random_layout_pairs(gpu_lib, row_wrap):
    """400 random valid layout pairs on random small models, each with a random bucket size: reshard,
    pack and unpack bit-exact against the oracle, the fused source -> bucket plan giving the same
    buckets, and the receiver plan rebuilding the destination set from the source set's buckets (of
    another size). Of the 400: 206 have byte-granular segments (odd widths
    put runs at every 16-byte phase), 203 convert between fp32 and bf16, 133 zero-fill pad rows, 177
    replicate KV heads and 141 have uneven pipeline stages. Run once with row-wrapping tiles for 2D
    segments (the default) and once with whole-row tiles and row slices."""
    import random

    old = emu.get_option(emu.OPT_ROW_WRAP)
    emu.set_option(emu.OPT_ROW_WRAP, row_wrap)
    try:
        _random_pairs(random.Random(41))
    finally:
        emu.set_option(emu.OPT_ROW_WRAP, old)


def _random_pairs(rng):
    n = 0
    while n < 400:
        nH = rng.choice([2, 4, 8])
        G = rng.choice([g for g in (1, 2, 4) if nH % g == 0])
        model = emu.Model(rng.randint(1, 5), rng.choice([8, 12, 16, 24]), nH, rng.choice([2, 4, 6]), G,
                          rng.choice([8, 16, 24]), rng.choice([8 * rng.randint(1, 5), rng.randint(6, 40)]))
        src = random_valid_layout(rng, model, rng.choice(["bf16", "fp32"]))
        dst = random_valid_layout(rng, model, rng.choice(["bf16", "fp32"]))
        es = 2 if dst.dtype == "bf16" else 4
        ess = 2 if src.dtype == "bf16" else 4  # the receiver's bucket size, from the pair index: same pairs
        run_pair(src, dst, seed=n, bucket_sizes=(es * rng.randint(1, 700),), fused=True,
                 receiver_bucket=ess * (1 + n * 7919 % 700))
        n += 1
    say(f"  {n} random layout pairs bit-exact")


def test_micro_general_path_is_exercised(gpu_lib):
    m = emu.Model(*MICRO)
    plan = emu.Plan(emu.Layout(m, 1, 1), emu.Layout(m, 4, 1))
    assert plan.info["n_general_segments"] > 0


def test_t_sub_paper_example_micro8(gpu_lib):
    """Section 6.1: (TP4, PP8) split to (TP4, PP2) units, merged into (TP8, PP2): two launches through the
    intermediate layout give the direct result, on the GPU."""
    import torch

    m = emu.Model(*MICRO8)
    a, b, c = emu.Layout(m, 4, 8), emu.Layout(m, 4, 2), emu.Layout(m, 8, 2)
    pab, pbc, pac = emu.Plan(a, b), emu.Plan(b, c), emu.Plan(a, c)
    wab, wbc, wac = pab.workspace(), pbc.workspace(), pac.workspace()
    A = pab.alloc(0, fill=0x5A, guard=GUARD)
    upload_shards(oracle.shard(full_model(o_layout(a).model, 3), o_layout(a)), A, tp=4)
    B, C1, C2 = (pab.alloc(1, fill=0xA5, guard=GUARD), pbc.alloc(1, fill=0xA5, guard=GUARD),
                 pac.alloc(1, fill=0xA5, guard=GUARD))
    for p, w, x, y in ((pab, wab, A, B), (pbc, wbc, B, C1), (pac, wac, A, C2)):
        g = Guard(keep=x.tensors, fills=[(y.tensors, 0xA5)], label="T_sub route")
        p.reshard(w, x.ptrs, y.ptrs)
        torch.cuda.synchronize()
        g.check()
    for x, y in zip(C1.tensors, C2.tensors):
        assert torch.equal(x, y)
    check_reshard(pac, A, C2, label="TP4PP8->TP8PP2")


def test_tiny_split_and_merge_back(gpu_lib):
    """The tiny decoder: Split TP1 PP1 -> TP2 PP1, then Merge back; the round trip is the identity."""
    import torch

    m = emu.Model(*TINY)
    a, b = emu.Layout(m, 1, 1), emu.Layout(m, 2, 1)
    fwd, back = emu.Plan(a, b), emu.Plan(b, a)
    assert fwd.info["bytes_read"] == 3_953_664 and back.info["bytes_read"] == 3_951_104
    wf, wb = fwd.workspace(), back.workspace()
    A = fwd.alloc(0, fill=0x5A, guard=GUARD)
    upload_shards(oracle.shard(full_model(o_layout(a).model, 1), o_layout(a)), A)
    B, A2 = fwd.alloc(1, fill=0xA5, guard=GUARD), back.alloc(1, fill=0xA5, guard=GUARD)
    for p, w, x, y in ((fwd, wf, A, B), (back, wb, B, A2)):
        g = Guard(keep=x.tensors, fills=[(y.tensors, 0xA5)], label="tiny split / merge")
        p.reshard(w, x.ptrs, y.ptrs)
        torch.cuda.synchronize()
        g.check()
    check_reshard(fwd, A, B, label="tiny TP1->TP2")
    check_reshard(back, B, A2, label="tiny TP2->TP1")
    for x, y in zip(A.tensors, A2.tensors):
        assert torch.equal(x, y)


def test_tiny_transition_in_a_hip_graph(gpu_lib):
    """The library only enqueues kernels on the caller's stream (no allocation, no synchronisation), so
    reshard + pack + unpack of the tiny decoder can be captured once in a HIP graph and replayed. Each
    replay runs on new source contents written eagerly between replays, and its destination tensors,
    buckets and unpacked tensors are checked against the oracle."""
    import torch

    m = emu.Model(*TINY)
    a, b = emu.Layout(m, 1, 1), emu.Layout(m, 2, 1)
    plan = emu.Plan(a, b)
    ws = plan.workspace()
    B = 1 << 16
    S = plan.alloc(0, fill=0x3C, guard=GUARD)
    D, R = plan.alloc(1, fill=0xA5, guard=GUARD), plan.alloc(1, fill=0x5A, guard=GUARD)
    bufs, bptrs = plan.alloc_buckets(1, B, fill=0x77, guard=GUARD)
    torch.cuda.synchronize()
    stream = torch.cuda.Stream()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        plan.reshard(ws, S.ptrs, D.ptrs)
        plan.pack(ws, 1, B, D.ptrs, bptrs)
        plan.unpack(ws, 1, B, bptrs, R.ptrs)
    oa, ob = o_layout(a), o_layout(b)
    for replay, seed in enumerate((21, 22, 23)):
        upload_shards(oracle.shard(full_model(oa.model, seed), oa), S)
        for t in D.bufs + R.bufs:
            t.fill_(replay + 1)
        torch.cuda.synchronize()
        g = Guard(keep=S.tensors, fills=[(D.tensors, replay + 1), (bufs, 0x77), (R.tensors, replay + 1)],
                  label=f"graph replay {replay}")
        graph.replay()
        torch.cuda.synchronize()
        g.check()
        check_reshard(plan, S, D, label=f"graph replay {replay}")
        dd = plan.tensors(1)
        ranks = {}
        for i, d in enumerate(dd):
            ranks.setdefault(d["rank"], []).append(host_view(D.tensors[i], d, "bf16"))
        check_buckets(plan, 1, B, [ranks[r] for r in sorted(ranks)], bufs, label=f"graph replay {replay}")
        for x, y in zip(D.tensors, R.tensors):
            assert torch.equal(x, y), f"graph replay {replay}: unpacked tensors differ"
    del graph


@pytest.mark.parametrize("opts", [
    {emu.OPT_TILE_VECS: 8}, {emu.OPT_TILE_VECS: 16}, {emu.OPT_XCD_REMAP: 1},
    {emu.OPT_BUCKET_WG_PER_CU: 1}, {emu.OPT_TILE_VECS: 16, emu.OPT_XCD_REMAP: 1}, {emu.OPT_BUCKET_TILES: 1},
    {emu.OPT_NONTEMPORAL: 0}, {emu.OPT_LDS_STAGING: 1}, {emu.OPT_LDS_STAGING: 1, emu.OPT_TILE_VECS: 16},
    {emu.OPT_TILE_VECS: 1}, {emu.OPT_TILE_VECS: 2, emu.OPT_WG_PER_CU: 6}, {emu.OPT_WG_PER_CU: 0},
    {emu.OPT_WG_PER_CU: 1, emu.OPT_LDS_STAGING: 1}, {emu.OPT_WG_PER_CU: 8, emu.OPT_BUCKET_TILES: 0},
    {emu.OPT_WG_PER_CU: 12}, {emu.OPT_WG_PER_CU: 24, emu.OPT_TILE_VECS: 2},
    {emu.OPT_WG_PER_CU: 32, emu.OPT_TILE_VECS: 1}, {emu.OPT_TILE_VECS: 4, emu.OPT_LDS_STAGING: 1},
    {emu.OPT_ROW_WRAP: 0}, {emu.OPT_ROW_WRAP: 0, emu.OPT_TILE_VECS: 1}, {emu.OPT_ROW_WRAP: 0, emu.OPT_TILE_VECS: 16},
])
def test_launch_options(gpu_lib, opts):
    defaults = {k: emu.get_option(k) for k in range(8)}
    try:
        m = emu.Model(*TINY)
        run_pair(emu.Layout(m, 2, 2, 128), emu.Layout(m, 1, 1, 0, "bf16", "separate", "separate"), options=opts)
        mm = emu.Model(*MICRO)
        run_pair(emu.Layout(mm, 1, 2), emu.Layout(mm, 4, 1, 2), options=opts)
    finally:
        for k, v in defaults.items():
            emu.set_option(k, v)


def test_padded_vocab_zero_fill_and_source_pad_not_read(gpu_lib):
    """Reverse of the padded case: destination pad rows are zeros although the destination buffer was
    prefilled with a sentinel; source pad rows (filled with garbage) never reach the destination."""
    import torch

    m = emu.Model(2, 256, 4, 64, 2, 688, 1000)
    a, b = emu.Layout(m, 2, 1, 0), emu.Layout(m, 2, 2, 128)
    p = emu.Plan(a, b)
    assert p.info["zero_fill_bytes"] == 2 * 24 * 256 * 2
    ws = p.workspace()
    S = p.alloc(0, fill=0x5A, guard=GUARD)
    upload_shards(oracle.shard(full_model(o_layout(a).model, 9), o_layout(a)), S, tp=2)
    D = p.alloc(1, fill=0xA5, guard=GUARD)
    g = Guard(keep=S.tensors, fills=[(D.tensors, 0xA5)], label="pad 0 -> pad 128")
    p.reshard(ws, S.ptrs, D.ptrs)
    torch.cuda.synchronize()
    g.check()
    check_reshard(p, S, D, label="pad 0 -> pad 128")
    back = emu.Plan(b, a)
    wb = back.workspace()
    for t, d in zip(D.tensors, back.tensors(0)):
        if d["kind"] in ("embed", "lm_head") and d["rank"] % 2 == 1:
            t.view(-1)[-24 * 256 * 2:] = 0xEE      # garbage in the source pad rows
    A2 = back.alloc(1, fill=0xA5, guard=GUARD)
    g = Guard(keep=D.tensors, fills=[(A2.tensors, 0xA5)], label="pad 128 -> pad 0")
    back.reshard(wb, D.ptrs, A2.ptrs)
    torch.cuda.synchronize()
    g.check()
    check_reshard(back, D, A2, label="pad 128 -> pad 0")
    for x, y, d in zip(S.tensors, A2.tensors, p.tensors(0)):
        if not (d["kind"].endswith("norm") and d["rank"] % 2):   # TP-rank-1 replicas were altered on upload
            assert torch.equal(x, y)


@pytest.mark.parametrize("tiles", [0, 1], ids=["persistent", "tile_per_wg"])
@pytest.mark.parametrize("B", [30, 1000, 4094, 65536, 65538, 1 << 20, 1 << 26])
def test_buckets_awkward_sizes(gpu_lib, B, tiles):
    m = emu.Model(*TINY)
    old = emu.get_option(emu.OPT_BUCKET_TILES)
    emu.set_option(emu.OPT_BUCKET_TILES, tiles)
    try:
        run_pair(emu.Layout(m, 1, 1), emu.Layout(m, 2, 1), bucket_sizes=(B,))
        run_pair(emu.Layout(m, 2, 2, 128), emu.Layout(m, 1, 2, 0, "bf16", "separate", "block"), bucket_sizes=(B,))
    finally:
        emu.set_option(emu.OPT_BUCKET_TILES, old)


@pytest.mark.parametrize("tiles", [1, 0])
def test_buckets_of_one_element(gpu_lib, tiles):
    """The smallest legal bucket, one bf16 element (2 bytes): every tensor boundary and every byte pair
    is its own piece: 1,680 buckets per rank of the micro model. Buckets larger than a whole rank
    stream (one short bucket per rank) are covered by the 2^26-byte case above."""
    m = emu.Model(*MICRO)
    old = emu.get_option(emu.OPT_BUCKET_TILES)
    emu.set_option(emu.OPT_BUCKET_TILES, tiles)
    try:
        run_pair(emu.Layout(m, 2, 2, 2), emu.Layout(m, 4, 1, 2), bucket_sizes=(2, 6))
    finally:
        emu.set_option(emu.OPT_BUCKET_TILES, old)


@pytest.mark.parametrize("tiles", [1, 0], ids=["tile_per_wg", "persistent"])
def test_buckets_beyond_128_ranks(gpu_lib, tiles):
    """256 destination ranks (TP16 PP16): ranks past the first 128 find their first bucket with the
    on-device wave64 reduction instead of the host's kernel argument, and odd bucket sizes give the
    ranks different bucket counts; the fused plan must produce the same buckets."""
    m = emu.Model(16, 32, 16, 2, 16, 32, 32)
    old = emu.get_option(emu.OPT_BUCKET_TILES)
    emu.set_option(emu.OPT_BUCKET_TILES, tiles)
    try:
        plan = run_pair(emu.Layout(m, 1, 1), emu.Layout(m, 16, 16), bucket_sizes=(6, 64, 1000), fused=True)
        assert plan.info["n_dst_ranks"] == 256
    finally:
        emu.set_option(emu.OPT_BUCKET_TILES, old)


def test_buckets_source_side_and_fp32(gpu_lib):
    import torch

    m = emu.Model(*TINY)
    a, b = emu.Layout(m, 2, 2, 0, "fp32"), emu.Layout(m, 1, 1, 0, "fp32")
    p = emu.Plan(a, b)
    ws = p.workspace()
    S = p.alloc(0, fill=0x5A, guard=GUARD)
    upload_shards(oracle.shard(full_model(o_layout(a).model, 4, "fp32"), o_layout(a)), S, tp=2)
    for B in (4, 1 << 16, 12345 * 4):
        bufs, bptrs = p.alloc_buckets(0, B, fill=0x77, guard=GUARD)
        g = Guard(keep=S.tensors, fills=[(bufs, 0x77)], label=f"source-side pack B={B}")
        p.pack(ws, 0, B, S.ptrs, bptrs)
        torch.cuda.synchronize()
        g.check()
        R = p.alloc(0, fill=0, guard=GUARD)
        g = Guard(keep=bufs, fills=[(R.tensors, 0)], label=f"source-side unpack B={B}")
        p.unpack(ws, 0, B, bptrs, R.ptrs)
        torch.cuda.synchronize()
        g.check()
        sd = p.tensors(0)
        ranks = {}
        for i, d in enumerate(sd):
            ranks.setdefault(d["rank"], []).append(host_view(S.tensors[i], d, "fp32"))
        check_buckets(p, 0, B, [ranks[r] for r in sorted(ranks)], bufs, label=f"src side B={B}")
        for x, y in zip(S.tensors, R.tensors):
            assert torch.equal(x, y)


def test_execute_errors(gpu_lib):
    import torch

    m = emu.Model(*TINY)
    p = emu.Plan(emu.Layout(m, 1, 1), emu.Layout(m, 2, 1))
    ws = p.workspace()
    S, D = p.alloc(0), p.alloc(1)
    small = torch.empty(256, dtype=torch.uint8, device="cuda")
    with pytest.raises(emu.EmuError) as e:
        p.upload(small)
    assert e.value.code == -5
    off = torch.empty(p.info["workspace_bytes"] + 512, dtype=torch.uint8, device="cuda")[16:]
    with pytest.raises(emu.EmuError) as e:
        p.reshard(off, S.ptrs, D.ptrs)
    assert e.value.code == -5
    with pytest.raises(emu.EmuError) as e:
        p.pack(ws, 1, 3, D.ptrs, D.ptrs)
    assert e.value.code == -6
    with pytest.raises(emu.EmuError) as e:
        emu.ptr_table([S.bufs[0][1:]])
    assert e.value.code == -7
    # workspace registry: refused on the host, before anything is launched -- by the binding, which
    # accepts only workspaces the plan uploaded to (and keeps alive), and by the library itself
    fresh = torch.empty(p.info["workspace_bytes"], dtype=torch.uint8, device="cuda")
    with pytest.raises(emu.EmuError) as e:
        p.reshard(fresh, S.ptrs, D.ptrs)                  # never uploaded
    assert e.value.code == -5 and "Plan.upload" in str(e.value)
    lib = emu.load()
    V = ctypes.c_void_p
    assert lib.emu_reshard(p._h, V(fresh.data_ptr()), V(S.ptrs.data_ptr()), V(D.ptrs.data_ptr()), None) == -5
    assert b"emu_plan_upload" in lib.emu_last_error()
    assert lib.emu_reshard(p._h, V(off.data_ptr()), V(S.ptrs.data_ptr()), V(D.ptrs.data_ptr()), None) == -5
    assert b"aligned" in lib.emu_last_error()
    _, fresh_bptrs = p.alloc_buckets(1, 1 << 16)
    with pytest.raises(emu.EmuError) as e:
        p.pack(fresh, 1, 1 << 16, D.ptrs, fresh_bptrs)
    assert e.value.code == -5
    with pytest.raises(ValueError):
        p.pack(ws, 1, 1 << 16, D.ptrs, D.ptrs)            # a table of the wrong length, refused on the host
    with pytest.raises(ValueError):
        p.reshard(ws, S.ptrs[:-1], D.ptrs)
    q = emu.Plan(emu.Layout(m, 2, 1), emu.Layout(m, 1, 1))
    assert q.info["workspace_bytes"] <= ws.numel()
    q.upload(ws)                                          # another plan's tables now fill p's workspace
    with pytest.raises(emu.EmuError) as e:
        p.reshard(ws, S.ptrs, D.ptrs)
    assert e.value.code == -5
    p.upload(ws)
    p.reshard(ws, S.ptrs, D.ptrs)                         # accepted again after p's own upload
    torch.cuda.synchronize()


def test_pending_hip_error_is_not_reported(gpu_lib):
    """An error that an earlier HIP call left pending on the thread (hipSetDevice of a device that does
    not exist) is not reported by reshard, pack or unpack, which run, return EMU_OK and match the oracle."""
    import ctypes

    import torch

    hip = ctypes.CDLL("libamdhip64.so.7")  # the runtime that torch and the library already share
    bad = torch.cuda.device_count() + 1000

    def leave_error():
        assert hip.hipSetDevice(ctypes.c_int(bad)) != 0
        assert hip.hipPeekAtLastError() != 0

    m = emu.Model(*TINY)
    src, dst = emu.Layout(m, 1, 1), emu.Layout(m, 2, 1)
    plan = emu.Plan(src, dst)
    ws = plan.workspace()
    S, D = plan.alloc(0, fill=0x5A, guard=GUARD), plan.alloc(1, fill=0xA5, guard=GUARD)
    os_ = o_layout(src)
    upload_shards(oracle.shard(full_model(os_.model, 9, "bf16"), os_), S, tp=1)
    torch.cuda.synchronize()
    g = Guard(keep=S.tensors, fills=[(D.tensors, 0xA5)], label="reshard after a pending error")
    leave_error()
    plan.reshard(ws, S.ptrs, D.ptrs)
    assert hip.hipPeekAtLastError() == 0
    torch.cuda.synchronize()
    g.check()
    check_reshard(plan, S, D, label="after a pending error")
    B = 12288
    bufs, bptrs = plan.alloc_buckets(1, B, fill=0x77, guard=GUARD)
    R = plan.alloc(1, fill=0x11, guard=GUARD)
    g = Guard(keep=D.tensors, fills=[(bufs, 0x77)], label="pack after a pending error")
    leave_error()
    plan.pack(ws, 1, B, D.ptrs, bptrs)
    torch.cuda.synchronize()
    g.check()
    g = Guard(keep=bufs, fills=[(R.tensors, 0x11)], label="unpack after a pending error")
    leave_error()
    plan.unpack(ws, 1, B, bptrs, R.ptrs)
    assert hip.hipPeekAtLastError() == 0
    torch.cuda.synchronize()
    g.check()
    for a, b in zip(D.tensors, R.tensors):
        assert torch.equal(a, b)


@pytest.mark.parametrize("B", [64, 1000, 4094, 65536, 65538])
def test_fused_reshard_to_buckets(gpu_lib, B):
    """emu_plan_to_buckets: source shards straight into the destination ranks' buckets; the receiver
    unpacks with the ordinary plan. Buckets and unpacked tensors against the oracle."""
    import torch

    m = emu.Model(*TINY)
    pairs = [(emu.Layout(m, 1, 1), emu.Layout(m, 2, 1)),
             (emu.Layout(m, 2, 2, 128), emu.Layout(m, 1, 1, 0, "bf16", "separate", "separate")),
             (emu.Layout(m, 2, 1, 0, "fp32"), emu.Layout(m, 1, 2, 0, "fp32"))]
    for src, dst in pairs:
        if B % (2 if src.dtype == "bf16" else 4):
            continue
        fused, base = emu.Plan(src, dst, bucket_bytes=B), emu.Plan(src, dst)
        wf, wb = fused.workspace(), base.workspace()
        os_, od = o_layout(src), o_layout(dst)
        S = base.alloc(0, fill=0x5A, guard=GUARD)
        upload_shards(oracle.shard(full_model(os_.model, 8, src.dtype), os_), S, tp=src.tp)
        K = fused.alloc(1, fill=0x77, guard=GUARD)          # side 1 of the fused plan = the buckets
        g = Guard(keep=S.tensors, fills=[(K.tensors, 0x77)], label=f"fused B={B}")
        fused.reshard(wf, S.ptrs, K.ptrs)
        torch.cuda.synchronize()
        g.check()
        R = base.alloc(1, fill=0x11, guard=GUARD)
        g = Guard(keep=K.tensors, fills=[(R.tensors, 0x11)], label=f"unpack of fused buckets B={B}")
        base.unpack(wb, 1, B, K.ptrs, R.ptrs)
        torch.cuda.synchronize()
        g.check()
        sd = base.tensors(0)
        ranks_src = {}
        for i, d in enumerate(sd):
            ranks_src.setdefault(d["rank"], []).append(host_view(S.tensors[i], d, src.dtype))
        want = oracle.reshard([ranks_src[r] for r in sorted(ranks_src)], os_, od)
        check_buckets(fused, 1, B, want, K.tensors, label=f"fused B={B}")
        flat = [np.ascontiguousarray(a).reshape(-1).view(np.uint8) for rank in want for a in rank]
        for i, (t, w) in enumerate(zip(R.tensors, flat)):
            assert np.array_equal(t.cpu().numpy(), w), f"unpacked tensor {i}"


@pytest.mark.parametrize("pair", [("fp32", "bf16"), ("bf16", "fp32")])
def test_converting_reshard_small(gpu_lib, pair):
    a, b = pair
    mm = emu.Model(*MICRO)
    n = 0
    for tp_s, pp_s, tp_d, pp_d, pad in ((1, 1, 2, 1, 0), (4, 2, 1, 4, 2), (2, 4, 4, 1, 0), (1, 2, 4, 2, 2)):
        for q, g in FORMATS:
            run_pair(emu.Layout(mm, tp_s, pp_s, pad, a, q, g), emu.Layout(mm, tp_d, pp_d, pad, b, "separate", g),
                     seed=n)
            n += 1
    m = emu.Model(*TINY)
    run_pair(emu.Layout(m, 2, 2, 128, a), emu.Layout(m, 1, 1, 0, b), bucket_sizes=(65536, 4096 + 4))


@pytest.mark.parametrize("tile_vecs", [1, 2, 8, 16])
@pytest.mark.parametrize("pair", [("fp32", "bf16"), ("bf16", "fp32")])
def test_converting_tile_sizes(gpu_lib, pair, tile_vecs):
    """Converting plans at every tile size, row-wrapping tiles and whole-row tiles: fp32 -> bf16 tiles of
    more than 8 vectors per lane are moved in passes of 8."""
    a, b = pair
    old = {k: emu.get_option(k) for k in (emu.OPT_TILE_VECS, emu.OPT_ROW_WRAP)}
    m = emu.Model(*TINY)
    try:
        for wrap in (1, 0):
            run_pair(emu.Layout(m, 2, 2, 128, a), emu.Layout(m, 1, 1, 0, b, "separate", "separate"),
                     options={emu.OPT_TILE_VECS: tile_vecs, emu.OPT_ROW_WRAP: wrap})
            run_pair(emu.Layout(m, 1, 1, 0, a), emu.Layout(m, 2, 2, 0, b), options={emu.OPT_TILE_VECS: tile_vecs,
                                                                                  emu.OPT_ROW_WRAP: wrap})
    finally:
        for k, v in old.items():
            emu.set_option(k, v)


def test_fp32_to_bf16_special_values(gpu_lib):
    """Every fp32 bit pattern class through the kernel: NaNs with payloads in either half, infinities,
    denormals, ties, overflow to infinity -- against the oracle's round-to-nearest-even."""
    import torch

    m = emu.Model(*TINY)
    src, dst = emu.Layout(m, 1, 1, 0, "fp32"), emu.Layout(m, 2, 1, 0, "bf16")
    p = emu.Plan(src, dst)
    ws = p.workspace()
    S = p.alloc(0, fill=0x5A, guard=GUARD)
    rng = np.random.default_rng(77)
    specials = np.array([0x3F808000, 0x3F818000, 0x7F7F8000, 0x7F7FFFFF, 0x7F800000, 0xFF800000, 0x7FC00000,
                         0x7F800001, 0xFFA00000, 0x80000000, 0x00000001, 0x00008000, 0x00018000, 0x007FFFFF],
                        dtype=np.uint32)
    for t in S.tensors:
        u = rng.integers(0, 1 << 32, size=t.numel() // 4, dtype=np.uint64).astype(np.uint32)
        u[:specials.size] = specials[:u.size]
        t.copy_(torch.from_numpy(u.view(np.uint8)))
    D = p.alloc(1, fill=0xA5, guard=GUARD)
    g = Guard(keep=S.tensors, fills=[(D.tensors, 0xA5)], label="fp32 bit patterns -> bf16")
    p.reshard(ws, S.ptrs, D.ptrs)
    torch.cuda.synchronize()
    g.check()
    check_reshard(p, S, D, label="fp32 bit patterns -> bf16")


def test_kv_replication_and_uneven_pp_small(gpu_lib):
    m = emu.Model(3, 16, 8, 2, 2, 16, 16)
    lays = [emu.Layout(m, tp, pp, pad, "bf16", q, g) for tp, pp, pad, (q, g) in
            itertools.product((1, 2, 4, 8), (1, 2, 3), (0, 2), FORMATS[:2])]
    for i, src in enumerate(lays):
        for dst in lays[i % 6::6]:
            run_pair(src, dst, seed=i)


def _scattered(plan, side, rng, fill):
    """One side's tensors at shuffled positions of one buffer, each at a random 16-byte (not 256-byte)
    aligned offset: the ABI promises only 16-byte alignment."""
    import torch

    descs = plan.tensors(side)
    order = list(range(len(descs)))
    rng.shuffle(order)
    offs, pos = [0] * len(descs), 0
    for i in order:
        pos += 16 * rng.randint(1, 15)
        offs[i] = pos
        pos = (pos + descs[i]["bytes"] + 15) // 16 * 16
    buf = torch.full((pos + 256,), fill, dtype=torch.uint8, device="cuda")
    tensors = [buf[o:o + d["bytes"]] for o, d in zip(offs, descs)]
    return emu.ShardSet([buf], tensors, emu.ptr_table(tensors))


def _scattered_buckets(plan, side, B, rng, fill):
    import torch

    nranks = plan.info["n_src_ranks" if side == 0 else "n_dst_ranks"]
    sizes = []
    for r in range(nranks):
        nb, sb = plan.bucket_layout(side, B, r)
        sizes += [min(B, sb - k * B) for k in range(nb)]
    offs, pos = [], 0
    for n in sizes:
        pos += 16 * rng.randint(1, 15)
        offs.append(pos)
        pos = (pos + n + 15) // 16 * 16
    buf = torch.full((pos + 256,), fill, dtype=torch.uint8, device="cuda")
    bufs = [buf[o:o + n] for o, n in zip(offs, sizes)]
    return bufs, emu.ptr_table(bufs)


@pytest.mark.parametrize("pair", [("bf16", "bf16"), ("fp32", "bf16"), ("bf16", "fp32")])
def test_tensors_at_16_byte_offsets(gpu_lib, pair):
    """Source, destination and bucket buffers placed at shuffled, merely 16-byte aligned addresses: the
    reshard (plain and converting), pack, unpack and the fused plan against the oracle."""
    import random

    import torch

    rng = random.Random(17)
    m = emu.Model(*TINY)
    src = emu.Layout(m, 2, 2, 128, pair[0])
    dst = emu.Layout(m, 1, 1, 0, pair[1], "separate", "block")
    plan = emu.Plan(src, dst)
    ws = plan.workspace()
    S, D = _scattered(plan, 0, rng, 0x5A), _scattered(plan, 1, rng, 0xA5)
    plan.check_tables(S.ptrs, D.ptrs)
    os_ = o_layout(src)
    upload_shards(oracle.shard(full_model(os_.model, 23, src.dtype), os_), S, tp=src.tp)

    def guarded(call, keep, fills, label):
        g = Guard(keep=keep, fills=fills, label=f"16-byte offsets {pair}: {label}")
        call()
        torch.cuda.synchronize()
        g.check()

    guarded(lambda: plan.reshard(ws, S.ptrs, D.ptrs), S.tensors, [(D.tensors, 0xA5)], "reshard")
    check_reshard(plan, S, D, label=f"16-byte offsets {pair}")
    B = 6000 if pair[1] == "bf16" else 6004
    bufs, bptrs = _scattered_buckets(plan, 1, B, rng, 0x77)
    plan.check_bucket_tables(1, B, D.ptrs, bptrs)
    guarded(lambda: plan.pack(ws, 1, B, D.ptrs, bptrs), D.tensors, [(bufs, 0x77)], "pack")
    R = _scattered(plan, 1, rng, 0x11)
    guarded(lambda: plan.unpack(ws, 1, B, bptrs, R.ptrs), bufs, [(R.tensors, 0x11)], "unpack")
    fused = emu.Plan(src, dst, bucket_bytes=B)
    fws = fused.workspace()
    fbufs, fbptrs = _scattered_buckets(plan, 1, B, rng, 0x33)
    guarded(lambda: fused.reshard(fws, S.ptrs, fbptrs), S.tensors, [(fbufs, 0x33)], "fused")
    dd = plan.tensors(1)
    ranks = {}
    for i, d in enumerate(dd):
        ranks.setdefault(d["rank"], []).append(host_view(D.tensors[i], d, dst.dtype))
    check_buckets(plan, 1, B, [ranks[r] for r in sorted(ranks)], bufs, label=f"16-byte offsets B={B}")
    for k, (a, b) in enumerate(zip(bufs, fbufs)):
        assert torch.equal(a, b), f"fused bucket {k}"
    for i, (a, b) in enumerate(zip(D.tensors, R.tensors)):
        assert torch.equal(a, b), f"unpacked tensor {i}"


@pytest.mark.parametrize("case", ["tiny", "zero_fill", "fp32_to_bf16"])
def test_reshard_groups_small(gpu_lib, case):
    """emu_reshard_groups: three shard sets of one plan (different contents) in one launch give what
    three emu_reshard calls give, and each group's result matches the oracle; write footprints guarded."""
    import torch

    if case == "tiny":
        m = emu.Model(*TINY)
        src, dst = emu.Layout(m, 2, 2), emu.Layout(m, 1, 1, 0, "bf16", "separate", "block")
    elif case == "zero_fill":                       # destination pad rows: the zero-fill instance runs too
        m = emu.Model(2, 256, 4, 64, 2, 688, 1000)
        src, dst = emu.Layout(m, 2, 1, 0), emu.Layout(m, 2, 2, 128)
    else:
        m = emu.Model(*TINY)
        src, dst = emu.Layout(m, 1, 1, 0, "fp32"), emu.Layout(m, 2, 2, 0, "bf16")
    plan = emu.Plan(src, dst)
    ws = plan.workspace()
    os_ = o_layout(src)
    S = [plan.alloc(0, fill=0x5A, guard=GUARD) for _ in range(3)]
    for k, s in enumerate(S):
        upload_shards(oracle.shard(full_model(os_.model, 60 + k, src.dtype), os_), s, tp=src.tp)
    G = [plan.alloc(1, fill=0xA5, guard=GUARD) for _ in range(3)]
    ref = [plan.alloc(1, fill=0xA5, guard=GUARD) for _ in range(3)]
    torch.cuda.synchronize()
    g = Guard(keep=[t for s in S for t in s.tensors], fills=[(d.tensors, 0xA5) for d in G], label=f"groups {case}")
    plan.reshard_groups(ws, emu.group_tables(S), emu.group_tables(G))
    torch.cuda.synchronize()
    g.check()
    for s, r in zip(S, ref):
        plan.reshard(ws, s.ptrs, r.ptrs)
    torch.cuda.synchronize()
    for k in range(3):
        for i, (a, b) in enumerate(zip(G[k].bufs, ref[k].bufs)):
            assert torch.equal(a, b), f"{case}: group {k} rank buffer {i} differs from emu_reshard"
        check_reshard(plan, S[k], G[k], label=f"groups {case}, group {k}")
    rc = emu.load().emu_reshard_groups(plan._h, ctypes.c_void_p(ws.data_ptr()), 0,
                                       ctypes.c_void_p(S[0].ptrs.data_ptr()), ctypes.c_void_p(G[0].ptrs.data_ptr()), None)
    assert rc == -10                                   # no group: refused on the host


def test_alias_plans_small(gpu_lib):
    """Plans that leave already-resident shards out (EMU_PLAN_ALIAS_RESIDENT): the destination set takes
    the source tensors for its alias tensors and its own buffers for the rest; every destination tensor
    matches the oracle, the kernel touches nothing outside the non-alias views, and the source is
    unchanged. Micro layouts, PP-only and mixed changes."""
    import torch

    mm = emu.Model(*MICRO)
    pairs = [(emu.Layout(mm, 2, 4), emu.Layout(mm, 2, 1)), (emu.Layout(mm, 4, 2, 2), emu.Layout(mm, 4, 1, 2)),
             (emu.Layout(mm, 2, 2), emu.Layout(mm, 2, 1, 0, "bf16", "separate", "separate")),
             (emu.Layout(mm, 1, 2), emu.Layout(mm, 4, 1)), (emu.Layout(mm, 2, 2, 0, "fp32"), emu.Layout(mm, 1, 4, 0, "fp32"))]
    for src, dst in pairs:
        plan = emu.Plan(src, dst, alias=True)
        assert plan.info["n_alias_tensors"] > 0, (src, dst)
        ws = plan.workspace()
        os_ = o_layout(src)
        S = plan.alloc(0, fill=0x5A, guard=GUARD)
        upload_shards(oracle.shard(full_model(os_.model, 71, src.dtype), os_), S, tp=src.tp)
        D = plan.alloc(1, fill=0xA5, guard=GUARD, alias=S)
        own = [t for t, d in zip(D.tensors, plan.tensors(1)) if d["alias"] < 0]
        g = Guard(keep=S.tensors, fills=[(own, 0xA5)] if own else [], label=f"alias {src} -> {dst}")
        plan.reshard(ws, S.ptrs, D.ptrs)
        torch.cuda.synchronize()
        g.check()
        if not own:
            assert all(bool((b == 0xA5).all()) for b in D.bufs)
        check_reshard(plan, S, D, label=f"alias {src.tp}x{src.pp} -> {dst.tp}x{dst.pp}")


def test_uploaded_workspace_matches_host_image():
    """emu_plan_upload derives the reshard's tile map and each side's stream offsets, rank records and
    4 KB chunk map on the device: the uploaded workspace equals the host's image byte for byte, for sides
    that differ in rank and tensor counts, zero-filled pad rows (a second tile-map section), uneven PP with
    KV replication, and fused plans whose bucket sides hold 30-byte buckets (many tensors inside one chunk)
    or buckets ending off the chunk grid."""
    m, mk = emu.Model(*TINY), emu.Model(*MICRO_KV)
    plans = [emu.Plan(emu.Layout(m, 1, 1), emu.Layout(m, 2, 1)),
             emu.Plan(emu.Layout(m, 2, 2, 128), emu.Layout(m, 1, 1, 0, "bf16", "separate", "separate")),
             emu.Plan(emu.Layout(m, 1, 1), emu.Layout(m, 2, 2, 384)),
             emu.Plan(emu.Layout(m, 2, 1), emu.Layout(m, 1, 2), bucket_bytes=(1 << 16) - 2),
             emu.Plan(emu.Layout(mk, 8, 3, 2), emu.Layout(mk, 2, 1)),
             emu.Plan(emu.Layout(mk, 1, 1), emu.Layout(mk, 4, 2), bucket_bytes=30)]
    for i, p in enumerate(plans):
        say(f"upload image plan {i}")
        check_upload(p, label=f"plan {i}")


def test_graft_entry_smoke(capsys):
    """The repository's smoke entry point (tiny decoder: reshard, pack and unpack against the oracle)."""
    import __graft_entry__

    __graft_entry__.smoke()
    assert "smoke ok" in capsys.readouterr().out


@pytest.mark.parametrize("dtype,fmt", [("bf16", ("interleaved", "block")), ("fp32", ("separate", "separate"))])
def test_same_layout_is_a_copy(dtype, fmt):
    """The identity plan (source layout == destination layout) is a plain copy. Shards of one full model
    hold equal replicas (norms on every TP rank, KV heads at TP4 over 2 KV heads), as real state does:
    every destination tensor then equals its source tensor byte for byte, except that with vocabulary
    padding the pad rows come out zero while the source's hold garbage that must never be read."""
    import torch

    m = emu.Model(*TINY)
    for tp, pp, pad in ((2, 2, 0), (4, 1, 0), (2, 2, 384)):
        lay = emu.Layout(m, tp, pp, pad, dtype, *fmt)
        plan = emu.Plan(lay, lay)
        assert plan.info["bytes_written"] == plan.info["dst_bytes"] == plan.info["src_bytes"]
        ol = o_layout(lay)
        ws = plan.workspace()
        S = plan.alloc(0, fill=0x5A, guard=GUARD)
        upload_shards(oracle.shard(full_model(ol.model, 29, dtype), ol), S, tweak_replicas=False)
        descs = plan.tensors(1)
        real = {}
        for i, d in enumerate(descs):  # garbage in the source pad rows
            if d["kind"] in ("embed", "lm_head"):
                rows, cols = d["shape"]
                n = max(0, min(rows, m.vocab - d["rank"] % tp * rows)) * (d["bytes"] // rows)
                real[i] = n
                S.tensors[i][n:] = 0x77
        D = plan.alloc(1, fill=0xA5, guard=GUARD)
        g = Guard(keep=S.tensors, fills=[(D.tensors, 0xA5)], label=f"identity TP{tp}PP{pp} pad {pad}")
        plan.reshard(ws, S.ptrs, D.ptrs)
        torch.cuda.synchronize()
        g.check()
        for i, (d, s_, t) in enumerate(zip(descs, S.tensors, D.tensors)):
            n = real.get(i, d["bytes"])
            assert torch.equal(t[:n], s_[:n]), (tp, pp, pad, d)
            assert int(t[n:].count_nonzero()) == 0, (tp, pp, pad, d)
        assert (pad == 0) == all(n == descs[i]["bytes"] for i, n in real.items())


@pytest.mark.parametrize("B", [30, 4096, (1 << 16) - 2])
def test_from_buckets_plans_small(B):
    """Receiver-side plans (emu_plan_from_buckets): source shards packed by the oracle into buckets of B
    bytes are restored -- or resharded into another layout -- by the reshard kernel in one pass, every
    byte against oracle.reshard, with the write footprint checked: unpack (same layout), a TP/PP change,
    format change with padded source rows, zero-filled destination pad rows, and the fp32 -> bf16 and
    bf16 -> fp32 conversions where B holds whole source elements."""
    import torch

    m = emu.Model(*TINY)
    L = lambda *a: emu.Layout(m, *a)
    pairs = [(L(2, 1), L(2, 1)), (L(1, 1), L(2, 1)),
             (L(2, 2, 128), L(1, 1, 0, "bf16", "separate", "separate")), (L(1, 1, 128), L(2, 2, 384)),
             (L(2, 1, 0, "fp32"), L(1, 2, 0, "bf16")), (L(1, 2, 0, "bf16"), L(2, 1, 0, "fp32"))]
    for src, dst in pairs:
        if B % (4 if src.dtype == "fp32" else 2):
            continue
        os_, od = o_layout(src), o_layout(dst)
        shards = oracle.shard(full_model(os_.model, 41, src.dtype), os_)
        plan = emu.Plan(src, dst, src_bucket_bytes=B)
        ws = plan.workspace()
        K = plan.alloc(0, fill=0x5A, guard=GUARD)  # the source side is the bucket list
        packed = [b for rank in shards for b in oracle.pack(rank, B)]
        assert len(packed) == len(K.tensors)
        for t, b in zip(K.tensors, packed):
            t.copy_(torch.from_numpy(np.ascontiguousarray(b).reshape(-1).view(np.uint8).copy()))
        D = plan.alloc(1, fill=0xA5, guard=GUARD)
        label = f"from buckets B={B} {src.dtype} TP{src.tp}PP{src.pp} -> {dst.dtype} TP{dst.tp}PP{dst.pp}"
        g = Guard(keep=K.tensors, fills=[(D.tensors, 0xA5)], label=label)
        plan.reshard(ws, K.ptrs, D.ptrs)
        torch.cuda.synchronize()
        g.check()
        want = [np.ascontiguousarray(a).reshape(-1).view(np.uint8) for rank in oracle.reshard(shards, os_, od)
                for a in rank]
        for i, (t, w) in enumerate(zip(D.tensors, want)):
            assert np.array_equal(t.cpu().numpy(), w), f"{label}: tensor {i}"


def test_callers_own_tensors_and_buckets():
    """A caller's own torch tensors (allocated one by one, in the plan's shapes and element type) and
    bucket buffers, wrapped by Plan.shard_set / Plan.bucket_set: reshard and pack match the oracle."""
    import torch

    m = emu.Model(*TINY)
    src, dst = emu.Layout(m, 2, 2, 128), emu.Layout(m, 1, 2, 0, "bf16", "separate", "separate")
    plan = emu.Plan(src, dst)
    ws = plan.workspace()
    os_, od = o_layout(src), o_layout(dst)
    shards = oracle.shard(full_model(os_.model, 43), os_)
    mine_s = [torch.from_numpy(np.ascontiguousarray(a).view(np.int16).copy()).view(torch.bfloat16).cuda()
              for rank in shards for a in rank]
    mine_d = [torch.empty(tuple(d["shape"]), dtype=torch.bfloat16, device="cuda") for d in plan.tensors(1)]
    S, D = plan.shard_set(0, mine_s), plan.shard_set(1, mine_d)
    plan.check_tables(S.ptrs, D.ptrs)
    plan.reshard(ws, S.ptrs, D.ptrs)
    B = 1000
    bufs = [torch.empty(b["bytes"], dtype=torch.uint8, device="cuda") for b in plan.bucket_info(1, B)]
    views, bptrs = plan.bucket_set(1, B, bufs)
    plan.pack(ws, 1, B, D.ptrs, bptrs)
    torch.cuda.synchronize()
    want = oracle.reshard(shards, os_, od)
    flat = [np.ascontiguousarray(a) for rank in want for a in rank]
    for i, (t, w) in enumerate(zip(mine_d, flat)):
        assert np.array_equal(t.view(torch.int16).cpu().numpy().reshape(-1), w.view(np.int16).reshape(-1)), i
    k = 0
    for rank in want:
        for b in oracle.pack(rank, B):
            assert np.array_equal(views[k].cpu().numpy(), b), k
            k += 1
    assert k == len(bufs)
