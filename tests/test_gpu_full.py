"""GPU parity at full benchmark sizes, in the launch configuration the benchmark times.

* 1B-class decoder, TP4 PP1 -> TP2 PP1 (bf16): every byte against the oracle.
* 8B decoder, TP2 PP2 -> TP4 PP1 (bf16, 16 GB each side): every byte against the oracle, streamed per
  tensor group; the benchmark's 2^28-byte buckets, from emu_pack_buckets and from the fused plan, every
  byte against the oracle, and unpacked; then the reverse transition checked as a round trip on the
  device.
* 8B, padded vocabulary, TP8 PP4 -> TP2 PP2, packed into 2^28-byte buckets (mid-row bucket boundaries)
  and unpacked on the receiver side: reshard, bucket bytes and unpacked tensors against the oracle;
  again with 2^28 - 2 byte buckets, which put tensor and bucket bytes at different 16-byte phases.
* Tensors over 4 GiB: a one-layer decoder with a 266,240-row vocabulary at hidden size 8192 in fp32
  (8.7 GB embedding and LM head), TP1 PP1 -> TP2 PP1, packed into 2^30-byte buckets and unpacked, then
  converted back to bf16 TP1 PP1: every byte against the oracle.
* 8B TP2 PP2 -> TP4 PP1 with non-default tiling and launch options, on sampled tensor groups.
* Resident shards aliased (EMU_PLAN_ALIAS_RESIDENT): 8B TP4 PP2 -> TP4 PP1, PP-only (nothing copied) and
  with the fused formats changed too; every destination tensor against the oracle.
* 8B conversions at full size: fp32 TP4 PP1 -> bf16 TP2 PP2 (the weight sync) and bf16 TP2 PP2 -> fp32
  TP4 PP1, each also fused into 2^28-byte buckets; every byte against the oracle.
* 8B training state, fp32 master + Adam m + v (96 GB in): TP4 PP1 -> TP1 PP1 in one emu_reshard_groups
  launch, then split back into the source buffers with one emu_reshard launch per group; master, m and v checked in full against the oracle,
  the back transition against a seeded regeneration of the original state.

Every call's write footprint is checked as well (tests.gpu_util.Guard): each tensor and bucket view sits
in a 4 KB guard band of a prefill byte, the call's input allocations must come out byte-identical (device
snapshots; regeneration from the seed or a device fingerprint for the 96 GB training state), and every
byte of its output allocations outside the views must still hold the prefill.

Inputs are seeded device draws (synthetic.device_fill); the oracle reads them back as its input.
"""
import gc
import time

import numpy as np
import pytest

import oracle
from paper_2609_34645_amd import emu
from tests.gpu_util import Guard, check_reshard, check_upload, fill_device, host_view, o_layout, say
from tests.shapes import EIGHT_B, HUGE_VOCAB, ONE_B

pytestmark = pytest.mark.gpu
GUARD = 4096  # bytes of prefilled guard band around every view: one reshard tile


def guarded(call, keep, fills, label, snapshot="device"):
    """Run one library call between a Guard's snapshot and its check."""
    import torch

    g = Guard(keep=keep, fills=fills, snapshot=snapshot, label=label)
    call()
    torch.cuda.synchronize()
    n = g.check()
    say(f"  {label}: inputs unchanged, {n} bytes around the outputs untouched")


def free_gb():
    import torch

    return torch.cuda.mem_get_info()[0] / 1e9


def cleanup():
    import torch

    gc.collect()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def make_consistent_replicas(plan, side, sset):
    """Copy each norm's TP-rank-0 replica over the other TP ranks' replicas (a consistent EMU state)."""
    descs = plan.tensors(side)
    lay = plan.src if side == 0 else plan.dst
    first = {}
    for i, d in enumerate(descs):
        if d["kind"].endswith("norm") and d["rank"] % lay.tp == 0:
            first[(d["rank"] // lay.tp, d["kind"], d["layer"])] = i
    for i, d in enumerate(descs):
        if d["kind"].endswith("norm") and d["rank"] % lay.tp:
            sset.tensors[i].copy_(sset.tensors[first[(d["rank"] // lay.tp, d["kind"], d["layer"])]])


def test_1b_tp4_to_tp2(gpu_lib):
    import torch

    m = emu.Model(*ONE_B)
    p = emu.Plan(emu.Layout(m, 4, 1), emu.Layout(m, 2, 1))
    assert p.info["bytes_read"] == 2_997_100_544
    ws = p.workspace()
    S = p.alloc(0, fill=0x5A, guard=GUARD)
    fill_device(p, 0, S, seed=21)
    D = p.alloc(1, fill=0xA5, guard=GUARD)
    guarded(lambda: p.reshard(ws, S.ptrs, D.ptrs), S.tensors, [(D.tensors, 0xA5)], "1B reshard")
    check_reshard(p, S, D, label="1B TP4PP1->TP2PP1")
    del S, D, ws
    cleanup()


def _l1b(tp, pp, pad=0, dtype="bf16", qkv="interleaved", mlp="block"):
    return emu.Layout(emu.Model(*ONE_B), tp, pp, pad, dtype, qkv, mlp)


# 1B layout pairs beyond the benchmark's: TP16 replicates each of the 8 KV heads on two ranks, PP3 splits
# the 16 layers 6/5/5, pad 128 pads the vocabulary (zero-filled destination rows, unread source rows),
# every format combination, and both element conversions.
LAYOUTS_1B = [
    (_l1b(8, 4, 128, qkv="separate", mlp="separate"), _l1b(1, 1, mlp="separate")),
    (_l1b(2, 2, dtype="fp32"), _l1b(4, 4, mlp="separate")),
    (_l1b(16, 3), _l1b(8, 2, 128, qkv="separate")),
    (_l1b(1, 4, qkv="separate"), _l1b(16, 1)),
    (_l1b(8, 3, mlp="separate"), _l1b(2, 1, 128, dtype="fp32", mlp="separate")),
    (_l1b(4, 1, 128, dtype="fp32"), _l1b(16, 3, 128, dtype="fp32", qkv="separate", mlp="separate")),
]


@pytest.mark.parametrize("k", range(len(LAYOUTS_1B)))
def test_1b_layout_pairs(gpu_lib, k):
    """Full-size reshards of the 1B decoder between the layouts above, every byte against the oracle with
    the write footprint checked; the even cases also pack and unpack the destination at a bucket size
    that is not a multiple of 16 bytes."""
    src, dst = LAYOUTS_1B[k]
    label = (f"1B {src.dtype} TP{src.tp}PP{src.pp} pad{src.pad} {src.qkv}/{src.mlp} -> "
             f"{dst.dtype} TP{dst.tp}PP{dst.pp} pad{dst.pad} {dst.qkv}/{dst.mlp}")
    say(f"  {label}")
    p = emu.Plan(src, dst)
    ws = p.workspace()
    S = p.alloc(0, fill=0x5A, guard=GUARD)
    fill_device(p, 0, S, seed=300 + k, dtype=src.dtype)  # source pad rows hold random values too
    D = p.alloc(1, fill=0xA5, guard=GUARD)
    guarded(lambda: p.reshard(ws, S.ptrs, D.ptrs), S.tensors, [(D.tensors, 0xA5)], label)
    check_reshard(p, S, D, label=label)
    if k % 2 == 0:
        es = 4 if dst.dtype == "fp32" else 2
        _pack_check(p, ws, D, (1 << 26) - es, f"{label}: buckets 2^26 - {es}")
    del S, D, ws
    cleanup()


def test_8b_tp2pp2_to_tp4pp1(gpu_lib):
    import torch

    m = emu.Model(*EIGHT_B)
    src, dst = emu.Layout(m, 2, 2), emu.Layout(m, 4, 1)
    p, back = emu.Plan(src, dst), emu.Plan(dst, src)
    assert p.info["bytes_read"] == 16_062_119_936
    ws, wb = p.workspace(), back.workspace()
    S = p.alloc(0, fill=0x5A, guard=GUARD)
    fill_device(p, 0, S, seed=1234)
    D = p.alloc(1, fill=0xA5, guard=GUARD)
    guarded(lambda: p.reshard(ws, S.ptrs, D.ptrs), S.tensors, [(D.tensors, 0xA5)], "8B reshard")
    check_reshard(p, S, D, label="8B TP2PP2->TP4PP1")
    _pack_check(p, ws, D, 1 << 28, "pack and fused reshard->buckets 2^28 (benchmark workload)", S=S, pack_too=True)
    # Merge back: the round trip reproduces the source; norm replicas of TP rank 1 come back as rank 0's
    A2 = back.alloc(1, fill=0x5A, guard=GUARD)
    guarded(lambda: back.reshard(wb, D.ptrs, A2.ptrs), D.tensors, [(A2.tensors, 0x5A)], "8B merge back")
    make_consistent_replicas(p, 0, S)
    for i, (x, y) in enumerate(zip(S.tensors, A2.tensors)):
        assert torch.equal(x, y), f"round trip differs in source tensor {i}"
    del S, D, A2, ws, wb
    cleanup()


def test_8b_uploaded_workspaces_match_host_image(gpu_lib):
    """The benchmark plans' workspaces, with the tile map (about 4 million entries), the stream tables
    and 4 KB chunk maps (about 4 million entries per side) derived on the device, equal the host's image
    byte for byte; the last plan zero-fills padded vocabulary rows."""
    m = emu.Model(*EIGHT_B)
    for src, dst, B in ((emu.Layout(m, 2, 2), emu.Layout(m, 4, 1), 0),
                        (emu.Layout(m, 2, 2), emu.Layout(m, 4, 1), (1 << 28) - 2),
                        (emu.Layout(m, 8, 4, 128), emu.Layout(m, 2, 2, 128), 0),
                        (emu.Layout(m, 4, 1), emu.Layout(m, 8, 4, 128), 0)):
        label = f"TP{src.tp}PP{src.pp}->TP{dst.tp}PP{dst.pp} B={B}"
        say(f"  upload image {label}")
        p = emu.Plan(src, dst, bucket_bytes=B)
        ws = check_upload(p, label)
        del ws, p
    cleanup()


def test_8b_receiver_plans_from_buckets(gpu_lib):
    """Receiver plans (emu_plan_from_buckets) on the benchmark transition: the TP4PP1 destination set
    packed into 2^28- and 2^28-2-byte buckets and restored by TP4PP1 -> TP4PP1 plans reading those
    buckets equals the destination set; the TP2PP2 source set packed into 2^28-byte buckets and resharded
    straight into TP4PP1 tensors equals emu_reshard's result, which is checked against the oracle."""
    import torch

    m = emu.Model(*EIGHT_B)
    src, dst = emu.Layout(m, 2, 2), emu.Layout(m, 4, 1)
    p = emu.Plan(src, dst)
    ws = p.workspace()
    S = p.alloc(0, fill=0x5A, guard=GUARD)
    fill_device(p, 0, S, seed=91)
    make_consistent_replicas(p, 0, S)  # buckets carry every replica; a consistent state holds equal ones
    D = p.alloc(1, fill=0xA5, guard=GUARD)
    guarded(lambda: p.reshard(ws, S.ptrs, D.ptrs), S.tensors, [(D.tensors, 0xA5)], "8B reshard")
    check_reshard(p, S, D, label="8B TP2PP2->TP4PP1 (reference for the receiver plans)")
    for B in (1 << 28, (1 << 28) - 2):
        bufs, bptrs = p.alloc_buckets(1, B, fill=0x77, guard=GUARD)
        guarded(lambda: p.pack(ws, 1, B, D.ptrs, bptrs), D.tensors, [(bufs, 0x77)], f"pack B={B}")
        u = emu.Plan(dst, dst, src_bucket_bytes=B)
        wu = u.workspace()
        R = u.alloc(1, fill=0x11, guard=GUARD)
        guarded(lambda: u.reshard(wu, bptrs, R.ptrs), bufs, [(R.tensors, 0x11)], f"receiver unpack B={B}")
        for i, (x, y) in enumerate(zip(D.tensors, R.tensors)):
            assert torch.equal(x, y), f"receiver unpack B={B}: tensor {i} differs"
        say(f"  receiver unpack B={B}: {len(R.tensors)} tensors equal the destination set")
        del bufs, bptrs, R, wu, u
        cleanup()
    B = 1 << 28
    sbufs, sbptrs = p.alloc_buckets(0, B, fill=0x33, guard=GUARD)
    guarded(lambda: p.pack(ws, 0, B, S.ptrs, sbptrs), S.tensors, [(sbufs, 0x33)], "pack source B=2^28")
    f = emu.Plan(src, dst, src_bucket_bytes=B)
    wf = f.workspace()
    R2 = f.alloc(1, fill=0x22, guard=GUARD)
    guarded(lambda: f.reshard(wf, sbptrs, R2.ptrs), sbufs, [(R2.tensors, 0x22)], "receiver reshard from buckets")
    for i, (x, y) in enumerate(zip(D.tensors, R2.tensors)):
        assert torch.equal(x, y), f"receiver reshard: tensor {i} differs"
    del S, D, sbufs, sbptrs, R2, ws, wf
    cleanup()


def test_8b_padded_receiver_plan_phase_shifted(gpu_lib):
    """The padded workload's receiver side: the TP8PP4 (vocabulary padded to TP*128) source set packed
    into 2^28-2-byte buckets, every bucket at another 16-byte phase, and resharded from them straight
    into TP2PP2 tensors (the byte-granular path at full size) equals emu_reshard's result, which is
    checked against the oracle; source pad rows hold random values and must not be read."""
    import torch

    m = emu.Model(*EIGHT_B)
    src, dst = emu.Layout(m, 8, 4, 128), emu.Layout(m, 2, 2, 128)
    p = emu.Plan(src, dst)
    ws = p.workspace()
    S = p.alloc(0, fill=0x5A, guard=GUARD)
    fill_device(p, 0, S, seed=57)
    D = p.alloc(1, fill=0xA5, guard=GUARD)
    guarded(lambda: p.reshard(ws, S.ptrs, D.ptrs), S.tensors, [(D.tensors, 0xA5)], "8B padded reshard")
    check_reshard(p, S, D, label="8B TP8PP4(pad)->TP2PP2 (reference for the receiver plan)")
    B = (1 << 28) - 2
    sbufs, sbptrs = p.alloc_buckets(0, B, fill=0x33, guard=GUARD)
    guarded(lambda: p.pack(ws, 0, B, S.ptrs, sbptrs), S.tensors, [(sbufs, 0x33)], "pack source B=2^28-2")
    f = emu.Plan(src, dst, src_bucket_bytes=B)
    assert f.info["n_general_segments"] > 0
    wf = f.workspace()
    R = f.alloc(1, fill=0x22, guard=GUARD)
    guarded(lambda: f.reshard(wf, sbptrs, R.ptrs), sbufs, [(R.tensors, 0x22)], "receiver reshard B=2^28-2")
    for i, (x, y) in enumerate(zip(D.tensors, R.tensors)):
        assert torch.equal(x, y), f"receiver reshard B=2^28-2: tensor {i} differs"
    del S, D, sbufs, sbptrs, R, ws, wf
    cleanup()


def _pack_check(p, ws, D, B, label, S=None, pack_too=False):
    """Fill buckets of size B -- with emu_pack_buckets from D, or, when the source set S is given, with
    the fused source -> bucket plan (and with emu_pack_buckets as well when pack_too) -- and compare every
    bucket with oracle.pack of the (oracle-verified) destination tensors rank by rank; then unpack the
    first set into a receiver set and compare it with D."""
    import torch

    sets = []
    if S is None or pack_too:
        bufs, bptrs = p.alloc_buckets(1, B, fill=0x77, guard=GUARD)
        guarded(lambda: p.pack(ws, 1, B, D.ptrs, bptrs), D.tensors, [(bufs, 0x77)], f"{label}: pack")
        sets.append(("pack", bufs, bptrs))
    if S is not None:
        bufs, bptrs = p.alloc_buckets(1, B, fill=0x33, guard=GUARD)
        fused = emu.Plan(p.src, p.dst, bucket_bytes=B)
        wf = fused.workspace()
        guarded(lambda: fused.reshard(wf, S.ptrs, bptrs), S.tensors, [(bufs, 0x33)], f"{label}: fused")
        sets.append(("fused", bufs, bptrs))
    dd = p.tensors(1)
    k = 0
    t = time.time()
    for r in range(p.info["n_dst_ranks"]):
        tensors = [host_view(D.tensors[i], d, p.dst.dtype) for i, d in enumerate(dd) if d["rank"] == r]
        for w in oracle.pack(tensors, B):
            for name, bufs, _ in sets:
                got = bufs[k].cpu().numpy()
                assert got.size == w.size and np.array_equal(got, w), f"{label}: {name} bucket {k} of rank {r} differs"
            k += 1
        del tensors
    for _, bufs, _ in sets:
        assert k == len(bufs)
    say(f"  {label}: {k} buckets x {len(sets)} checked against the oracle in {time.time() - t:.1f} s")
    bufs, bptrs = sets[0][1], sets[0][2]
    R = p.alloc(1, fill=0x11, guard=GUARD)
    guarded(lambda: p.unpack(ws, 1, B, bptrs, R.ptrs), bufs, [(R.tensors, 0x11)], f"{label}: unpack")
    for i, (x, y) in enumerate(zip(D.tensors, R.tensors)):
        assert torch.equal(x, y), f"{label}: unpacked tensor {i} differs"
    del R, sets, bufs, bptrs
    cleanup()


def test_8b_weight_sync_fp32_tp4_to_bf16_tp2pp2(gpu_lib):
    """Training state -> generation weights: fp32 TP4 PP1 master to bf16 TP2 PP2 with the layout change
    and the rounding in one pass, then fused into 2^28-byte buckets; every byte against the oracle."""
    import torch

    m = emu.Model(*EIGHT_B)
    src, dst = emu.Layout(m, 4, 1, 0, "fp32"), emu.Layout(m, 2, 2, 0, "bf16")
    p = emu.Plan(src, dst)
    assert p.info["converts"] == 1 and p.info["bytes_read"] == 2 * p.info["bytes_written"]
    ws = p.workspace()
    S = p.alloc(0, fill=0x5A, guard=GUARD)
    fill_device(p, 0, S, seed=404, dtype="fp32")
    D = p.alloc(1, fill=0xA5, guard=GUARD)
    guarded(lambda: p.reshard(ws, S.ptrs, D.ptrs), S.tensors, [(D.tensors, 0xA5)], "8B fp32 -> bf16 reshard")
    check_reshard(p, S, D, label="8B fp32 TP4PP1 -> bf16 TP2PP2")
    _pack_check(p, ws, D, 1 << 28, "fused fp32 -> bf16 buckets 2^28", S=S)
    del S, D, ws
    cleanup()


def test_8b_bf16_tp2pp2_to_fp32_tp4pp1(gpu_lib):
    """Generation weights -> fp32 state: bf16 TP2 PP2 to fp32 TP4 PP1, the exact widening and the layout
    change in one pass (each destination vector reads 8 bytes), then fused into 2^28-byte buckets;
    every byte against the oracle."""
    import torch

    m = emu.Model(*EIGHT_B)
    src, dst = emu.Layout(m, 2, 2, 0, "bf16"), emu.Layout(m, 4, 1, 0, "fp32")
    p = emu.Plan(src, dst)
    assert p.info["converts"] == 2 and 2 * p.info["bytes_read"] == p.info["bytes_written"]
    ws = p.workspace()
    S = p.alloc(0, fill=0x5A, guard=GUARD)
    fill_device(p, 0, S, seed=405, dtype="bf16")
    D = p.alloc(1, fill=0xA5, guard=GUARD)
    guarded(lambda: p.reshard(ws, S.ptrs, D.ptrs), S.tensors, [(D.tensors, 0xA5)], "8B bf16 -> fp32 reshard")
    check_reshard(p, S, D, label="8B bf16 TP2PP2 -> fp32 TP4PP1")
    _pack_check(p, ws, D, 1 << 28, "fused bf16 -> fp32 buckets 2^28", S=S)
    del S, D, ws
    cleanup()


@pytest.mark.parametrize("opts", [
    {emu.OPT_ROW_WRAP: 0},
    {emu.OPT_LDS_STAGING: 1, emu.OPT_XCD_REMAP: 0, emu.OPT_NONTEMPORAL: 0, emu.OPT_WG_PER_CU: 0},
    {emu.OPT_TILE_VECS: 16, emu.OPT_WG_PER_CU: 2},
], ids=["whole_rows", "lds_plain_order_cached_uncapped", "16k_tiles_cap2"])
def test_8b_non_default_launch_options(gpu_lib, opts):
    """The benchmark transition at full size with non-default tiling and launch options, checked against
    the oracle on the embedding, layers 0, 1 and 31 and the final norm + LM head."""
    import torch

    defaults = {k: emu.get_option(k) for k in range(8)}
    try:
        for k, v in opts.items():
            emu.set_option(k, v)
        m = emu.Model(*EIGHT_B)
        p = emu.Plan(emu.Layout(m, 2, 2), emu.Layout(m, 4, 1))
        ws = p.workspace()
        S = p.alloc(0, fill=0x5A, guard=GUARD)
        fill_device(p, 0, S, seed=77)
        D = p.alloc(1, fill=0xA5, guard=GUARD)
        guarded(lambda: p.reshard(ws, S.ptrs, D.ptrs), S.tensors, [(D.tensors, 0xA5)], f"8B reshard with {opts}")
        check_reshard(p, S, D, groups=["embed", 0, 1, 31, "final"], label=f"8B with {opts}")
        del S, D, ws
        cleanup()
    finally:
        for k, v in defaults.items():
            emu.set_option(k, v)


def test_8b_kv_replication_uneven_pp(gpu_lib):
    """TP2 PP2 -> TP16 PP3: every KV head copied to two ranks, 32 layers over 3 stages (11/11/10)."""
    import torch

    m = emu.Model(*EIGHT_B)
    p = emu.Plan(emu.Layout(m, 2, 2), emu.Layout(m, 16, 3))
    ws = p.workspace()
    S = p.alloc(0, fill=0x5A, guard=GUARD)
    fill_device(p, 0, S, seed=616)
    D = p.alloc(1, fill=0xA5, guard=GUARD)
    guarded(lambda: p.reshard(ws, S.ptrs, D.ptrs), S.tensors, [(D.tensors, 0xA5)], "8B TP2PP2 -> TP16PP3 reshard")
    check_reshard(p, S, D, label="8B TP2PP2 -> TP16PP3")
    del S, D, ws
    cleanup()


def test_8b_padded_tp8pp4_to_tp2pp2_buckets(gpu_lib):
    import torch

    m = emu.Model(*EIGHT_B)
    p = emu.Plan(emu.Layout(m, 8, 4, 128), emu.Layout(m, 2, 2, 128))
    assert p.info["src_vocab_padded"] == 129024 and p.info["dst_vocab_padded"] == 128256
    assert p.bucket_layout(1, 1 << 28, -1) == (60, 16_061_054_976)
    ws = p.workspace()
    S = p.alloc(0, fill=0x5A, guard=GUARD)
    fill_device(p, 0, S, seed=55)    # source pad rows hold random values: they must never be read
    D = p.alloc(1, fill=0xA5, guard=GUARD)
    guarded(lambda: p.reshard(ws, S.ptrs, D.ptrs), S.tensors, [(D.tensors, 0xA5)], "8B padded reshard")
    check_reshard(p, S, D, label="8B TP8PP4(pad)->TP2PP2")
    _pack_check(p, ws, D, 1 << 28, "buckets 2^28")
    _pack_check(p, ws, D, (1 << 28) - 2, "buckets 2^28-2 (phase-shifted)")
    emu.set_option(emu.OPT_BUCKET_TILES, 0)
    try:
        _pack_check(p, ws, D, 1 << 28, "buckets 2^28, persistent kernel")
        _pack_check(p, ws, D, (1 << 28) - 2, "buckets 2^28-2, persistent kernel")
    finally:
        emu.set_option(emu.OPT_BUCKET_TILES, 1)
    _pack_check(p, ws, D, 1 << 28, "fused reshard->buckets 2^28", S=S)
    _pack_check(p, ws, D, (1 << 28) - 2, "fused reshard->buckets 2^28-2", S=S)
    del D, S, ws
    cleanup()


def test_tensors_over_4gib(gpu_lib):
    """fp32 embedding and LM head of 8.7 GB (266,240 x 8192): source tensors, destination shards
    (4.4 GB), segment runs and bucket positions all pass 2^32 bytes, which only 64-bit offsets reach."""
    import torch

    m = emu.Model(*HUGE_VOCAB)
    a, b, c = emu.Layout(m, 1, 1, 0, "fp32"), emu.Layout(m, 2, 1, 0, "fp32"), emu.Layout(m, 1, 1, 0, "bf16")
    p = emu.Plan(a, b)
    assert max(d["bytes"] for d in p.tensors(1)) > 1 << 32
    ws = p.workspace()
    S = p.alloc(0, fill=0x5A, guard=GUARD)
    fill_device(p, 0, S, seed=606, dtype="fp32")
    D = p.alloc(1, fill=0xA5, guard=GUARD)
    guarded(lambda: p.reshard(ws, S.ptrs, D.ptrs), S.tensors, [(D.tensors, 0xA5)], "huge vocab fp32 TP1 -> TP2")
    check_reshard(p, S, D, label="huge vocab fp32 TP1 PP1 -> TP2 PP1")
    del S
    cleanup()
    _pack_check(p, ws, D, 1 << 30, "huge vocab buckets 2^30")
    q = emu.Plan(b, c)
    wq = q.workspace()
    E = q.alloc(1, fill=0x5A, guard=GUARD)
    guarded(lambda: q.reshard(wq, D.ptrs, E.ptrs), D.tensors, [(E.tensors, 0x5A)], "huge vocab fp32 TP2 -> bf16 TP1")
    check_reshard(q, D, E, label="huge vocab fp32 TP2 PP1 -> bf16 TP1 PP1")
    del D, E, ws, wq
    cleanup()


@pytest.mark.parametrize("mixed", [False, True], ids=["pp_only", "pp_and_formats"])
def test_8b_alias_resident_shards(gpu_lib, mixed):
    """Shards already resident are not copied (section 6.2): 8B TP4 PP2 -> TP4 PP1 with the alias plan.
    PP-only, every destination tensor is a source tensor and the reshard moves nothing; with the fused
    formats changed to separate ones as well, the qkv and gate/up tensors are copied and the embedding,
    norms, o, down and LM head are aliased. Every destination tensor against the oracle; bytes read
    drop by exactly the alias bytes."""
    import torch

    m = emu.Model(*EIGHT_B)
    src = emu.Layout(m, 4, 2)
    dst = emu.Layout(m, 4, 1, qkv="separate", mlp="separate") if mixed else emu.Layout(m, 4, 1)
    full, p = emu.Plan(src, dst), emu.Plan(src, dst, alias=True)
    assert p.info["bytes_read"] == full.info["bytes_read"] - p.info["alias_bytes"]
    assert p.info["bytes_written"] == full.info["bytes_written"] - p.info["alias_bytes"]
    if not mixed:
        assert p.info["n_alias_tensors"] == p.info["n_dst_tensors"] and p.info["bytes_read"] == 0
    ws = p.workspace()
    S = p.alloc(0, fill=0x5A, guard=GUARD)
    fill_device(p, 0, S, seed=808)
    make_consistent_replicas(p, 0, S)
    D = p.alloc(1, fill=0xA5, guard=GUARD, alias=S)
    own = [t for t, d in zip(D.tensors, p.tensors(1)) if d["alias"] < 0]
    assert len(own) == p.info["n_dst_tensors"] - p.info["n_alias_tensors"]
    guarded(lambda: p.reshard(ws, S.ptrs, D.ptrs), S.tensors, [(own, 0xA5)] if own else [],
            f"8B alias plan {'mixed' if mixed else 'PP-only'}")
    check_reshard(p, S, D, label=f"8B TP4PP2->TP4PP1 aliased ({'formats changed' if mixed else 'PP only'})")
    say(f"  alias plan: {p.info['n_alias_tensors']} of {p.info['n_dst_tensors']} tensors aliased, "
        f"{p.info['alias_bytes'] / 1e9:.2f} GB not copied, {p.info['bytes_read'] / 1e9:.2f} GB read")
    del S, D, ws
    cleanup()


def regenerate(fwd, name, dist, seed):
    """The training-state group `name` as the fixture made it, in a fresh, identically laid out set."""
    ref = fwd.alloc(0, fill=0x5A, guard=GUARD)
    fill_device(fwd, 0, ref, seed=seed, dtype="fp32", dist_override=None if name == "master" else dist)
    make_consistent_replicas(fwd, 0, ref)
    return ref


@pytest.fixture(scope="module")
def train_state(gpu_lib):
    """fp32 master, Adam m and v in the TP4 PP1 layout, resharded to TP1 PP1 in one grouped launch.
    The sources must come out of it unchanged (whole allocations, against a seeded
    regeneration) and the destination allocations untouched outside their views."""
    import torch

    need = 2 * 96.4 + 33
    if free_gb() < need:
        pytest.skip(f"needs {need:.0f} GB of free device memory, {free_gb():.0f} GB free")
    m = emu.Model(*EIGHT_B)
    a, b = emu.Layout(m, 4, 1, 0, "fp32"), emu.Layout(m, 1, 1, 0, "fp32")
    fwd, back = emu.Plan(a, b), emu.Plan(b, a)
    wf, wb = fwd.workspace(), back.workspace()
    groups = {"master": ("weight", 301), "adam_m": ("adam_m", 302), "adam_v": ("adam_v", 303)}
    S, D = {}, {}
    t = time.time()
    for name, (dist, seed) in groups.items():
        S[name] = regenerate(fwd, name, dist, seed)
        D[name] = fwd.alloc(1, fill=0xA5, guard=GUARD)
    torch.cuda.synchronize()
    say(f"  fp32 state filled ({3 * fwd.info['src_bytes'] / 1e9:.1f} GB) in {time.time() - t:.1f} s")
    guards = [Guard(fills=[(D[name].tensors, 0xA5)], label=f"fp32 {name} TP4->TP1") for name in groups]
    # master, m and v in one launch (emu_reshard_groups); the back transition below takes one launch each
    fwd.reshard_groups(wf, emu.group_tables([S[n] for n in groups]), emu.group_tables([D[n] for n in groups]))
    torch.cuda.synchronize()
    n = sum(g.check() for g in guards)
    for name, (dist, seed) in groups.items():
        ref = regenerate(fwd, name, dist, seed)
        for r, (x, y) in enumerate(zip(ref.bufs, S[name].bufs)):
            assert torch.equal(x, y), f"{name}: source buffer of rank {r} changed by the forward reshard"
        del ref
        cleanup()
    say(f"  fp32 state TP4->TP1: sources unchanged, {n} bytes around the destinations untouched")
    yield dict(fwd=fwd, back=back, wf=wf, wb=wb, S=S, D=D, groups=groups)
    S.clear()
    D.clear()
    cleanup()


def test_8b_fp32_master_full(train_state):
    st = train_state
    assert st["fwd"].info["bytes_read"] * 3 == 96_363_134_976
    check_reshard(st["fwd"], st["S"]["master"], st["D"]["master"], label="fp32 master TP4->TP1")


@pytest.mark.parametrize("name", ["adam_m", "adam_v"])
def test_8b_fp32_adam_full(train_state, name):
    st = train_state
    check_reshard(st["fwd"], st["S"][name], st["D"][name], label=f"fp32 {name} TP4->TP1")


def test_8b_fp32_split_back_in_place(train_state):
    """Split back into the original source buffers, one launch per group: the destination sets (read
    only) keep their device fingerprint, the bytes around the rewritten source views keep their
    prefill, and every source allocation equals a seeded regeneration of the original state."""
    import torch

    st = train_state
    fwd, back = st["fwd"], st["back"]
    assert back.info["bytes_read"] * 3 == 96_372_719_616
    guards = [Guard(keep=st["D"][name].tensors, fills=[(st["S"][name].tensors, 0x5A)], snapshot="hash",
                    label=f"fp32 {name} TP1->TP4") for name in st["groups"]]
    for name in st["groups"]:
        back.reshard(st["wb"], st["D"][name].ptrs, st["S"][name].ptrs)   # into the original source buffers
    torch.cuda.synchronize()
    for g in guards:
        g.check()
    for name, (dist, seed) in st["groups"].items():
        ref = regenerate(fwd, name, dist, seed)
        for r, (x, y) in enumerate(zip(ref.bufs, st["S"][name].bufs)):
            assert torch.equal(x, y), f"{name}: buffer of rank {r} differs after the round trip"
        del ref
        cleanup()
    say("  fp32 training state round trip TP4->TP1->TP4 bit-exact")
