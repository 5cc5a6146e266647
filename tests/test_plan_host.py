"""Host-side checks of libemu.so (no GPU needed): symbols, plan compiler, bucket geometry, errors.

The plan compiler is checked against the oracle through a test-only interpreter of its segment
table (tests/plan_interp.py) and for exact cover: every destination byte written exactly once.
"""
import ctypes
import itertools
import os
import re

import numpy as np
import pytest

import oracle
from paper_2609_34645_amd import emu
from synthetic import host_tensor
from tests.plan_interp import coverage, run_plan
from tests.shapes import EIGHT_B, MICRO, MICRO8, MICRO_KV, ONE_B, TINY

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FMT = {("interleaved", "block"), ("separate", "separate"), ("interleaved", "separate"), ("separate", "block")}


def o_layout(lay):
    m = lay.model
    om = oracle.Model(m.num_layers, m.hidden, m.num_heads, m.head_dim, m.num_kv_heads, m.ffn_hidden, m.vocab)
    return oracle.Layout(om, lay.tp, lay.pp, lay.pad, lay.dtype, lay.qkv, lay.mlp)


def header_functions():
    text = open(os.path.join(ROOT, "include", "emu.h")).read()
    return sorted(set(re.findall(r"^(?:int|void|const char\*)\s+(emu_\w+)\s*\(", text, re.M)))


def test_library_exports_every_declared_function():
    lib = emu.load()
    names = header_functions()
    assert len(names) >= 14
    for n in names:
        assert hasattr(lib, n), n
    assert lib.emu_version() == 2


def full_model(model, seed=11, dtype="bf16"):
    full = {}
    for i, (_, key, shape, kind) in enumerate(oracle.logical_tensors(model)):
        full[key] = host_tensor(seed, (1, i), shape, "norm" if kind.endswith("norm") else "weight", dtype)
    return full


def check_pair(src, dst, full=None, seed=11):
    plan = emu.Plan(src, dst)
    os_, od = o_layout(src), o_layout(dst)
    # tensor inventory matches the oracle's
    for side, ol in ((0, os_), (1, od)):
        descs = plan.tensors(side)
        inv = [s for specs in oracle.rank_inventory(ol) for s in specs]
        assert [(d["kind"], d["layer"], tuple(d["shape"])) for d in descs] == \
            [(s.kind, s.layer, tuple(s.shape)) for s in inv]
    if full is None:
        full = full_model(os_.model, seed, src.dtype)
    src_shards = oracle.shard(full, os_)
    # replicas on TP ranks > 0 get different values: the plan must read TP rank 0
    for r, specs in enumerate(oracle.rank_inventory(os_)):
        for j, s in enumerate(specs):
            if s.kind.endswith("norm") and r % os_.tp:
                src_shards[r][j] = src_shards[r][j] ^ np.array(0x5A5A, dtype=src_shards[r][j].dtype) \
                    if src_shards[r][j].dtype == np.uint16 else src_shards[r][j] * 3
    flat_src = [np.ascontiguousarray(a).reshape(-1).view(np.uint8) for rank in src_shards for a in rank]
    want = [np.ascontiguousarray(a).reshape(-1).view(np.uint8) for rank in oracle.reshard(src_shards, os_, od)
            for a in rank]
    got = run_plan(plan.segments(), flat_src, [w.size for w in want])
    for j, (g, w) in enumerate(zip(got, want)):
        assert np.array_equal(g, w), (src, dst, j)
    info = plan.info
    assert info["bytes_written"] == sum(w.size for w in want)
    return plan


def micro_layouts(shape=MICRO):
    m = emu.Model(*shape)
    return [emu.Layout(m, tp, pp, pad, "bf16", q, g)
            for tp, pp, pad, (q, g) in itertools.product((1, 2, 4), (1, 2, 4), (0, 2), sorted(FMT))]


MICRO_LAYS = micro_layouts()


@pytest.mark.parametrize("i", range(0, len(MICRO_LAYS), 3))
def test_plan_interpreter_matches_oracle_micro(i):
    src = MICRO_LAYS[i]
    full = full_model(o_layout(src).model)
    for dst in MICRO_LAYS[::2] + MICRO_LAYS[1::7]:
        check_pair(src, dst, full)


def test_plan_interpreter_matches_oracle_tiny_config():
    m = emu.Model(*TINY)
    a, b = emu.Layout(m, 1, 1), emu.Layout(m, 2, 1)
    check_pair(a, b)
    check_pair(b, a)
    check_pair(emu.Layout(m, 2, 2, 128), emu.Layout(m, 1, 1, 0, "bf16", "separate", "separate"))


def test_plan_interpreter_fp32_micro8_t_sub():
    m = emu.Model(*MICRO8)
    for pad in (0, 2):
        check_pair(emu.Layout(m, 4, 8, pad, "fp32"), emu.Layout(m, 8, 2, pad, "fp32"))
        check_pair(emu.Layout(m, 4, 8, pad, "fp32"), emu.Layout(m, 4, 2, pad, "fp32"))


def test_interrupted_plan_never_writes_the_source():
    """A transition stopped partway loses no state (section 6.2, safe concurrent execution): running
    any prefix of the copy map reads the source only."""
    m = emu.Model(*TINY)
    src, dst = emu.Layout(m, 2, 1), emu.Layout(m, 1, 1)
    plan = emu.Plan(src, dst)
    segs = plan.segments()
    os_ = o_layout(src)
    flat = [np.ascontiguousarray(a).reshape(-1).view(np.uint8) for rank in oracle.shard(full_model(os_.model), os_)
            for a in rank]
    before = [x.copy() for x in flat]
    sizes = [d["bytes"] for d in plan.tensors(1)]
    for k in (0, 1, len(segs) // 2, len(segs)):
        run_plan(segs, flat, sizes, prefix=k)
        assert all(np.array_equal(a, b) for a, b in zip(before, flat))


def exact_cover(plan):
    sizes = [d["bytes"] for d in plan.tensors(1)]
    for n, iv in zip(sizes, coverage(plan.segments(), sizes)):
        pos = 0
        for a, b in iv:
            assert a == pos, "gap or overlap in destination coverage"
            pos = b
        assert pos == n


@pytest.mark.parametrize("src,dst,read", [
    ((ONE_B, 4, 1, 0), (ONE_B, 2, 1, 0), 2_997_100_544),
    ((EIGHT_B, 2, 2, 0), (EIGHT_B, 4, 1, 0), 16_062_119_936),
    ((EIGHT_B, 8, 4, 128), (EIGHT_B, 2, 2, 128), 16_061_054_976),
    ((EIGHT_B, 2, 2, 128), (EIGHT_B, 8, 4, 128), None),
])
def test_exact_cover_and_bytes_at_benchmark_shapes(src, dst, read):
    ms, md = emu.Model(*src[0]), emu.Model(*dst[0])
    plan = emu.Plan(emu.Layout(ms, *src[1:]), emu.Layout(md, *dst[1:]))
    exact_cover(plan)
    if read is not None:
        assert plan.info["bytes_read"] == read == plan.info["bytes_written"]
    else:
        # reverse of the padded case: the 768 destination pad rows of the embedding (rank t=7, p=0) and
        # of the LM head (rank t=7, p=3) are zero-filled
        assert plan.info["zero_fill_bytes"] == 2 * (129024 - 128256) * 4096 * 2
        assert plan.info["n_general_segments"] == 0


def test_fp32_training_state_bytes():
    m = emu.Model(*EIGHT_B)
    a = emu.Plan(emu.Layout(m, 4, 1, 0, "fp32"), emu.Layout(m, 1, 1, 0, "fp32"))
    b = emu.Plan(emu.Layout(m, 1, 1, 0, "fp32"), emu.Layout(m, 4, 1, 0, "fp32"))
    assert a.info["bytes_read"] == 96_363_134_976 // 3
    assert b.info["bytes_read"] == 96_372_719_616 // 3
    exact_cover(a)


def test_bucket_layout_padded_case():
    m = emu.Model(*EIGHT_B)
    plan = emu.Plan(emu.Layout(m, 8, 4, 128), emu.Layout(m, 2, 2, 128))
    assert plan.bucket_layout(1, 2**28, 0) == (15, 4_015_259_648)
    assert plan.bucket_layout(1, 2**28, 3) == (15, 4_015_267_840)
    assert plan.bucket_layout(1, 2**28, -1) == (60, 16_061_054_976)
    descs = plan.tensors(1)
    assert [d["stream_offset"] for d in descs[:3]] == [0, 525_336_576, 525_344_768]


def test_error_codes():
    lib = emu.load()
    m = emu.Model(*TINY)
    assert emu.layout_check(emu.Layout(m, 2, 2)) == 0
    assert emu.layout_check(emu.Layout(m, 4, 1)) == 0           # tp > KV heads: KV replication
    assert emu.layout_check(emu.Layout(m, 3, 1)) == -2          # tp > KV heads but not a multiple
    assert emu.layout_check(emu.Layout(m, 1, 3)) == -2          # pp does not divide L
    assert emu.layout_check(emu.Layout(emu.Model(2, 256, 4, 64, 2, 688, 1023), 2, 1)) == -2
    assert emu.layout_check(emu.Layout(emu.Model(2, 256, 4, 64, 2, 688, 1023), 2, 1, pad=64)) == 0
    assert emu.Plan(emu.Layout(m, 1, 1), emu.Layout(m, 1, 1, dtype="fp32")).info["converts"] == 2
    with pytest.raises(emu.EmuError) as e:
        emu.Plan(emu.Layout(m, 1, 1), emu.Layout(emu.Model(*MICRO), 1, 1))
    assert e.value.code == -3
    deep = emu.Model(400, 16, 2, 8, 2, 16, 16)                  # 2,403 tensors on one rank at PP1
    with pytest.raises(emu.EmuError) as e:
        emu.Plan(emu.Layout(deep, 1, 2), emu.Layout(deep, 1, 1))
    assert e.value.code == -4
    assert emu.Plan(emu.Layout(deep, 1, 2), emu.Layout(deep, 2, 2)).info["n_dst_tensors"] == 2 * (2 * 6 * 200 + 3)
    huge = emu.Model(1, 8192, 64, 128, 8, 2048, 1 << 30)         # 16 TiB embedding: 2^32 tiles of 4 KB
    with pytest.raises(emu.EmuError) as e:
        emu.Plan(emu.Layout(huge, 1, 1), emu.Layout(huge, 2, 1))
    assert e.value.code == -4 and "too many tiles" in str(e.value)
    plan = emu.Plan(emu.Layout(m, 1, 1), emu.Layout(m, 2, 1))
    with pytest.raises(emu.EmuError) as e:
        plan.bucket_layout(1, 0)
    assert e.value.code == -6
    with pytest.raises(emu.EmuError) as e:
        plan.bucket_layout(1, 3)                                 # not a multiple of 2 bytes
    assert e.value.code == -6
    with pytest.raises(emu.EmuError) as e:
        plan.bucket_layout(1, 1024, 2)
    assert e.value.code == -10
    d = emu.c_tensor_desc()
    assert lib.emu_tensor_info(plan._h, 2, 0, ctypes.byref(d)) == -10
    assert lib.emu_tensor_info(plan._h, 0, 10**6, ctypes.byref(d)) == -10
    assert lib.emu_plan(None, None, None) == -1
    h = plan._h
    plan.close()
    info = emu.c_plan_info()
    assert lib.emu_plan_info(h, ctypes.byref(info)) == -9        # freed handle
    assert lib.emu_plan_free(h) == -9
    assert lib.emu_reshard(h, None, None, None, None) == -9
    assert b"live plan" in lib.emu_last_error()
    assert lib.emu_set_option(0, 5) == -11
    assert lib.emu_set_option(99, 1) == -10
    assert lib.emu_set_option(emu.OPT_WG_PER_CU, 33) == -11 and lib.emu_set_option(emu.OPT_WG_PER_CU, -2) == -11
    assert lib.emu_set_option(8, 0) == -10 and lib.emu_set_option(emu.OPT_ROW_WRAP, 2) == -11
    for s in range(-11, 1):
        assert lib.emu_status_str(s).startswith(b"EMU_")


def _expected_aliases(src, dst):
    """Brute force from the oracle's per-element coordinates: destination tensor j is a whole copy of
    source tensor i iff both hold the same logical elements in the same order (no pad rows), in the same
    element type, and source tensor i is the first holder of every one of its elements (replicated
    elements are read from their first holder: norms from TP rank 0, replicated KV heads from their
    first rank)."""
    from oracle import coords

    if src.dtype != dst.dtype:
        return None
    sid = [tuple(ids) for rank in coords.element_ids(o_layout(src)) for ids in rank]
    owner = {}
    for i, ids in enumerate(sid):
        for e in ids:
            owner.setdefault(e, i)
    clean = {ids: i for i, ids in enumerate(sid) if all(owner[e] == i for e in ids)}
    out = []
    for ids in (tuple(x) for rank in coords.element_ids(o_layout(dst)) for x in rank):
        out.append(clean.get(ids, -1) if min(ids) >= 0 else -1)
    return out


def check_alias_pair(src, dst, seed=17):
    """The alias plan against the oracle: alias tensors are exactly the brute-force whole copies, each
    equals its source tensor in the oracle's reshard (with unequal norm replicas, so a wrong replica
    shows), the map writes every other destination byte exactly once and nothing of an alias tensor,
    and the read/write counts drop by the alias bytes."""
    full_plan = emu.Plan(src, dst)
    plan = emu.Plan(src, dst, alias=True)
    descs = plan.tensors(1)
    got_alias = [d["alias"] for d in descs]
    assert got_alias == [d["alias"] for d in full_plan.tensors(1)]      # detection does not depend on the flag
    want_alias = _expected_aliases(src, dst)
    assert got_alias == (want_alias if want_alias is not None else [-1] * len(descs)), (src, dst)
    os_, od = o_layout(src), o_layout(dst)
    src_shards = oracle.shard(full_model(os_.model, seed, src.dtype), os_)
    for r, specs in enumerate(oracle.rank_inventory(os_)):
        for j, sp in enumerate(specs):
            if sp.kind.endswith("norm") and r % os_.tp:
                src_shards[r][j] = src_shards[r][j] + np.array(1, dtype=src_shards[r][j].dtype)
    flat_src = [np.ascontiguousarray(a).reshape(-1).view(np.uint8) for rank in src_shards for a in rank]
    want = [np.ascontiguousarray(a).reshape(-1).view(np.uint8) for rank in oracle.reshard(src_shards, os_, od)
            for a in rank]
    got = run_plan(plan.segments(), flat_src, [w.size for w in want])
    cover = coverage(plan.segments(), [w.size for w in want])
    nbytes = 0
    for j, (g, w, a) in enumerate(zip(got, want, got_alias)):
        if a >= 0:
            assert np.array_equal(flat_src[a], w), (src, dst, j)
            assert cover[j] == [], (src, dst, j)
            nbytes += w.size
        else:
            assert np.array_equal(g, w), (src, dst, j)
    info, full_info = plan.info, full_plan.info
    assert info["aliased"] == 1 and full_info["aliased"] == 0
    assert info["n_alias_tensors"] == full_info["n_alias_tensors"] == sum(a >= 0 for a in got_alias)
    assert info["alias_bytes"] == full_info["alias_bytes"] == nbytes
    assert info["bytes_written"] == full_info["bytes_written"] - nbytes
    assert info["bytes_read"] == full_info["bytes_read"] - nbytes
    return plan


@pytest.mark.parametrize("i", range(0, len(MICRO_LAYS), 4))
def test_alias_plans_match_oracle_micro(i):
    src = MICRO_LAYS[i]
    for dst in MICRO_LAYS[::3] + [src, emu.Layout(src.model, src.tp, 1, src.pad, src.dtype, src.qkv, src.mlp)]:
        check_alias_pair(src, dst)


def test_alias_kv_replication_uneven_pp_and_conversion():
    m = emu.Model(3, 16, 8, 2, 2, 16, 16)
    for a, b in ((emu.Layout(m, 8, 3), emu.Layout(m, 8, 1)), (emu.Layout(m, 4, 2), emu.Layout(m, 8, 3)),
                 (emu.Layout(m, 2, 3, 2), emu.Layout(m, 2, 2, 2)), (emu.Layout(m, 2, 1), emu.Layout(m, 2, 1, 0, "fp32"))):
        check_alias_pair(a, b)


def test_alias_counts_8b():
    """8B: a PP-only change aliases every destination tensor (nothing is copied); TP2 PP2 -> TP4 PP1
    aliases every norm (each a whole copy of TP rank 0's norm of its layer's stage) and nothing else; a
    PP-only change that also changes the fused formats aliases the tensors the formats leave alone."""
    m = emu.Model(*EIGHT_B)
    pp_only = emu.Plan(emu.Layout(m, 4, 2), emu.Layout(m, 4, 1), alias=True)
    assert pp_only.info["n_alias_tensors"] == pp_only.info["n_dst_tensors"] == 780
    assert pp_only.info["bytes_read"] == 0 and pp_only.info["n_tiles"] == 0
    tp = emu.Plan(emu.Layout(m, 2, 2), emu.Layout(m, 4, 1), alias=True)
    norms = [d for d in tp.tensors(1) if d["kind"].endswith("norm")]
    assert tp.info["n_alias_tensors"] == len(norms) == 4 * (2 * 32 + 1)
    mixed = emu.Plan(emu.Layout(m, 4, 2), emu.Layout(m, 4, 1, qkv="separate", mlp="separate"), alias=True)
    kinds = {d["kind"] for d in mixed.tensors(1) if d["alias"] >= 0}
    assert kinds == {"embed", "attn_norm", "o", "mlp_norm", "down", "final_norm", "lm_head"}


@pytest.mark.parametrize("B", [2, 30, 4094, 65538, 1 << 20])
def test_bucket_info_matches_oracle_pack(B):
    """emu_bucket_info: each bucket's rank, index, stream offset and size equal what oracle.pack makes of
    each destination rank's tensors; sub-ranges return the same entries; a range past the end fails."""
    m = emu.Model(*TINY)
    src, dst = emu.Layout(m, 2, 2, 128), emu.Layout(m, 1, 2, 0, "bf16", "separate", "block")
    plan = emu.Plan(src, dst)
    od = o_layout(dst)
    want = []
    for r, specs in enumerate(oracle.rank_inventory(od)):
        tensors = [np.zeros(sp.shape, dtype=np.uint16) for sp in specs]
        off = 0
        for k, b in enumerate(oracle.pack(tensors, B)):
            want.append(dict(rank=r, index=k, stream_offset=off, bytes=b.size))
            off += b.size
    got = plan.bucket_info(1, B)
    assert got == want
    n = len(want)
    lib = emu.load()
    arr = (emu.c_bucket_desc * 3)()
    assert lib.emu_bucket_info(plan._h, 1, B, n - 3, 3, arr) == 0
    assert [dict(rank=a.rank, index=a.index, stream_offset=a.stream_offset, bytes=a.bytes) for a in arr] == want[-3:]
    assert lib.emu_bucket_info(plan._h, 1, B, n - 2, 3, arr) == -10
    assert lib.emu_bucket_info(plan._h, 1, B, n, 0, arr) == 0
    assert lib.emu_bucket_info(plan._h, 1, 3, 0, 1, arr) == -6
    assert lib.emu_bucket_info(plan._h, 2, B, 0, 1, arr) == -10


def test_noalloc_size_limit_is_checked_before_any_gpu_call():
    """emu_reshard_noalloc refuses a plan whose tables exceed its 32 MiB static array with
    EMU_ERR_WORKSPACE before any HIP call (so here, without a GPU, too); the 8B fp32 training-state plan
    at the default 4 KB tiles (31.4 MB of tables, the largest workload) passes the check and only then
    meets the missing device (EMU_ERR_HIP)."""
    lib = emu.load()
    m = emu.Model(*EIGHT_B)
    a, b = emu.Layout(m, 4, 1, 0, "fp32"), emu.Layout(m, 1, 1, 0, "fp32")
    fits = emu.Plan(a, b)
    fake = ctypes.c_void_p(1 << 20)   # 8-byte aligned, never dereferenced: the call stops on the host
    assert lib.emu_reshard_noalloc(fits._h, fake, fake, None) == -8
    old = emu.get_option(emu.OPT_TILE_VECS)
    emu.set_option(emu.OPT_TILE_VECS, 1)                          # 1 KB tiles: 4x the tile map
    try:
        big = emu.Plan(a, b)
    finally:
        emu.set_option(emu.OPT_TILE_VECS, old)
    assert big.info["n_tiles"] * 4 > 32 << 20
    assert lib.emu_reshard_noalloc(big._h, fake, fake, None) == -5
    assert b"static scratch" in lib.emu_last_error()
    assert lib.emu_reshard_noalloc(big._h, None, fake, None) == -1


# ------------------------------------------------------------------------------------------------
# fused reshard -> buckets (emu_plan_to_buckets)
# ------------------------------------------------------------------------------------------------

def check_fused(src, dst, B, full=None, seed=13):
    plan = emu.Plan(src, dst, bucket_bytes=B)
    os_, od = o_layout(src), o_layout(dst)
    if full is None:
        full = full_model(os_.model, seed, src.dtype)
    src_shards = oracle.shard(full, os_)
    for r, specs in enumerate(oracle.rank_inventory(os_)):
        for j, s in enumerate(specs):
            if s.kind.endswith("norm") and r % os_.tp:
                src_shards[r][j] = src_shards[r][j] + np.array(1, dtype=src_shards[r][j].dtype)
    flat_src = [np.ascontiguousarray(a).reshape(-1).view(np.uint8) for rank in src_shards for a in rank]
    want = [b for rank in oracle.reshard(src_shards, os_, od) for b in oracle.pack(rank, B)]
    descs = plan.tensors(1)
    assert [d["kind"] for d in descs] == ["bucket"] * len(want)
    assert [d["bytes"] for d in descs] == [w.size for w in want]
    got = run_plan(plan.segments(), flat_src, [w.size for w in want])
    for k, (g, w) in enumerate(zip(got, want)):
        assert np.array_equal(g, w), (src, dst, B, k)
    return plan


@pytest.mark.parametrize("B", [8, 30, 64, 1000, 4094, 1 << 20])
def test_fused_plan_matches_oracle_micro(B):
    lays = MICRO_LAYS[::5]
    full = full_model(o_layout(lays[0]).model)
    for i, src in enumerate(lays):
        for dst in lays[i % 3::3]:
            check_fused(src, dst, B, full)


def test_fused_plan_matches_oracle_tiny_and_fp32():
    m = emu.Model(*TINY)
    for B in (1 << 16, (1 << 16) - 2, 12345 * 2):
        check_fused(emu.Layout(m, 1, 1), emu.Layout(m, 2, 1), B)
        check_fused(emu.Layout(m, 2, 2, 128), emu.Layout(m, 1, 1, 0, "bf16", "separate", "separate"), B)
    check_fused(emu.Layout(m, 2, 1, 0, "fp32"), emu.Layout(m, 1, 2, 0, "fp32"), 4 * 1001)


@pytest.mark.parametrize("B", [1 << 28, (1 << 28) - 2, 256 * 10**6])
def test_fused_plan_exact_cover_8b(B):
    m = emu.Model(*EIGHT_B)
    plan = emu.Plan(emu.Layout(m, 2, 2), emu.Layout(m, 4, 1), bucket_bytes=B)
    base = emu.Plan(emu.Layout(m, 2, 2), emu.Layout(m, 4, 1))
    nb, sb = base.bucket_layout(1, B, -1)
    assert plan.info["n_dst_tensors"] == nb and plan.info["bytes_written"] == sb == base.info["bytes_written"]
    exact_cover(plan)
    if B % 16 == 0:
        assert plan.info["n_general_segments"] == 0


def test_fused_plan_errors():
    m = emu.Model(*TINY)
    lib = emu.load()
    a, b, h = emu.Layout(m, 1, 1).c(), emu.Layout(m, 2, 1).c(), ctypes.c_void_p()
    assert lib.emu_plan_to_buckets(ctypes.byref(a), ctypes.byref(b), 0, ctypes.byref(h)) == -6
    assert lib.emu_plan_to_buckets(ctypes.byref(a), ctypes.byref(b), 3, ctypes.byref(h)) == -6
    assert lib.emu_plan_to_buckets(None, ctypes.byref(b), 64, ctypes.byref(h)) == -1
    # a fused plan may hold any number of buckets, but packing its bucket side (more than 2048 buckets
    # on one rank) is rejected before anything is launched
    p = emu.Plan(emu.Layout(m, 1, 1), emu.Layout(m, 2, 1), bucket_bytes=64)
    assert p.info["n_dst_tensors"] == 2 * -(-1_976_832 // 64)
    ws = ctypes.create_string_buffer(512)
    addr = (ctypes.addressof(ws) + 255) // 256 * 256
    fake = ctypes.c_void_p(addr)
    assert lib.emu_pack_buckets(p._h, fake, 1, 64, fake, fake, None) == -4


def check_from_buckets(src, dst, B, full=None, seed=13):
    """The receiver's plan (source side: the source ranks' buckets of size B) against the oracle: the
    source shards packed by oracle.pack, run through the plan's segment table, must give
    oracle.reshard of the shards. Replicas past their first holder are perturbed, so that reading
    one shows."""
    plan = emu.Plan(src, dst, src_bucket_bytes=B)
    os_, od = o_layout(src), o_layout(dst)
    if full is None:
        full = full_model(os_.model, seed, src.dtype)
    src_shards = oracle.shard(full, os_)
    for r, specs in enumerate(oracle.rank_inventory(os_)):
        for j, sp in enumerate(specs):
            if sp.kind.endswith("norm") and r % os_.tp:
                src_shards[r][j] = src_shards[r][j] + np.array(1, dtype=src_shards[r][j].dtype)
    buckets = [b for rank in src_shards for b in oracle.pack(rank, B)]
    descs = plan.tensors(0)
    assert [d["kind"] for d in descs] == ["bucket"] * len(buckets)
    assert [d["bytes"] for d in descs] == [b.size for b in buckets]
    want = [np.ascontiguousarray(a).reshape(-1).view(np.uint8) for rank in oracle.reshard(src_shards, os_, od)
            for a in rank]
    got = run_plan(plan.segments(), buckets, [w.size for w in want])
    for i, (g, w) in enumerate(zip(got, want)):
        assert np.array_equal(g, w), (src, dst, B, i)
    return plan


@pytest.mark.parametrize("B", [8, 30, 64, 1000, 4094, 1 << 20])
def test_from_buckets_plan_matches_oracle_micro(B):
    lays = MICRO_LAYS[::5]
    full = full_model(o_layout(lays[0]).model)
    for i, src in enumerate(lays):
        for dst in lays[i % 3::3] + [src]:  # dst == src: the plan is an unpack
            check_from_buckets(src, dst, B, full)


def test_from_buckets_plan_matches_oracle_tiny_kv_and_conversion():
    m = emu.Model(*TINY)
    for B in (1 << 16, (1 << 16) - 2, 12345 * 2):
        check_from_buckets(emu.Layout(m, 1, 1), emu.Layout(m, 2, 1), B)
        check_from_buckets(emu.Layout(m, 2, 2, 128), emu.Layout(m, 1, 1, 0, "bf16", "separate", "separate"), B)
        check_from_buckets(emu.Layout(m, 1, 1, 128), emu.Layout(m, 2, 2, 384), B)  # zero-filled pad rows
    check_from_buckets(emu.Layout(m, 2, 1, 0, "fp32"), emu.Layout(m, 1, 2, 0, "bf16"), 4 * 1001)
    check_from_buckets(emu.Layout(m, 2, 1, 0, "bf16"), emu.Layout(m, 4, 2, 0, "fp32"), 2 * 1001)
    mk = emu.Model(*MICRO_KV)
    full = full_model(o_layout(emu.Layout(mk, 1, 1)).model, 23)
    for B in (6, 40, 4096):
        check_from_buckets(emu.Layout(mk, 8, 3, 2), emu.Layout(mk, 2, 1), B, full)
        check_from_buckets(emu.Layout(mk, 1, 2), emu.Layout(mk, 8, 3, 2), B, full)


@pytest.mark.parametrize("B", [1 << 28, (1 << 28) - 2, 256 * 10**6])
def test_from_buckets_plan_exact_cover_8b(B):
    m = emu.Model(*EIGHT_B)
    for src, dst in ((emu.Layout(m, 4, 1), emu.Layout(m, 4, 1)), (emu.Layout(m, 2, 2), emu.Layout(m, 4, 1))):
        plan = emu.Plan(src, dst, src_bucket_bytes=B)
        base = emu.Plan(src, dst)
        nb, sb = base.bucket_layout(0, B, -1)
        assert plan.info["n_src_tensors"] == nb
        assert plan.info["bytes_read"] == base.info["bytes_read"] and plan.info["bytes_written"] == base.info["bytes_written"]
        exact_cover(plan)
        if B % 16 == 0:
            assert plan.info["n_general_segments"] == 0


def test_from_buckets_plan_reports_no_aliases():
    """A receiver plan's source side is the bucket list: no destination tensor is a byte copy of a source
    tensor any more, so none is reported as one (the plain plan of the same layouts reports 30)."""
    m = emu.Model(*TINY)
    a, b = emu.Layout(m, 2, 2), emu.Layout(m, 2, 1)
    assert emu.Plan(a, b).info["n_alias_tensors"] == 30
    p = emu.Plan(a, b, src_bucket_bytes=1 << 16)
    assert p.info["n_alias_tensors"] == 0 and p.info["alias_bytes"] == 0 and p.info["aliased"] == 0
    assert all(d["alias"] == -1 for d in p.tensors(1))


def test_from_buckets_plan_errors():
    m = emu.Model(*TINY)
    lib = emu.load()
    a, b, h = emu.Layout(m, 1, 1).c(), emu.Layout(m, 2, 1).c(), ctypes.c_void_p()
    f, fb = emu.Layout(m, 1, 1, 0, "fp32").c(), emu.Layout(m, 2, 1, 0, "bf16").c()
    assert lib.emu_plan_from_buckets(ctypes.byref(a), ctypes.byref(b), 0, ctypes.byref(h)) == -6
    assert lib.emu_plan_from_buckets(ctypes.byref(a), ctypes.byref(b), 3, ctypes.byref(h)) == -6
    assert lib.emu_plan_from_buckets(ctypes.byref(f), ctypes.byref(fb), 6, ctypes.byref(h)) == -6  # fp32 source
    assert lib.emu_plan_from_buckets(ctypes.byref(f), ctypes.byref(fb), 8, ctypes.byref(h)) == 0
    assert lib.emu_plan_free(h) == 0
    assert lib.emu_plan_from_buckets(None, ctypes.byref(b), 64, ctypes.byref(h)) == -1
    with pytest.raises(ValueError):
        emu.Plan(emu.Layout(m, 1, 1), emu.Layout(m, 2, 1), bucket_bytes=64, src_bucket_bytes=64)


# ------------------------------------------------------------------------------------------------
# element-converting reshard (fp32 training state <-> bf16 generation weights)
# ------------------------------------------------------------------------------------------------

@pytest.mark.parametrize("pair", [("fp32", "bf16"), ("bf16", "fp32")])
def test_converting_plan_matches_oracle(pair):
    a, b = pair
    mm = emu.Model(*MICRO)
    lays_a = [emu.Layout(mm, tp, pp, pad, a, q, g) for tp, pp, pad, (q, g) in
              itertools.product((1, 4), (1, 2), (0, 2), sorted(FMT)[:2])]
    lays_b = [emu.Layout(mm, tp, pp, pad, b, q, g) for tp, pp, pad, (q, g) in
              itertools.product((2, 4), (1, 4), (0, 2), sorted(FMT)[1:3])]
    full = full_model(o_layout(lays_a[0]).model, 17, a)
    for src in lays_a:
        for dst in lays_b:
            p = check_pair(src, dst, full)
            assert p.info["converts"] == (1 if a == "fp32" else 2)
    m = emu.Model(*TINY)
    check_pair(emu.Layout(m, 2, 2, 0, a), emu.Layout(m, 1, 1, 128, b))
    check_fused(emu.Layout(m, 2, 1, 0, a), emu.Layout(m, 1, 2, 0, b), 65536 + 8)


def test_converting_plan_bytes_8b():
    m = emu.Model(*EIGHT_B)
    p = emu.Plan(emu.Layout(m, 4, 1, 0, "fp32"), emu.Layout(m, 2, 2, 0, "bf16"))
    # every bf16 destination element reads one fp32 source element
    assert p.info["bytes_written"] == 16_061_054_976 and p.info["bytes_read"] == 2 * 16_061_054_976
    assert p.info["converts"] == 1 and p.info["n_general_segments"] == 0
    exact_cover(p)


# ------------------------------------------------------------------------------------------------
# KV-head replication (tp > KV heads) and uneven pipeline stages
# ------------------------------------------------------------------------------------------------



def test_kv_replication_and_uneven_pp_match_oracle():
    m = emu.Model(*MICRO_KV)
    lays = [emu.Layout(m, tp, pp, pad, "bf16", q, g)
            for tp, pp, pad, (q, g) in itertools.product((1, 2, 4, 8), (1, 2, 3), (0, 2), sorted(FMT)[:2])]
    full = full_model(o_layout(lays[0]).model, 23)
    for i, src in enumerate(lays):
        for dst in lays[i % 4::4]:
            check_pair(src, dst, full)


def test_kv_replication_8b_tp16():
    """Llama-8B shapes at TP16 (each of the 8 KV heads held by two ranks) and an uneven 32-layer PP3."""
    m = emu.Model(*EIGHT_B)
    p = emu.Plan(emu.Layout(m, 2, 2), emu.Layout(m, 16, 1, 128))
    exact_cover(p)
    descs = p.tensors(1)
    qkv = [d for d in descs if d["kind"] == "qkv"]
    assert qkv[0]["shape"] == ((32 // 16 + 2) * 128, 4096)
    p3 = emu.Plan(emu.Layout(m, 4, 1), emu.Layout(m, 2, 3))
    exact_cover(p3)
    layers = [sorted({d["layer"] for d in p3.tensors(1) if d["rank"] == r and d["layer"] >= 0}) for r in (0, 2, 4)]
    assert layers == [list(range(0, 11)), list(range(11, 22)), list(range(22, 32))]


def test_plan_offsets_beyond_4gib():
    """The one-layer 266,240 x 8192 fp32 vocabulary model: destination shards, segment runs and source
    offsets pass 2^32 bytes; the map covers every destination byte once (exact cover on the host)."""
    from tests.shapes import HUGE_VOCAB

    m = emu.Model(*HUGE_VOCAB)
    plan = emu.Plan(emu.Layout(m, 1, 1, 0, "fp32"), emu.Layout(m, 2, 1, 0, "fp32"))
    segs = plan.segments()
    assert max(g["run"] for g in segs) > 1 << 32
    assert max(g["src_offset"] for g in segs) >= 1 << 32
    dd = plan.tensors(1)
    cover = {}
    for g in segs:
        cover[g["dst_tensor"]] = cover.get(g["dst_tensor"], 0) + g["rows"] * g["run"]
    assert all(cover[i] == d["bytes"] for i, d in enumerate(dd))
    assert plan.info["bytes_written"] == sum(d["bytes"] for d in dd) > 2 * (1 << 32)


# Llama-shaped 70B and 405B decoders (L, H, heads, head_dim, KV heads, MLP, vocab): host-only plans
SEVENTY_B = (80, 8192, 64, 128, 8, 28672, 128256)
FOUR_O_FIVE_B = (126, 16384, 128, 128, 8, 53248, 128256)


def test_large_model_plans():
    """Plans beyond one GPU's memory compile and stay exact: the 70B decoder TP8 PP1 -> TP4 PP2 (141 GB of
    shards, about 18M tiles) covers every destination byte once, with the oracle's per-rank inventory;
    the 405B decoder TP8 PP2 -> TP16 PP1 (KV heads replicated to two ranks each; about 106M tiles)
    reads and writes exactly its destination shards, whose sizes are the oracle's."""
    m70 = emu.Model(*SEVENTY_B)
    a, b = emu.Layout(m70, 8, 1), emu.Layout(m70, 4, 2)
    plan = emu.Plan(a, b)
    exact_cover(plan)
    ob = o_layout(b)
    want = [(r, s.kind, s.layer, tuple(s.shape), s.numel * ob.esize)
            for r, specs in enumerate(oracle.rank_inventory(ob)) for s in specs]
    got = [(d["rank"], d["kind"], d["layer"], tuple(d["shape"]), d["bytes"]) for d in plan.tensors(1)]
    assert got == want
    assert plan.info["bytes_read"] == plan.info["bytes_written"] == sum(w[4] for w in want) == 141_115_326_464
    assert plan.info["n_tiles"] * plan.info["tile_bytes"] >= plan.info["bytes_written"]

    m405 = emu.Model(*FOUR_O_FIVE_B)
    a, b = emu.Layout(m405, 8, 2), emu.Layout(m405, 16, 1)
    plan = emu.Plan(a, b)
    ob = o_layout(b)
    dst = sum(s.numel * ob.esize for specs in oracle.rank_inventory(ob) for s in specs)
    assert plan.info["bytes_read"] == plan.info["bytes_written"] == plan.info["dst_bytes"] == dst
    assert plan.info["n_tiles"] > 1 << 26 and plan.info["zero_fill_bytes"] == 0


# ------------------------------------------------------------------------------------------------
# host-side pointer-table checks (emu_check_tables / emu_check_bucket_tables)
# ------------------------------------------------------------------------------------------------

def _packed(sizes, base, gap=256):
    """Addresses of buffers laid out back to back from `base`, each start rounded up to `gap`."""
    out, a = [], base
    for n in sizes:
        out.append(a)
        a = (a + n + gap - 1) // gap * gap
    return out


def test_check_tables_accepts_disjoint_and_rejects_each_fault():
    m = emu.Model(*MICRO)
    plan = emu.Plan(emu.Layout(m, 2, 2, 2), emu.Layout(m, 4, 1, 2))
    ss = [d["bytes"] for d in plan.tensors(0)]
    ds = [d["bytes"] for d in plan.tensors(1)]
    src, dst = _packed(ss, 1 << 20), _packed(ds, 1 << 30)
    plan.check_tables(src, dst)
    plan.check_tables(src, _packed(ds, 1 << 30, gap=16))       # abutting destinations are fine
    aliased = list(src)
    aliased[1] = aliased[0]                                     # sources may alias each other
    plan.check_tables(aliased, dst)
    cases = [
        ([0] + src[1:], dst, emu.STATUS_CODE["EMU_ERR_NULL"]),
        (src, dst[:3] + [dst[3] + 8] + dst[4:], emu.STATUS_CODE["EMU_ERR_ALIGN"]),
        (src, dst[:1] + [dst[0] + 16] + dst[2:], emu.ERR_OVERLAP),          # destination over destination
        (src, [src[2] + 16] + dst[1:], emu.ERR_OVERLAP),                    # destination inside a source
        ([dst[5] - 16] + src[1:], dst, emu.ERR_OVERLAP),                    # source reaching into a destination
    ]
    for s_, d_, code in cases:
        with pytest.raises(emu.EmuError) as e:
            plan.check_tables(s_, d_)
        assert e.value.code == code, e.value


def test_check_tables_sweep_matches_pairwise_brute_force():
    """Random tables (aligned ranges placed at random in windows from 2x to 3000x their total size, so
    that both outcomes are common): the library's sorted sweep reports an overlap exactly when some pair
    of ranges with at least one destination intersects."""
    import random

    m = emu.Model(*MICRO)
    plan = emu.Plan(emu.Layout(m, 1, 1), emu.Layout(m, 2, 1))
    ss = [d["bytes"] for d in plan.tensors(0)]
    ds = [d["bytes"] for d in plan.tensors(1)]
    rng = random.Random(3)
    seen = {0: 0, emu.ERR_OVERLAP: 0}
    for _ in range(300):
        window = int((sum(ss) + sum(ds)) * 10 ** rng.uniform(0.3, 3.5))
        src = [0x10000 + 16 * rng.randrange(window // 16) for _ in ss]
        dst = [0x10000 + 16 * rng.randrange(window // 16) for _ in ds]
        ranges = [(a, a + n, False) for a, n in zip(src, ss)] + [(a, a + n, True) for a, n in zip(dst, ds)]
        clash = any(x[0] < y[1] and y[0] < x[1] and (x[2] or y[2])
                    for i, x in enumerate(ranges) for y in ranges[i + 1:])
        try:
            plan.check_tables(src, dst)
            rc = 0
        except emu.EmuError as e:
            rc = e.code
        assert rc == (emu.ERR_OVERLAP if clash else 0)
        seen[rc] += 1
    assert min(seen.values()) > 20


def test_check_bucket_tables():
    m = emu.Model(*TINY)
    plan = emu.Plan(emu.Layout(m, 1, 1), emu.Layout(m, 2, 1))
    B = 100_000
    ts = [d["bytes"] for d in plan.tensors(1)]
    bs = []
    for r in range(plan.info["n_dst_ranks"]):
        nb, sb = plan.bucket_layout(1, B, r)
        bs += [min(B, sb - k * B) for k in range(nb)]
    tp, bp = _packed(ts, 1 << 24), _packed(bs, 1 << 32, gap=16)
    plan.check_bucket_tables(1, B, tp, bp)
    with pytest.raises(emu.EmuError) as e:
        plan.check_bucket_tables(1, B, tp, bp[:2] + [bp[2] - 16] + bp[3:])   # bucket 2 starts inside bucket 1
    assert e.value.code == emu.ERR_OVERLAP
    with pytest.raises(emu.EmuError) as e:
        plan.check_bucket_tables(1, B, tp, [tp[4]] + bp[1:])                 # a bucket over a tensor
    assert e.value.code == emu.ERR_OVERLAP
    with pytest.raises(emu.EmuError) as e:
        plan.check_bucket_tables(1, 0, tp, bp)
    assert e.value.code == emu.STATUS_CODE["EMU_ERR_BUCKET"]


def test_layout_validation_and_inventory_match_oracle_random():
    """Random small models and layouts, valid or not (tp up to 8 with and without KV replication, pp up
    to L + 1, uneven stages, pad multiples, both formats, both element types): emu_layout_check accepts
    exactly the layouts oracle.check_layout accepts, and for those the library's per-rank tensor inventory
    (rank, kind, layer, shape, bytes, canonical order) is the oracle's."""
    import random

    rng = random.Random(17)
    seen = {True: 0, False: 0}
    for _ in range(500):
        nH = rng.choice([2, 4, 6, 8])
        G = rng.choice([g for g in (1, 2, 3, 4, 8) if nH % g == 0])
        L = rng.randint(1, 5)
        shape = (L, rng.choice([8, 16, 24]), nH, rng.choice([2, 4]), G, rng.choice([6, 8, 16, 24]),
                 rng.choice([8 * rng.randint(1, 5), rng.randint(6, 40)]))
        args = (rng.choice([1, 1, 2, 2, 3, 4, 8]), rng.randint(1, L + 1), rng.choice([0, 0, 1, 2, 3]),
                rng.choice(["bf16", "fp32"]), rng.choice(["interleaved", "separate"]), rng.choice(["block", "separate"]))
        lay = emu.Layout(emu.Model(*shape), *args)
        ol = o_layout(lay)
        try:
            oracle.check_layout(ol)
            valid = True
        except oracle.LayoutError:
            valid = False
        assert (emu.layout_check(lay) == 0) == valid, (shape, args)
        seen[valid] += 1
        if not valid:
            continue
        got = [(d["rank"], d["kind"], d["layer"], tuple(d["shape"]), d["bytes"]) for d in emu.Plan(lay, lay).tensors(0)]
        want = [(r, s.kind, s.layer, tuple(s.shape), s.numel * ol.esize)
                for r, specs in enumerate(oracle.rank_inventory(ol)) for s in specs]
        assert got == want, (shape, args)
    assert min(seen.values()) > 100, seen


def test_binding_rejects_unknown_format_names():
    """A misspelt format or dtype must not silently select another format."""
    m = emu.Model(*TINY)
    for kw in ({"qkv": "interleave"}, {"mlp": "interleaved"}, {"dtype": "fp16"}):
        with pytest.raises(ValueError):
            emu.Layout(m, 1, 1, **kw)
    assert emu.Layout(m, 1, 1, 0, "fp32", "separate", "separate").c().mlp_format == 1


def test_binding_refuses_tables_the_kernels_would_overrun():
    """The binding checks pointer tables on the host before any library call: int64, exactly the
    entries the plan indexes, contiguous, on the device."""
    import torch

    m = emu.Model(*TINY)
    plan = emu.Plan(emu.Layout(m, 1, 1), emu.Layout(m, 2, 1))
    ns, nd = plan.info["n_src_tensors"], plan.info["n_dst_tensors"]
    ws = torch.zeros(plan.info["workspace_bytes"], dtype=torch.uint8)
    ok_s, ok_d = torch.zeros(ns, dtype=torch.int64), torch.zeros(nd, dtype=torch.int64)
    cases = [
        (lambda: plan.reshard(ws, ok_s[:-1], ok_d), "entries"),
        (lambda: plan.reshard(ws, ok_s, torch.zeros(nd + 1, dtype=torch.int64)), "entries"),
        (lambda: plan.reshard(ws, ok_s.to(torch.int32), ok_d), "int64"),
        (lambda: plan.reshard(ws, [0] * ns, ok_d), "int64"),
        (lambda: plan.reshard(ws, torch.zeros(2 * ns, dtype=torch.int64)[::2], ok_d), "contiguous"),
        (lambda: plan.reshard(ws, ok_s, ok_d), "device"),
        (lambda: plan.pack(ws, 1, 1 << 16, ok_d, ok_d), "entries"),
        (lambda: plan.unpack(ws, 1, 1 << 16, ok_d, ok_d), "entries"),
        (lambda: plan.pack(ws, 2, 1 << 16, ok_d, ok_d), "side"),
        (lambda: plan.unpack(ws, 1, -2, ok_d, ok_d), "positive"),
    ]
    for call, word in cases:
        with pytest.raises(ValueError) as e:
            call()
        assert word in str(e.value), (word, str(e.value))


def _ws_tail_tables(plan):
    """Split the tail of plan.workspace_image() into each side's device-built tables (stream offsets,
    rank records, 4 KB chunk map), which close the workspace in that order, 256-byte aligned each."""
    img = plan.workspace_image()
    assert len(img) == plan.info["workspace_bytes"]
    a = lambda x: (x + 255) // 256 * 256
    C = 4096
    shapes = []
    for side in (0, 1):
        descs = plan.tensors(side)
        nranks = plan.info["n_src_ranks" if side == 0 else "n_dst_ranks"]
        rank_bytes = [0] * nranks
        for d in descs:
            rank_bytes[d["rank"]] += d["bytes"]
        nch = sum(-(-b // C) for b in rank_bytes)
        nmap = -(-nch // 8) * 8
        shapes.append((descs, nranks, rank_bytes, nmap))
    off = len(img) - sum(a(len(d) * 8) + a(n * 32) + a(m * 4) for d, n, _, m in shapes)
    assert off > 0
    out = []
    for descs, nranks, rank_bytes, nmap in shapes:
        so = np.frombuffer(img, np.uint64, len(descs), off); off += a(len(descs) * 8)
        ri = np.frombuffer(img, np.uint64, nranks * 4, off).reshape(nranks, 4); off += a(nranks * 32)
        cm = np.frombuffer(img, np.uint32, nmap, off); off += a(nmap * 4)
        out.append((descs, rank_bytes, so, ri, cm))
    assert off == len(img)
    return out


def _check_stream_tables(plan):
    C = 4096
    for descs, rank_bytes, so, ri, cm in _ws_tail_tables(plan):
        ranks = [d["rank"] for d in descs]
        assert ranks == sorted(ranks)
        first_chunk, end = 0, 0
        for r, rb in enumerate(rank_bytes):
            idx = [i for i, q in enumerate(ranks) if q == r]
            end += len(idx)
            pos = 0
            for i in idx:  # stream offsets: the tensors of a rank back to back, in global order
                assert so[i] == pos == descs[i]["stream_offset"]
                pos += descs[i]["bytes"]
            assert pos == rb
            nch = -(-rb // C)
            assert list(ri[r]) == [first_chunk, rb, end, 0]
            for j in range(nch):  # chunk j starts in the last tensor of the rank whose offset is <= j*C
                owner = max(i for i in idx if so[i] <= j * C)
                assert cm[first_chunk + j] == (r << 20) | owner, (r, j)
                assert so[owner] <= j * C < (so[owner] + descs[owner]["bytes"] if owner != idx[-1] else rb)
            first_chunk += nch
        assert (cm[first_chunk:] == 0xFFFFFFFF).all() and len(cm) - first_chunk < 8


def test_workspace_image_stream_tables():
    """The tables the upload derives on the device, as the host computes them (the GPU tests compare the
    uploaded workspace with this image byte for byte): stream offsets, rank records and the chunk map,
    against the tensor inventory. Covers several ranks, uneven PP, KV replication and fused plans'
    bucket sides, including 30-byte buckets (many tensors start inside one 4 KB chunk)."""
    m = emu.Model(*TINY)
    _check_stream_tables(emu.Plan(emu.Layout(m, 1, 1), emu.Layout(m, 2, 1)))
    _check_stream_tables(emu.Plan(emu.Layout(m, 2, 2, 128), emu.Layout(m, 1, 1, 0, "bf16", "separate", "separate")))
    _check_stream_tables(emu.Plan(emu.Layout(m, 2, 1), emu.Layout(m, 1, 2), bucket_bytes=(1 << 16) - 2))
    mk = emu.Model(*MICRO_KV)
    _check_stream_tables(emu.Plan(emu.Layout(mk, 8, 3, 2), emu.Layout(mk, 2, 1)))
    _check_stream_tables(emu.Plan(emu.Layout(mk, 1, 1), emu.Layout(mk, 4, 2), bucket_bytes=30))


def test_workspace_image_tile_map():
    """The head of the workspace image: the segment records (80 bytes each, the first map index of the
    segment's tiles in the last 8), their tile counts, and the tile map the upload derives on the device
    -- each segment's index on its own tiles, copy segments' tiles first, each section padded with
    0xFFFFFFFF to a multiple of 8 entries, and every tile of the plan on the map exactly once."""
    a = lambda x: (x + 255) // 256 * 256
    m = emu.Model(*TINY)
    for plan in (emu.Plan(emu.Layout(m, 1, 1), emu.Layout(m, 2, 1)),
                 emu.Plan(emu.Layout(m, 2, 2, 128), emu.Layout(m, 1, 1, 0, "bf16", "separate", "separate")),
                 emu.Plan(emu.Layout(m, 1, 1), emu.Layout(m, 2, 2, 384)),  # zero-filled pad rows
                 emu.Plan(emu.Layout(m, 2, 1), emu.Layout(m, 1, 2), bucket_bytes=(1 << 16) - 2)):
        img = plan.workspace_image()
        n = plan.info["n_segments"]
        segs = plan.segments()
        tile0 = np.frombuffer(img, np.uint64, n * 10).reshape(n, 10)[:, 9]
        counts = np.frombuffer(img, np.uint32, n, a(n * 80))
        assert counts.sum() == plan.info["n_tiles"]
        zero = np.array([s["src_tensor"] < 0 for s in segs])
        n_copy, n_zero = int(counts[~zero].sum()), int(counts[zero].sum())
        z0 = -(-n_copy // 8) * 8
        n_map = z0 + -(-n_zero // 8) * 8
        tm = np.frombuffer(img, np.uint32, n_map, a(n * 80) + a(n * 4))
        want = np.full(n_map, 0xFFFFFFFF, np.uint32)
        nxt = [0, z0]
        assert n_zero > 0 or plan.info["zero_fill_bytes"] == 0
        for i in range(n):  # tiles in segment order within each section
            sec = int(zero[i])
            assert tile0[i] == nxt[sec]
            want[nxt[sec]:nxt[sec] + counts[i]] = i
            nxt[sec] += int(counts[i])
        assert nxt == [n_copy, z0 + n_zero]
        assert np.array_equal(tm, want)


def test_sender_and_receiver_plans_compose():
    """The transport end to end on the host: a sender's fused plan L -> L' into buckets of B, then a
    receiver plan L' -> L'' out of those buckets, gives the oracle's direct reshard L -> L'' (the
    composition through an intermediate layout, section 6.1's T_sub route, with the contiguous transfer
    of section 6.2 between the two halves)."""
    m = emu.Model(*MICRO)
    lays = [emu.Layout(m, tp, pp, pad, "bf16", q, g) for tp, pp, pad, (q, g) in
            ((1, 1, 0, ("interleaved", "block")), (2, 2, 2, ("separate", "separate")), (4, 1, 0, ("interleaved", "separate")),
             (2, 4, 2, ("separate", "block")))]
    full = full_model(o_layout(lays[0]).model, 31)
    for a, b, c in itertools.permutations(lays, 3):
        oa, oc = o_layout(a), o_layout(c)
        shards = oracle.shard(full, oa)
        flat = [np.ascontiguousarray(x).reshape(-1).view(np.uint8) for rank in shards for x in rank]
        for B in (6, 64, 1000):
            send = emu.Plan(a, b, bucket_bytes=B)
            buckets = run_plan(send.segments(), flat, [d["bytes"] for d in send.tensors(1)])
            recv = emu.Plan(b, c, src_bucket_bytes=B)
            assert [d["bytes"] for d in recv.tensors(0)] == [x.size for x in buckets]
            got = run_plan(recv.segments(), buckets, [d["bytes"] for d in recv.tensors(1)])
            want = [np.ascontiguousarray(x).reshape(-1).view(np.uint8) for rank in oracle.reshard(shards, oa, oc)
                    for x in rank]
            for i, (g, w) in enumerate(zip(got, want)):
                assert np.array_equal(g, w), (a, b, c, B, i)


def test_shard_set_and_bucket_set_refuse_wrong_buffers():
    """The binding's checks on a caller's own tensors and buckets, before any library call: count, byte
    size, contiguity and 16-byte alignment (on host tensors, so that the device check comes last)."""
    import torch

    m = emu.Model(*TINY)
    plan = emu.Plan(emu.Layout(m, 1, 1), emu.Layout(m, 2, 1))
    descs = plan.tensors(1)
    good = [torch.empty(d["bytes"] // 2, dtype=torch.bfloat16) for d in descs]
    with pytest.raises(ValueError, match="tensors"):
        plan.shard_set(1, good[:-1])
    bad = list(good)
    bad[3] = torch.empty(descs[3]["bytes"] // 2 + 1, dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="bytes, the plan needs"):
        plan.shard_set(1, bad)
    bad = list(good)
    bad[2] = torch.empty(2, descs[2]["bytes"] // 2, dtype=torch.bfloat16)[:, : descs[2]["bytes"] // 4].t()
    with pytest.raises(ValueError):  # a strided view: wrong size or not contiguous
        plan.shard_set(1, bad)
    raw = torch.empty(descs[0]["bytes"] + 64, dtype=torch.uint8)
    off = (16 - raw.data_ptr() % 16) % 16 + 2
    bad = list(good)
    bad[0] = raw[off:off + descs[0]["bytes"]]
    with pytest.raises(emu.EmuError):
        plan.shard_set(1, bad)
    with pytest.raises(ValueError, match="device"):
        plan.shard_set(1, good)
    info = plan.bucket_info(1, 1 << 16)
    bufs = [torch.empty(b["bytes"], dtype=torch.uint8) for b in info]
    with pytest.raises(ValueError, match="buckets"):
        plan.bucket_set(1, 1 << 16, bufs[1:])
    bad = list(bufs)
    bad[-1] = torch.empty(info[-1]["bytes"] + 2, dtype=torch.uint8)
    with pytest.raises(ValueError, match="bytes, the plan needs"):
        plan.bucket_set(1, 1 << 16, bad)
    with pytest.raises(ValueError, match="device"):
        plan.bucket_set(1, 1 << 16, bufs)
