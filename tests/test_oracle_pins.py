"""Pins of the CPU oracle against facts that do not come from the oracle itself.

* brute force: every destination element, located by the pure-Python coordinate formulas, must hold the
  source element with the same logical coordinate (exhaustive over micro-model layout pairs);
* invariants: unshard(shard(X)) == X, Merge o Split == identity, composition through an intermediate
  layout (the reward-inference example of section 6.1: TP4 PP8 -> four TP4 PP2 units -> TP8 PP2),
  reshard to the same layout == copy;
* special cases: a TP1 PP1 layout with separate formats is literally the logical model; with fused
  formats it equals a closed form written with reshapes;
* provenance tags: every element written exactly once, norm replicas read from TP rank 0, pad rows
  zero-filled and never read.
"""
import itertools

import numpy as np
import pytest

import oracle
from oracle import coords
from synthetic import host_tensor
from tests.shapes import MICRO, MICRO8, MICRO_KV, TINY

FORMATS = [("interleaved", "block"), ("separate", "separate"), ("interleaved", "separate"),
           ("separate", "block")]


def micro_layouts(shape=MICRO, tps=(1, 2, 4), pps=(1, 2, 4), pads=(0, 2), dtype="fp32"):
    m = oracle.Model(*shape)
    out = []
    for tp, pp, pad, (q, g) in itertools.product(tps, pps, pads, FORMATS):
        out.append(oracle.Layout(m, tp, pp, pad, dtype, q, g))
    return out


def random_full(model, seed=7, dtype="bf16"):
    full = {}
    for i, (_, key, shape, kind) in enumerate(oracle.logical_tensors(model)):
        dist = "norm" if kind.endswith("norm") else "weight"
        full[key] = host_tensor(seed, (0, i), shape, dist, dtype)
    return full


def assert_sets_equal(a, b):
    assert len(a) == len(b)
    for ra, rb in zip(a, b):
        assert len(ra) == len(rb)
        for x, y in zip(ra, rb):
            assert x.shape == y.shape and x.dtype == y.dtype
            assert np.array_equal(x.view(np.uint8), y.view(np.uint8))


# ------------------------------------------------------------------------------------------------
# brute force with provenance tags
# ------------------------------------------------------------------------------------------------

_IDS = {}


def ids_of(lay):
    if lay not in _IDS:
        _IDS[lay] = coords.element_ids(lay)
    return _IDS[lay]


# tag type, replica mark and pad sentinel per element type (bf16 tags need fewer than 2^15 elements)
TAGS = {"fp32": (np.uint32, 0x8000_0000, 0xFFFF_FFFF), "bf16": (np.uint16, 0x8000, 0xFFFF)}


def tagged_source(lay):
    """Source shards whose elements carry (logical id + 1); pad rows hold a sentinel that must never be
    read; every replica of a logical element held by an earlier rank (norms on TP ranks > 0, replicated
    KV heads past their first rank) carries a marked tag that must never be copied."""
    dt, replica, sentinel = TAGS[lay.dtype]
    out = []
    seen = set()
    for r, (specs, ids) in enumerate(zip(oracle.rank_inventory(lay), ids_of(lay))):
        per = []
        for s, i in zip(specs, ids):
            a = np.array(i, dtype=np.int64)
            assert a.max() + 1 < replica
            tag = np.where(a < 0, sentinel, a + 1)
            rep = np.array([x >= 0 and x in seen for x in i], dtype=bool)
            tag = np.where(rep, tag | replica, tag)
            seen.update(x for x in i if x >= 0)
            per.append(tag.astype(dt).reshape(s.shape))
        out.append(per)
    return out


def expected_tags(lay):
    dt = TAGS[lay.dtype][0]
    out = []
    for specs, ids in zip(oracle.rank_inventory(lay), ids_of(lay)):
        out.append([np.where(np.array(i) < 0, 0, np.array(i) + 1).astype(dt).reshape(s.shape)
                    for s, i in zip(specs, ids)])
    return out


MICRO_LAYOUTS = micro_layouts()
# KV replication (tp up to 4x the KV heads) and uneven pipeline stages (L = 3)
KV_LAYOUTS = micro_layouts(MICRO_KV, tps=(1, 2, 4, 8), pps=(1, 2, 3), pads=(0, 2), dtype="fp32")


@pytest.mark.parametrize("src", MICRO_LAYOUTS, ids=lambda l: f"tp{l.tp}pp{l.pp}m{l.pad}{l.qkv[0]}{l.mlp[0]}")
def test_brute_force_all_pairs(src):
    s = tagged_source(src)
    for dst in MICRO_LAYOUTS:
        got = oracle.reshard(s, src, dst)
        assert_sets_equal(got, expected_tags(dst))


MICRO_LAYOUTS_BF16 = micro_layouts(dtype="bf16")


@pytest.mark.parametrize("src", MICRO_LAYOUTS_BF16[::4], ids=lambda l: f"tp{l.tp}pp{l.pp}m{l.pad}{l.qkv[0]}{l.mlp[0]}")
def test_brute_force_bf16_tags(src):
    """The same with 16-bit tags on bf16 layouts: the oracle moves 2-byte elements as they are."""
    s = tagged_source(src)
    for dst in MICRO_LAYOUTS_BF16[1::3]:
        got = oracle.reshard(s, src, dst)
        assert_sets_equal(got, expected_tags(dst))


@pytest.mark.parametrize("src", KV_LAYOUTS[::2], ids=lambda l: f"tp{l.tp}pp{l.pp}m{l.pad}{l.qkv[0]}{l.mlp[0]}")
def test_brute_force_kv_replication_and_uneven_pp(src):
    s = tagged_source(src)
    for dst in KV_LAYOUTS:
        got = oracle.reshard(s, src, dst)
        assert_sets_equal(got, expected_tags(dst))


def test_element_ids_cover_model_once():
    """The id formulas cover every logical element, and only norms and replicated KV heads appear on more
    than one rank."""
    for lay in MICRO_LAYOUTS[::5] + KV_LAYOUTS[::7]:
        total = sum(int(np.prod(s)) if len(s) > 1 else s[0] for _, _, s, _ in oracle.logical_tensors(lay.model))
        count = np.zeros(total, dtype=np.int64)
        for r, (specs, ids) in enumerate(zip(oracle.rank_inventory(lay), ids_of(lay))):
            for spec, i in zip(specs, ids):
                a = np.array([x for x in i if x >= 0], dtype=np.int64)
                np.add.at(count, a, 1)
                if not spec.kind.endswith("norm") and spec.kind not in ("qkv", "k", "v"):
                    assert len(set(a.tolist())) == a.size
        assert count.min() == 1
        if lay.tp <= lay.model.G:
            # without KV replication only the norms are held more than once (once per TP rank)
            assert count.max() == lay.tp


# ------------------------------------------------------------------------------------------------
# invariants on random data
# ------------------------------------------------------------------------------------------------

@pytest.mark.parametrize("shape", [MICRO, TINY], ids=["micro", "tiny"])
def test_unshard_shard_identity(shape):
    m = oracle.Model(*shape)
    full = random_full(m)
    tps = [t for t in (1, 2, 4) if m.G % t == 0]
    pps = [p for p in (1, 2, 4) if m.L % p == 0]
    for tp, pp, pad, (q, g) in itertools.product(tps, pps, (0, 2), FORMATS):
        lay = oracle.Layout(m, tp, pp, pad, "bf16", q, g)
        back = oracle.unshard(oracle.shard(full, lay), lay)
        assert back.keys() == full.keys()
        for k in full:
            assert np.array_equal(back[k], full[k]), (lay, k)


def test_tp1pp1_separate_is_the_logical_model():
    m = oracle.Model(*TINY)
    full = random_full(m)
    lay = oracle.Layout(m, 1, 1, 0, "bf16", "separate", "separate")
    (rank0,) = oracle.shard(full, lay)
    keys = [key for _, key, _, _ in oracle.logical_tensors(m)]
    # canonical order: embed, per layer [attn_norm, q, k, v, o, mlp_norm, gate, up, down], final, lm_head
    assert len(rank0) == len(keys)
    for a, k in zip(rank0, keys):
        assert np.array_equal(a, full[k])


def test_tp1pp1_fused_closed_form():
    m = oracle.Model(*TINY)
    full = random_full(m)
    lay = oracle.Layout(m, 1, 1)
    (rank0,) = oracle.shard(full, lay)
    specs = oracle.rank_inventory(lay)[0]
    qpg = m.nH // m.G
    for spec, a in zip(specs, rank0):
        pre = f"layers.{spec.layer}."
        if spec.kind == "qkv":
            q = full[pre + "q"].reshape(m.G, qpg * m.hd, m.H)
            k = full[pre + "k"].reshape(m.G, m.hd, m.H)
            v = full[pre + "v"].reshape(m.G, m.hd, m.H)
            assert np.array_equal(a, np.concatenate([q, k, v], axis=1).reshape(-1, m.H))
        if spec.kind == "gate_up":
            assert np.array_equal(a, np.concatenate([full[pre + "gate"], full[pre + "up"]]))


def test_column_and_row_parallel_reduce_to_split():
    """At PP1, separate formats, no pad: every shard is one piece of np.split along the sharded axis."""
    m = oracle.Model(*TINY)
    full = random_full(m)
    for tp in (1, 2):
        lay = oracle.Layout(m, tp, 1, 0, "bf16", "separate", "separate")
        sh = oracle.shard(full, lay)
        for t in range(tp):
            for spec, a in zip(oracle.rank_inventory(lay)[t], sh[t]):
                key = f"layers.{spec.layer}.{spec.kind}" if spec.layer >= 0 else spec.kind
                x = full[key]
                if spec.kind in ("o", "down"):
                    ref = np.split(x, tp, axis=1)[t]
                elif spec.kind.endswith("norm"):
                    ref = x
                else:
                    ref = np.split(x, tp, axis=0)[t]
                assert np.array_equal(a, ref), spec


@pytest.mark.parametrize("shape", [MICRO, TINY], ids=["micro", "tiny"])
def test_merge_split_roundtrip(shape):
    m = oracle.Model(*shape)
    full = random_full(m)
    tps = [t for t in (1, 2, 4) if m.G % t == 0]
    pps = [p for p in (1, 2, 4) if m.L % p == 0]
    lays = [oracle.Layout(m, tp, pp, pad, "bf16", q, g)
            for tp, pp, pad, (q, g) in itertools.product(tps, pps, (0, 2), FORMATS[:2])]
    for a in lays:
        sa = oracle.shard(full, a)
        for b in lays[::3]:
            assert_sets_equal(oracle.reshard(oracle.reshard(sa, a, b), b, a), sa)


def test_same_layout_is_a_copy():
    m = oracle.Model(*TINY)
    full = random_full(m)
    for lay in (oracle.Layout(m, 2, 2), oracle.Layout(m, 1, 1, 128)):
        s = oracle.shard(full, lay)
        assert_sets_equal(oracle.reshard(s, lay, lay), s)


def test_composition_through_t_sub_paper_example():
    """Section 6.1 example: a (TP4, PP8) unit is split into (TP4, PP2) units that merge into (TP8, PP2).
    Going through the intermediate layout must equal the direct reshard."""
    m = oracle.Model(*MICRO8)
    full = random_full(m)
    for pad in (0, 2):
        a = oracle.Layout(m, 4, 8, pad)
        b = oracle.Layout(m, 4, 2, pad)
        c = oracle.Layout(m, 8, 2, pad)
        sa = oracle.shard(full, a)
        two_phase = oracle.reshard(oracle.reshard(sa, a, b), b, c)
        assert_sets_equal(two_phase, oracle.reshard(sa, a, c))
        assert_sets_equal(two_phase, oracle.shard(full, c))


def test_reshard_equals_shard_of_full_on_tiny():
    """The tiny decoder's Split TP1 PP1 -> TP2 PP1 and its Merge back."""
    m = oracle.Model(*TINY)
    full = random_full(m)
    a, b = oracle.Layout(m, 1, 1), oracle.Layout(m, 2, 1)
    sa = oracle.shard(full, a)
    sb = oracle.reshard(sa, a, b)
    assert_sets_equal(sb, oracle.shard(full, b))
    assert_sets_equal(oracle.reshard(sb, b, a), sa)


# ------------------------------------------------------------------------------------------------
# layout validity
# ------------------------------------------------------------------------------------------------

def test_layout_validation():
    m = oracle.Model(*TINY)
    oracle.check_layout(oracle.Layout(m, 2, 2))
    oracle.check_layout(oracle.Layout(m, 4, 1))              # tp > KV heads: KV heads replicated
    with pytest.raises(oracle.LayoutError):
        oracle.check_layout(oracle.Layout(m, 3, 1))          # tp > KV heads, not a multiple of them
    with pytest.raises(oracle.LayoutError):
        oracle.check_layout(oracle.Layout(m, 1, 3))          # more stages than layers
    assert [list(oracle.stage_layers(oracle.Layout(oracle.Model(*MICRO), 1, 3), p)) for p in range(3)] == \
        [[0, 1], [2], [3]]
    m2 = oracle.Model(4, 16, 8, 2, 4, 12, 21)                # odd vocabulary
    with pytest.raises(oracle.LayoutError):
        oracle.check_layout(oracle.Layout(m2, 2, 1))
    oracle.check_layout(oracle.Layout(m2, 2, 1, pad=2))      # padding makes it valid
    assert oracle.padded_vocab(oracle.Layout(m2, 2, 1, pad=2)) == 24
    m3 = oracle.Model(4, 16, 8, 2, 4, 10, 20)                # MLP width 10
    with pytest.raises(oracle.LayoutError):
        oracle.check_layout(oracle.Layout(m3, 4, 1))
    with pytest.raises(oracle.LayoutError):
        oracle.reshard([], oracle.Layout(m, 1, 1), oracle.Layout(oracle.Model(*MICRO), 1, 1))
