"""Pins of the oracle's bucket pack/unpack and of its shard inventory sizes.

The stream and bucket rule (section 6.2: each shard is sent once as one contiguous buffer) is pinned by
its definition written independently here (byte concatenation + fixed-size cuts), by pack/unpack
round trips over awkward bucket sizes, and by hand-derived boundary positions on the 8B shapes.
"""
import os

import numpy as np
import pytest

import oracle
from synthetic import host_bytes
from tests.shapes import EIGHT_B, TINY

HERE = os.path.dirname(__file__)


def golden(name):
    vals = {}
    with open(os.path.join(HERE, "golden", name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                k, v = line.split()
                vals[k] = int(v)
    return vals


def test_inventory_matches_hand_derived_sizes():
    g = golden("llama8b_inventory.txt")
    m = oracle.Model(*EIGHT_B)
    assert sum(int(np.prod(s)) for _, _, s, _ in oracle.logical_tensors(m)) == g["logical_params"]

    def rank_bytes(lay):
        return [sum(s.numel for s in specs) * lay.esize for specs in oracle.rank_inventory(lay)]

    tp4 = oracle.Layout(m, 4, 1)
    rb = rank_bytes(tp4)
    assert sum(rb) == g["tp4pp1_total_bytes"] and set(rb) == {g["tp4pp1_rank_bytes"]}
    assert {len(x) for x in oracle.rank_inventory(tp4)} == {g["tp4pp1_rank_tensors"]}
    tp2 = oracle.Layout(m, 2, 2)
    rb = rank_bytes(tp2)
    assert rb == [g["tp2pp2_rank_bytes_p0"]] * 2 + [g["tp2pp2_rank_bytes_p1"]] * 2
    assert [len(x) for x in oracle.rank_inventory(tp2)] == [g["tp2pp2_rank_tensors_p0"]] * 2 + \
        [g["tp2pp2_rank_tensors_p1"]] * 2
    tp8 = oracle.Layout(m, 8, 4, pad=128)
    assert oracle.padded_vocab(tp8) == g["tp8pp4_pad128_vocab"]
    rb = rank_bytes(tp8)
    assert rb[0] == g["tp8pp4_pad128_rank_bytes_p0"] and rb[8] == g["tp8pp4_pad128_rank_bytes_p1"]
    assert rb[31] == g["tp8pp4_pad128_rank_bytes_p3"]


@pytest.mark.parametrize("B", [1, 2, 7, 16, 30, 1000, 4096, 10**6])
def test_pack_unpack_roundtrip(B):
    rng = np.random.default_rng(B)
    tensors = [rng.integers(0, 2**16, size=s, dtype=np.uint16) for s in [(3, 5), (16,), (7, 9), (1,), (40, 2)]]
    stream = b"".join(t.tobytes() for t in tensors)
    buckets = oracle.pack(tensors, B)
    assert len(buckets) == -(-len(stream) // B)
    assert all(b.size == B for b in buckets[:-1]) and 0 < buckets[-1].size <= B
    for k, b in enumerate(buckets):
        assert b.tobytes() == stream[k * B:(k + 1) * B]
    back = oracle.unpack(buckets, tensors)
    for a, b in zip(tensors, back):
        assert np.array_equal(a, b) and a.dtype == b.dtype and a.shape == b.shape


def test_unpack_rejects_wrong_sizes():
    t = [np.zeros((4, 4), np.uint16)]
    with pytest.raises(ValueError):
        oracle.unpack([np.zeros(10, np.uint8)], t)


def test_random_bytes_roundtrip_tiny_model():
    m = oracle.Model(*TINY)
    lay = oracle.Layout(m, 2, 1)
    for r, specs in enumerate(oracle.rank_inventory(lay)):
        tensors = [host_bytes(3, (r, j), s.numel * 2).view(np.uint16).reshape(s.shape) for j, s in enumerate(specs)]
        for B in (2**12, 2**12 - 2, 12345 * 2):
            back = oracle.unpack(oracle.pack(tensors, B), tensors)
            assert all(np.array_equal(a, b) for a, b in zip(tensors, back))


def _hand_stream_8b_tp2pp2(p):
    """(kind, bytes, row_bytes) of rank (t, p) of the 8B TP2 PP2 layout, written out by hand."""
    layer = [("attn_norm", 8192, 8192), ("qkv", 3072 * 4096 * 2, 8192), ("o", 4096 * 2048 * 2, 4096),
             ("mlp_norm", 8192, 8192), ("gate_up", 14336 * 4096 * 2, 8192), ("down", 4096 * 7168 * 2, 14336)]
    out = [("embed", 64128 * 4096 * 2, 8192)] if p == 0 else []
    out += layer * 16
    if p == 1:
        out += [("final_norm", 8192, 8192), ("lm_head", 64128 * 4096 * 2, 8192)]
    return out


@pytest.mark.parametrize("B,expect", [(2**28, {0: 4, 1: 1}), (256 * 10**6, {0: None, 1: 3}),
                                      (2**28 - 2, {0: 14, 1: 14})])
def test_mid_row_bucket_boundaries_8b(B, expect):
    """Bucket boundaries that cut a row, on the 8B TP2 PP2 destination of the padded-vocabulary case."""
    m = oracle.Model(*EIGHT_B)
    lay = oracle.Layout(m, 2, 2, pad=128)
    for p in (0, 1):
        hand = _hand_stream_8b_tp2pp2(p)
        specs = oracle.rank_inventory(lay)[p * 2]
        assert [(s.kind, s.numel * 2) for s in specs] == [(k, n) for k, n, _ in hand]
        total = sum(n for _, n, _ in hand)
        nb = oracle.bucket_count(total, B)
        offs = np.cumsum([0] + [n for _, n, _ in hand])
        mid = []
        for k in range(1, nb):
            pos = k * B
            i = int(np.searchsorted(offs, pos, side="right")) - 1
            kind, n, row = hand[i]
            if (pos - offs[i]) % row:
                mid.append(kind)
        if expect[p] is not None:
            assert len(mid) == expect[p], (p, mid)
        if B == 2**28:
            assert nb == 15 and set(mid) == {"down"}
            assert total - 14 * B == (257163264 if p == 0 else 257171456)
