"""Planted mistakes in the oracle must be caught by its pins.

Each test swaps in a plausible wrong version of one oracle step (on the CPU, through monkeypatch) and
checks that the brute-force tag pin or a closed-form pin fails. This guards the pins themselves: a pin
that cannot see a dropped term, a swapped operand or a wrong index is no pin.
"""
import numpy as np
import pytest

import oracle
import oracle.sharding as R
from tests.test_oracle_pins import MICRO_LAYOUTS, assert_sets_equal, expected_tags, tagged_source


def pins_fail():
    """Run the brute-force tag pin over a spread of layout pairs; True if any pair disagrees."""
    lays = MICRO_LAYOUTS[::7] + [MICRO_LAYOUTS[-1]]
    for src in lays:
        s = tagged_source(src)
        for dst in lays:
            try:
                assert_sets_equal(oracle.reshard(s, src, dst), expected_tags(dst))
            except AssertionError:
                return True
    return False


def test_unmutated_oracle_passes():
    assert not pins_fail()


def _wrap_shard(monkeypatch, kind, f):
    orig = R._shard_one

    def mutant(lay, k, layer, t, full):
        out = orig(lay, k, layer, t, full)
        return f(lay, out) if k == kind else out

    monkeypatch.setattr(R, "_shard_one", mutant)


def test_swapped_k_and_v_is_caught(monkeypatch):
    def swap(lay, out):
        m = lay.model
        qpg, hd = m.nH // m.G, m.hd
        b = out.reshape(-1, qpg + 2, hd, out.shape[-1]).copy()
        b[:, [qpg, qpg + 1]] = b[:, [qpg + 1, qpg]]
        return b.reshape(out.shape)
    _wrap_shard(monkeypatch, "qkv", swap)
    assert pins_fail()


def test_pad_rows_not_zeroed_is_caught(monkeypatch):
    orig = R._shard_one

    def mutant(lay, k, layer, t, full):
        out = orig(lay, k, layer, t, full)
        if k in ("embed", "lm_head") and lay.pad:
            rows = oracle.padded_vocab(lay) // lay.tp
            real = max(0, min(rows, lay.model.V - t * rows))
            out = out.copy()
            out[real:] = 1     # garbage instead of zeros in the pad rows
        return out
    monkeypatch.setattr(R, "_shard_one", mutant)
    assert pins_fail()


def test_row_split_instead_of_column_split_is_caught(monkeypatch):
    orig = R._shard_one

    def mutant(lay, k, layer, t, full):
        if k == "o":
            x = full[f"layers.{layer}.o"]
            return np.ascontiguousarray(np.split(x, lay.tp, axis=0)[t].reshape(x.shape[0], -1))
        return orig(lay, k, layer, t, full)
    monkeypatch.setattr(R, "_shard_one", mutant)
    assert pins_fail()


def test_norm_read_from_last_tp_rank_is_caught(monkeypatch):
    orig = R.rank_of

    def mutant(lay, t, p):
        return orig(lay, lay.tp - 1 if t == 0 else t, p)
    monkeypatch.setattr(R, "rank_of", mutant)
    assert pins_fail()


def test_gate_up_halves_swapped_is_caught(monkeypatch):
    def swap(lay, out):
        h = out.shape[0] // 2
        return np.concatenate([out[h:], out[:h]])
    _wrap_shard(monkeypatch, "gate_up", swap)
    assert pins_fail()


def test_off_by_one_group_in_interleaved_qkv_is_caught(monkeypatch):
    def shift(lay, out):
        return np.roll(out, out.shape[0] // max(1, lay.model.G // lay.tp), axis=0)
    _wrap_shard(monkeypatch, "qkv", shift)
    assert pins_fail()


def test_wrong_bucket_cut_is_caught():
    """A pack that drops the last partial bucket breaks the round trip."""
    tensors = [np.arange(10, dtype=np.uint16)]
    buckets = oracle.pack(tensors, 6)[:-1]
    with pytest.raises(ValueError):
        oracle.unpack(buckets, tensors)
