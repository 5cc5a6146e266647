"""Pins of the oracle's fp32 <-> bf16 conversion and of the converting reshard.

* a hand-derived table of round-to-nearest-even cases (tests/golden/bf16_rounding.txt);
* exhaustive: every one of the 65,536 bf16 bit patterns survives widening and narrowing unchanged
  (NaNs come back quieted);
* on finite values the result is the nearest bf16 (ties to even), checked against both neighbours in
  float64, and agrees with torch's CPU float32 -> bfloat16 cast;
* the converting reshard equals the same-type reshard followed by the conversion (the layout change
  and the element conversion commute) and equals shard(convert(full)).
"""
import os

import numpy as np
import pytest

import oracle
from oracle.convert import bf16_to_f32, f32_to_bf16
from tests.shapes import MICRO, TINY
from tests.test_oracle_pins import assert_sets_equal, random_full

HERE = os.path.dirname(__file__)


def test_golden_rounding_table():
    rows = []
    with open(os.path.join(HERE, "golden", "bf16_rounding.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                a, b = line.split()[:2]
                rows.append((int(a, 16), int(b, 16)))
    assert len(rows) >= 20
    x = np.array([a for a, _ in rows], dtype=np.uint32).view(np.float32)
    got = f32_to_bf16(x)
    for (a, b), g in zip(rows, got):
        assert int(g) == b, f"{a:08X}: got {int(g):04X}, want {b:04X}"


def test_every_bf16_pattern_round_trips():
    b = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    back = f32_to_bf16(bf16_to_f32(b))
    is_nan = ((b & 0x7FFF) > 0x7F80)
    assert np.array_equal(back[~is_nan], b[~is_nan])
    assert np.array_equal(back[is_nan], b[is_nan] | 0x0040)
    assert np.array_equal(bf16_to_f32(b).view(np.uint32) >> 16, b.astype(np.uint32))


def test_nearest_even_against_neighbours():
    rng = np.random.default_rng(5)
    u = rng.integers(0, 1 << 32, size=200_000, dtype=np.uint64).astype(np.uint32)
    x = u.view(np.float32)
    fin = np.isfinite(x) & (np.abs(x) < np.float32(3.38e38))
    x = x[fin]
    r = f32_to_bf16(x)
    down = (x.view(np.uint32) >> 16).astype(np.uint16)                     # truncation toward zero
    up = down + np.uint16(1)
    xd = bf16_to_f32(down).astype(np.float64)
    xu = bf16_to_f32(up).astype(np.float64)
    xv = x.astype(np.float64)
    dd, du = np.abs(xv - xd), np.abs(xu - xv)
    want = np.where(dd < du, down, np.where(du < dd, up, np.where(down % 2 == 0, down, up)))
    assert np.array_equal(r, want)


def test_agrees_with_torch_cpu_cast_on_finite_values():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(9)
    x = (rng.standard_normal(500_000) * np.exp(rng.uniform(-60, 60, 500_000))).astype(np.float32)
    x = x[np.isfinite(x)]
    t = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(f32_to_bf16(x), t)


@pytest.mark.parametrize("shape", [MICRO, TINY], ids=["micro", "tiny"])
def test_converting_reshard_commutes(shape):
    m = oracle.Model(*shape)
    full32 = random_full(m, seed=3, dtype="fp32")
    tps = [t for t in (1, 2, 4) if m.G % t == 0]
    for tp_s in tps:
        for tp_d in tps:
            a = oracle.Layout(m, tp_s, 1, 0, "fp32")
            b32 = oracle.Layout(m, tp_d, m.L // 2 if m.L >= 2 else 1, 2, "fp32", "separate", "block")
            b16 = oracle.Layout(m, tp_d, b32.pp, 2, "bf16", "separate", "block")
            sa = oracle.shard(full32, a)
            direct = oracle.reshard(sa, a, b16)
            via = [[f32_to_bf16(t) for t in rank] for rank in oracle.reshard(sa, a, b32)]
            assert_sets_equal(direct, via)
            full16 = {k: f32_to_bf16(v) for k, v in full32.items()}
            assert_sets_equal(direct, oracle.shard(full16, b16))
            # widening back is exact
            assert_sets_equal(oracle.reshard(direct, b16, b32),
                              [[bf16_to_f32(t) for t in rank] for rank in direct])
