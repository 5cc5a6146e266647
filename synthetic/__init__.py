"""Seeded synthetic inputs for the EMU reshard, shared by the CPU oracle tests and the GPU path.

This module knows nothing about layouts, shards or buckets: callers pass it a tensor key and a
shape and get back seeded values. It holds none of the reshard's arithmetic; it only draws numbers.

Value recipes stand in for the paper's Llama checkpoints (evaluation setup, section 7.1), which are
not available: weights ~ N(0, 0.02), RMSNorm weights 1 + N(0, 0.02), fp32 Adam first moment
~ N(0, 1e-3) and second moment |N(0, 1e-6)| (the second argument read as a standard deviation).

Two generators:

* :func:`host_tensor` draws with NumPy's PCG64 from ``SeedSequence(entropy=seed, spawn_key=key)``,
  so every logical tensor has its own reproducible stream. bf16 values are produced by rounding the
  fp32 draw to nearest-even and are returned as their uint16 bit patterns.
* :func:`device_fill` fills torch device tensors in place from a torch generator seeded per tensor.
  It is used where the host generator would be too slow (multi-GB shard sets); the oracle then reads
  the filled buffers back as its input.
"""
from __future__ import annotations

import numpy as np

#: distribution name -> (location, scale, absolute value?)
DISTS = {
    "weight": (0.0, 0.02, False),
    "norm": (1.0, 0.02, False),
    "adam_m": (0.0, 1e-3, False),
    "adam_v": (0.0, 1e-6, True),
}

DTYPE_BYTES = {"bf16": 2, "fp32": 4}


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest, ties to even); return uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bfloat16 bit patterns (uint16) to float32 values."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def host_tensor(seed: int, key: tuple, shape, dist: str = "weight", dtype: str = "bf16") -> np.ndarray:
    """Draw one seeded tensor on the host.

    ``key`` is a tuple of non-negative ints naming the tensor (it becomes the SeedSequence spawn key).
    Returns uint16 bit patterns for ``bf16`` and float32 for ``fp32``.
    """
    loc, scale, absval = DISTS[dist]
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(entropy=seed, spawn_key=tuple(key))))
    x = rng.standard_normal(size=tuple(shape), dtype=np.float32)
    x *= np.float32(scale)
    if absval:
        np.abs(x, out=x)
    if loc:
        x += np.float32(loc)
    if dtype == "bf16":
        return f32_to_bf16_bits(x)
    if dtype == "fp32":
        return x
    raise ValueError(f"unknown dtype {dtype!r}")


def host_bytes(seed: int, key: tuple, nbytes: int) -> np.ndarray:
    """Uniform random bytes (used for bucket contents and filler that must not leak into outputs)."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(entropy=seed, spawn_key=tuple(key))))
    return rng.integers(0, 256, size=int(nbytes), dtype=np.uint8)


def device_fill(tensors, seed: int, dists, dtype: str = "bf16", key_base: int = 0) -> None:
    """Fill torch device tensors in place with seeded values.

    ``tensors`` is a sequence of torch tensors (uint8/int16/int32 storage or real dtypes); ``dists`` is
    a same-length sequence of distribution names. Tensor ``i`` is drawn from a torch generator seeded
    with ``seed * 1_000_003 + key_base * 65_537 + i``. The values are written through a bf16 or fp32
    view of the tensor's bytes (so the tensor's byte size must be a multiple of the element size).
    """
    import torch

    tdt = {"bf16": torch.bfloat16, "fp32": torch.float32}[dtype]
    for i, (t, dist) in enumerate(zip(tensors, dists)):
        if t.numel() == 0:
            continue
        loc, scale, absval = DISTS[dist]
        g = torch.Generator(device=t.device)
        g.manual_seed((seed * 1_000_003 + key_base * 65_537 + i) & 0x7FFF_FFFF_FFFF_FFFF)
        view = t.view(torch.uint8).view(tdt)
        # draw in fp32 then round once to the storage type
        step = 1 << 27
        flat = view.view(-1)
        for s in range(0, flat.numel(), step):
            n = min(step, flat.numel() - s)
            x = torch.randn(n, generator=g, device=t.device, dtype=torch.float32)
            x.mul_(scale)
            if absval:
                x.abs_()
            if loc:
                x.add_(loc)
            flat[s:s + n].copy_(x)
