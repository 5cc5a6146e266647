"""Contiguous transfer buckets (test infrastructure; see package header).

The transport sends each shard once as a contiguous buffer (section 6.2, transport paragraph), and
layout changes stay local while transfers remain contiguous (section 6.2, resharding-transport
interplay). Reading taken here: a rank's shard tensors are concatenated, in the rank's canonical order
and without padding between tensors, into one byte stream; the stream is cut into buckets of B bytes,
bucket k holding stream bytes [k*B, (k+1)*B); the last bucket is short. Buckets of all ranks are listed
rank 0 first.
"""
from __future__ import annotations

import numpy as np


def stream_bytes(tensors) -> int:
    """Length in bytes of a rank's stream."""
    return int(sum(np.asarray(a).nbytes for a in tensors))


def bucket_count(nbytes: int, B: int) -> int:
    """Number of buckets of B bytes needed for a stream of ``nbytes`` bytes."""
    if B <= 0:
        raise ValueError("bucket size must be positive")
    return -(-int(nbytes) // int(B))


def pack(tensors, B: int) -> list:
    """Cut a rank's stream into buckets; returns a list of uint8 arrays."""
    stream = np.concatenate([np.ascontiguousarray(a).reshape(-1).view(np.uint8) for a in tensors]) \
        if tensors else np.zeros(0, np.uint8)
    return [stream[k * B:(k + 1) * B].copy() for k in range(bucket_count(stream.size, B))]


def unpack(buckets, like) -> list:
    """Inverse of pack: rebuild tensors shaped and typed like ``like`` from a rank's buckets."""
    stream = np.concatenate([np.asarray(b, dtype=np.uint8) for b in buckets]) if buckets \
        else np.zeros(0, np.uint8)
    out, off = [], 0
    for a in like:
        a = np.asarray(a)
        n = a.nbytes
        out.append(stream[off:off + n].view(a.dtype).reshape(a.shape).copy())
        off += n
    if off != stream.size:
        raise ValueError("bucket bytes do not match the tensor sizes")
    return out
