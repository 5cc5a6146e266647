"""Test-only host interpreter of a compiled copy map.

Executes the segment table that ``emu_plan`` produced with NumPy byte copies on host buffers, so that
the plan compiler can be checked against the oracle on a machine without a GPU. It is neither the
oracle (it implements the library's segment semantics, not the definition) nor a product path.
"""
import numpy as np

SENTINEL = 0xA5


def run_plan(segments, src_bytes, dst_sizes, prefix=None):
    """src_bytes: list of uint8 arrays (global source order); returns a list of destination arrays,
    initialised to a sentinel, after executing the first ``prefix`` segments (all by default)."""
    dst = [np.full(n, SENTINEL, dtype=np.uint8) for n in dst_sizes]
    for g in segments[:prefix]:
        d = dst[g["dst_tensor"]]
        for i in range(g["rows"]):
            do = g["dst_offset"] + i * g["dst_stride"]
            if g["src_tensor"] < 0:
                d[do:do + g["run"]] = 0
            else:
                so = g["src_offset"] + i * g["src_stride"]
                d[do:do + g["run"]] = src_bytes[g["src_tensor"]][so:so + g["run"]]
    return dst


def coverage(segments, dst_sizes):
    """Per destination tensor, sorted (start, end) byte intervals written by the plan."""
    iv = [[] for _ in dst_sizes]
    for g in segments:
        for i in range(g["rows"]):
            o = g["dst_offset"] + i * g["dst_stride"]
            iv[g["dst_tensor"]].append((o, o + g["run"]))
    return [sorted(x) for x in iv]
