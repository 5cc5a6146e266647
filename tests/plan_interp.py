"""Test-only host interpreter of a compiled copy map.

Executes the segment table that ``emu_plan`` produced with NumPy byte copies on host buffers, so that
the plan compiler can be checked against the oracle on a machine without a GPU. It is neither the
oracle (it implements the library's segment semantics, not the definition) nor a product path.
"""
import numpy as np

SENTINEL = 0xA5


def _convert(raw: np.ndarray, src_run: int, run: int) -> np.ndarray:
    """Element conversion of one row, by torch's CPU casts (fp32 -> bf16 rounds to nearest even)."""
    if src_run == run:
        return raw
    import torch

    if src_run == 2 * run:      # fp32 -> bf16
        t = torch.from_numpy(raw.copy().view(np.float32)).to(torch.bfloat16)
        return t.view(torch.int16).numpy().view(np.uint8)
    if 2 * src_run == run:      # bf16 -> fp32
        t = torch.from_numpy(raw.copy().view(np.int16)).view(torch.bfloat16).to(torch.float32)
        return t.numpy().view(np.uint8)
    raise ValueError("unexpected run lengths")


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
                d[do:do + g["run"]] = _convert(src_bytes[g["src_tensor"]][so:so + g["src_run"]], g["src_run"], g["run"])
    return dst


def coverage(segments, dst_sizes):
    """Per destination tensor, sorted (start, end) byte intervals written by the plan."""
    iv = [[] for _ in dst_sizes]
    for g in segments:
        for i in range(g["rows"]):
            o = g["dst_offset"] + i * g["dst_stride"]
            iv[g["dst_tensor"]].append((o, o + g["run"]))
    return [sorted(x) for x in iv]
