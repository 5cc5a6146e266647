"""Per-element coordinate formulas for shard tensors (test infrastructure; see package header).

These map one element of one shard tensor to the logical tensor element it holds, with plain integer
arithmetic and pure-Python loops, no slicing, reshaping or concatenation. They restate the sharding
readings of ``oracle.model`` element by element and serve as an independent brute-force pin of the
slicing code in ``oracle.reshard``, on tiny models only.
"""
from __future__ import annotations

from .model import Layout, padded_vocab, rank_inventory


def logical_of(lay: Layout, rank: int, kind: str, layer: int, i: int, c: int):
    """(key, row, col) held by element (row i, col c) of a shard tensor, or None for a vocab pad row.

    One-dimensional norm tensors use row 0.
    """
    m, tp = lay.model, lay.tp
    t = rank % tp
    hd = m.hd
    pre = f"layers.{layer}." if layer >= 0 else ""
    if kind in ("attn_norm", "mlp_norm", "final_norm"):
        return (pre + kind, 0, c)
    if kind in ("embed", "lm_head"):
        row = t * (padded_vocab(lay) // tp) + i
        return None if row >= m.V else (kind, row, c)
    if tp > m.G and kind in ("qkv", "k", "v"):
        g, nq = t * m.G // tp, m.nH // tp * hd  # replicated KV head of this rank, its query rows
        if kind == "qkv" and i < nq:
            return (pre + "q", t * nq + i, c)
        w = i - nq if kind == "qkv" else i
        if kind == "k" or (kind == "qkv" and w < hd):
            return (pre + "k", g * hd + w, c)
        return (pre + "v", g * hd + (w - hd if kind == "qkv" else w), c)
    if kind == "qkv":
        qpg = m.nH // m.G                     # query heads per KV group
        per_group = (qpg + 2) * hd            # rows of one group: its q heads, its k head, its v head
        g = t * (m.G // tp) + i // per_group  # global KV group of this row
        w = i % per_group
        if w < qpg * hd:
            return (pre + "q", g * qpg * hd + w, c)
        if w < (qpg + 1) * hd:
            return (pre + "k", g * hd + (w - qpg * hd), c)
        return (pre + "v", g * hd + (w - (qpg + 1) * hd), c)
    if kind == "q":
        return (pre + "q", t * (m.nH // tp) * hd + i, c)
    if kind in ("k", "v"):
        return (pre + kind, t * (m.G // tp) * hd + i, c)
    if kind == "o":
        return (pre + "o", i, t * (m.nH * hd // tp) + c)
    if kind == "gate_up":
        n = m.I // tp
        return (pre + "gate", t * n + i, c) if i < n else (pre + "up", t * n + (i - n), c)
    if kind in ("gate", "up"):
        return (pre + kind, t * (m.I // tp) + i, c)
    if kind == "down":
        return (pre + "down", i, t * (m.I // tp) + c)
    raise KeyError(kind)


def logical_numbering(model) -> dict:
    """A global element numbering of the logical model: key -> (first id, row length)."""
    from .sharding import logical_tensors

    base, out = 0, {}
    for _, key, shape, _ in logical_tensors(model):
        ncol = shape[-1]
        nrow = shape[0] if len(shape) == 2 else 1
        out[key] = (base, ncol)
        base += nrow * ncol
    return out


def element_ids(lay: Layout) -> list:
    """For every shard tensor of the layout, a nested Python list of logical element ids (-1 = pad).

    Computed element by element with :func:`logical_of`; O(model size) Python work, tiny models only.
    """
    num = logical_numbering(lay.model)
    out = []
    for r, specs in enumerate(rank_inventory(lay)):
        per_rank = []
        for s in specs:
            rows, cols = (1, s.shape[0]) if len(s.shape) == 1 else s.shape
            ids = []
            for i in range(rows):
                for c in range(cols):
                    loc = logical_of(lay, r, s.kind, s.layer, i, c)
                    if loc is None:
                        ids.append(-1)
                    else:
                        b, ncol = num[loc[0]]
                        ids.append(b + loc[1] * ncol + loc[2])
            per_rank.append(ids)
        out.append(per_rank)
    return out
