"""Plain definition of the EMU Split/Merge reshard (test infrastructure; see package header).

Split (section 5.2 (a)) and Merge (section 5.2 (b)) move an EMU's parameter and optimizer shards between
two TP/PP layouts of the same model-stage without changing its logical state (section 6.2, preserving
training semantics). Whatever route an implementation takes, the result is the one obtained by

    full = unshard(src_shards, L_src)      # rebuild every logical tensor
    dst  = shard(full, L_dst)              # cut it again for the destination layout

which is what this module does, tensor group by tensor group (the embedding, each layer, the final
norm + LM head), so that multi-GB models can be streamed through host memory. Readings of the sharding
conventions are listed in ``oracle.model``; the direction-free form covers the paper's Split, its Merge,
and compositions of the two.

Arrays are NumPy arrays of any element type (bf16 is carried as uint16 bit patterns). Between layouts
of the same element type nothing rounds or converts: the reshard is a selection and permutation of
elements. Between an fp32 and a bf16 layout (training state to generation weights) the logical tensors
are converted by ``oracle.convert`` between unshard and shard.
"""
from __future__ import annotations

import numpy as np

from .convert import convert
from .model import Layout, LayoutError, check_layout, group_of, groups, kv_local, padded_vocab, rank_inventory, \
    rank_of, stage_of_layer

LAYER_TENSORS = ("attn_norm", "q", "k", "v", "o", "mlp_norm", "gate", "up", "down")


def _key(name: str, layer: int) -> str:
    return f"layers.{layer}.{name}" if layer >= 0 else name


def logical_tensors(model) -> list:
    """(group, key, shape, kind) for every logical tensor of the model, in group order.

    Full Llama-style tensors, row-major, as a HuggingFace checkpoint stores them: q [nH*hd, H],
    k and v [G*hd, H], o [H, nH*hd], gate and up [I, H], down [H, I], norms [H], embedding and
    LM head [V, H] (untied).
    """
    m = model
    shapes = {
        "attn_norm": (m.H,), "q": (m.nH * m.hd, m.H), "k": (m.G * m.hd, m.H), "v": (m.G * m.hd, m.H),
        "o": (m.H, m.nH * m.hd), "mlp_norm": (m.H,), "gate": (m.I, m.H), "up": (m.I, m.H),
        "down": (m.H, m.I),
    }
    out = [("embed", "embed", (m.V, m.H), "embed")]
    for layer in range(m.L):
        for name in LAYER_TENSORS:
            out.append((layer, _key(name, layer), shapes[name], name))
    out.append(("final", "final_norm", (m.H,), "final_norm"))
    out.append(("final", "lm_head", (m.V, m.H), "lm_head"))
    return out


def _index(lay: Layout) -> dict:
    """(rank, kind, layer) -> position of that shard tensor in the rank's ordered list."""
    idx = {}
    for r, specs in enumerate(rank_inventory(lay)):
        for j, s in enumerate(specs):
            idx[(r, s.kind, s.layer)] = j
    return idx


def _owner_stage(lay: Layout, layer: int, kind: str) -> int:
    if kind == "embed":
        return 0
    if kind in ("final_norm", "lm_head"):
        return lay.pp - 1
    return stage_of_layer(lay, layer)


# ----------------------------------------------------------------------------------------------
# shard: full logical tensors -> the shard tensors of one layout
# ----------------------------------------------------------------------------------------------

def _shard_one(lay: Layout, kind: str, layer: int, t: int, full: dict) -> np.ndarray:
    m, tp = lay.model, lay.tp
    hd, qpg, gl = m.hd, m.nH // m.G, m.G // tp
    if tp > m.G and kind in ("qkv", "k", "v"):
        # KV replication: rank t holds nH/tp query heads and a replica of KV head t*G/tp
        g, nq = t * m.G // tp, m.nH // tp * hd
        q, k, v = (full[_key(n, layer)] for n in ("q", "k", "v"))
        if kind == "qkv":
            return np.concatenate([q[t * nq:(t + 1) * nq], k[g * hd:(g + 1) * hd], v[g * hd:(g + 1) * hd]], axis=0)
        return (k if kind == "k" else v)[g * hd:(g + 1) * hd].copy()
    if kind in ("attn_norm", "mlp_norm", "final_norm"):
        # replicated on every TP rank of the owning stage
        return full[_key(kind, layer)].copy()
    if kind in ("embed", "lm_head"):
        x = full[kind]
        vp = padded_vocab(lay)
        padded = np.concatenate([x, np.zeros((vp - m.V, m.H), dtype=x.dtype)], axis=0)
        rows = vp // tp
        return padded[t * rows:(t + 1) * rows].copy()
    if kind == "qkv":
        q, k, v = (full[_key(n, layer)] for n in ("q", "k", "v"))
        parts = []
        for g in range(t * gl, (t + 1) * gl):
            parts += [q[g * qpg * hd:(g + 1) * qpg * hd], k[g * hd:(g + 1) * hd], v[g * hd:(g + 1) * hd]]
        return np.concatenate(parts, axis=0)
    if kind == "q":
        n = m.nH // tp * hd
        return full[_key("q", layer)][t * n:(t + 1) * n].copy()
    if kind in ("k", "v"):
        n = gl * hd
        return full[_key(kind, layer)][t * n:(t + 1) * n].copy()
    if kind == "o":
        n = m.nH * hd // tp
        return full[_key("o", layer)][:, t * n:(t + 1) * n].copy()
    if kind == "gate_up":
        n = m.I // tp
        return np.concatenate([full[_key("gate", layer)][t * n:(t + 1) * n],
                               full[_key("up", layer)][t * n:(t + 1) * n]], axis=0)
    if kind in ("gate", "up"):
        n = m.I // tp
        return full[_key(kind, layer)][t * n:(t + 1) * n].copy()
    if kind == "down":
        n = m.I // tp
        return full[_key("down", layer)][:, t * n:(t + 1) * n].copy()
    raise KeyError(kind)


def shard_group(lay: Layout, group, full: dict) -> dict:
    """Shard tensors of one group for layout ``lay``: {(rank, position): array}."""
    out = {}
    for r, specs in enumerate(rank_inventory(lay)):
        t = r % lay.tp
        for j, s in enumerate(specs):
            if group_of(s) == group:
                out[(r, j)] = _shard_one(lay, s.kind, s.layer, t, full)
    return out


# ----------------------------------------------------------------------------------------------
# unshard: the shard tensors of one layout -> full logical tensors
# ----------------------------------------------------------------------------------------------

def unshard_group(lay: Layout, group, get) -> dict:
    """Rebuild the logical tensors of one group. ``get(rank, position)`` returns a shard tensor."""
    check_layout(lay)
    m, tp = lay.model, lay.tp
    idx = _index(lay)
    hd, qpg, gl = m.hd, m.nH // m.G, m.G // tp

    def shards(kind, layer):
        p = _owner_stage(lay, layer, kind)
        return [get(rank_of(lay, t, p), idx[(rank_of(lay, t, p), kind, layer)]) for t in range(tp)]

    def first(kind, layer):
        # replicated tensors are read from TP rank 0 of the owning stage
        p = _owner_stage(lay, layer, kind)
        r = rank_of(lay, 0, p)
        return np.array(get(r, idx[(r, kind, layer)]))

    full = {}
    if group == "embed":
        full["embed"] = np.concatenate(shards("embed", -1), axis=0)[:m.V]
        return full
    if group == "final":
        full["final_norm"] = first("final_norm", -1)
        full["lm_head"] = np.concatenate(shards("lm_head", -1), axis=0)[:m.V]
        return full
    layer = group
    full[_key("attn_norm", layer)] = first("attn_norm", layer)
    full[_key("mlp_norm", layer)] = first("mlp_norm", layer)
    if tp > m.G:
        # KV replication: queries from every rank, each KV head from its first replica (rank g*tp/G)
        rep, nq = tp // m.G, m.nH // tp * hd
        blks = [np.asarray(b) for b in shards("qkv" if lay.qkv == "interleaved" else "q", layer)]
        full[_key("q", layer)] = np.concatenate([b[:nq] for b in blks], axis=0)
        if lay.qkv == "interleaved":
            full[_key("k", layer)] = np.concatenate([blks[g * rep][nq:nq + hd] for g in range(m.G)], axis=0)
            full[_key("v", layer)] = np.concatenate([blks[g * rep][nq + hd:nq + 2 * hd] for g in range(m.G)], axis=0)
        else:
            for n in ("k", "v"):
                kb = [np.asarray(b) for b in shards(n, layer)]
                full[_key(n, layer)] = np.concatenate([kb[g * rep] for g in range(m.G)], axis=0)
    elif lay.qkv == "interleaved":
        qs, ks, vs = [], [], []
        for blk in shards("qkv", layer):
            b = np.asarray(blk).reshape(gl, qpg + 2, hd, m.H)
            qs.append(b[:, :qpg].reshape(-1, m.H))
            ks.append(b[:, qpg].reshape(-1, m.H))
            vs.append(b[:, qpg + 1].reshape(-1, m.H))
        full[_key("q", layer)] = np.concatenate(qs, axis=0)
        full[_key("k", layer)] = np.concatenate(ks, axis=0)
        full[_key("v", layer)] = np.concatenate(vs, axis=0)
    else:
        for n in ("q", "k", "v"):
            full[_key(n, layer)] = np.concatenate(shards(n, layer), axis=0)
    full[_key("o", layer)] = np.concatenate(shards("o", layer), axis=1)
    if lay.mlp == "block":
        half = m.I // tp
        blks = [np.asarray(b) for b in shards("gate_up", layer)]
        full[_key("gate", layer)] = np.concatenate([b[:half] for b in blks], axis=0)
        full[_key("up", layer)] = np.concatenate([b[half:] for b in blks], axis=0)
    else:
        for n in ("gate", "up"):
            full[_key(n, layer)] = np.concatenate(shards(n, layer), axis=0)
    full[_key("down", layer)] = np.concatenate(shards("down", layer), axis=1)
    return full


# ----------------------------------------------------------------------------------------------
# whole-model forms
# ----------------------------------------------------------------------------------------------

def _same_state(src: Layout, dst: Layout) -> None:
    check_layout(src)
    check_layout(dst)
    if src.model != dst.model:
        raise LayoutError("source and destination layouts describe different models")


def reshard_group(get, src: Layout, dst: Layout, group) -> dict:
    """Destination shard tensors of one group: shard(convert(unshard(src)), dst). The conversion is the
    identity when both layouts store the same element type (see oracle.convert)."""
    _same_state(src, dst)
    full = unshard_group(src, group, get)
    if src.dtype != dst.dtype:
        full = {k: convert(v, src.dtype, dst.dtype) for k, v in full.items()}
    return shard_group(dst, group, full)


def shard(full: dict, lay: Layout) -> list:
    """All shard tensors of a layout, as a list (rank order) of lists (canonical order)."""
    inv = rank_inventory(lay)
    out = [[None] * len(specs) for specs in inv]
    for g in groups(lay.model):
        for (r, j), a in shard_group(lay, g, full).items():
            out[r][j] = a
    return out


def unshard(shards: list, lay: Layout) -> dict:
    """Full logical tensors from a complete shard set."""
    full = {}
    for g in groups(lay.model):
        full.update(unshard_group(lay, g, lambda r, j: shards[r][j]))
    return full


def reshard(shards: list, src: Layout, dst: Layout) -> list:
    """Destination shard set from a source shard set (the Split/Merge reshard, with an element-type
    conversion when the two layouts store different types)."""
    _same_state(src, dst)
    inv = rank_inventory(dst)
    out = [[None] * len(specs) for specs in inv]
    for g in groups(src.model):
        for (r, j), a in reshard_group(lambda rr, jj: shards[rr][jj], src, dst, g).items():
            out[r][j] = a
    return out
