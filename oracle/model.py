"""Model shapes, EMU layouts and the per-rank shard inventory (test infrastructure; see package header).

Paper anchors:
  * EMU definition (section 5): a unit has layout T_tp x pp over |R| = tp * pp GPUs and holds shards
    theta_i for i = 1..tp*pp; optimizer shards follow the same layout; no sharding across DP (ZeRO-0).
  * Primitives (section 5.2): Split and Merge are defined for any integer factor between compatible
    layouts; the planner only searches power-of-two degrees. Validity below therefore asks only for
    divisibility, never for powers of two.

Readings (the paper is silent on all of these):
  * Sharding rules follow Megatron-LM, which the system integrates with (section 2): q/k/v and gate/up are
    column-parallel, o and down are row-parallel, embedding and LM head are vocab-parallel, norms are
    replicated on every TP rank.
  * Fused QKV is head-interleaved per KV group: per local group, its query heads, its k head, its v head.
    A KV head is never split. With tp <= kv_heads, tp divides the KV-head count and each rank holds
    kv_heads/tp whole groups. With tp > kv_heads (the Megatron/vLLM convention), tp must be a multiple of
    the KV-head count and divide the query heads: rank t holds nH/tp query heads and one replica of KV head
    t * kv_heads / tp, which is read back from its first replica (the lowest rank holding it).
  * PP stages hold contiguous layer ranges; when pp does not divide L, the first L mod pp stages hold
    one extra layer. The embedding sits on stage 0, the final norm and the LM head on the last stage.
    Embeddings are untied.
  * Rank order inside a unit is r = p * tp + t (TP fastest).
  * Vocabulary padding: with pad multiple m > 0 the padded vocabulary is ceil(V / (tp*m)) * tp * m;
    with m = 0 there is no padding and tp must divide V.
"""
from __future__ import annotations

from dataclasses import dataclass

DTYPE_BYTES = {"bf16": 2, "fp32": 4}


class LayoutError(ValueError):
    """The layout does not divide the model (an invalid EMU layout)."""


@dataclass(frozen=True)
class Model:
    """Llama-style decoder shape. L layers, hidden H, nH query heads of size hd, G KV heads, MLP width I,
    vocabulary V."""
    L: int
    H: int
    nH: int
    hd: int
    G: int
    I: int
    V: int


@dataclass(frozen=True)
class Layout:
    """An EMU layout T_tp x pp plus the storage conventions of its shards.

    qkv: "interleaved" (one fused tensor per rank, per KV group [q heads; k; v]) or "separate".
    mlp: "block" (one fused tensor per rank, [gate_t; up_t]) or "separate".
    """
    model: Model
    tp: int
    pp: int
    pad: int = 0
    dtype: str = "bf16"
    qkv: str = "interleaved"
    mlp: str = "block"

    @property
    def nranks(self) -> int:
        return self.tp * self.pp

    @property
    def esize(self) -> int:
        return DTYPE_BYTES[self.dtype]


@dataclass(frozen=True)
class TensorSpec:
    """One shard tensor: its kind, its layer (-1 for global tensors) and its row-major shape."""
    kind: str
    layer: int
    shape: tuple

    @property
    def numel(self) -> int:
        n = 1
        for s in self.shape:
            n *= s
        return n


def check_layout(lay: Layout) -> None:
    """Raise LayoutError unless ``lay`` is a valid layout of its model."""
    m = lay.model
    for name in ("L", "H", "nH", "hd", "G", "I", "V"):
        if getattr(m, name) <= 0:
            raise LayoutError(f"model dimension {name} must be positive")
    if lay.tp <= 0 or lay.pp <= 0 or lay.pad < 0:
        raise LayoutError("tp, pp must be positive and the pad multiple non-negative")
    if lay.dtype not in DTYPE_BYTES:
        raise LayoutError(f"unknown dtype {lay.dtype!r}")
    if lay.qkv not in ("interleaved", "separate") or lay.mlp not in ("block", "separate"):
        raise LayoutError("unknown fused-weight format")
    if m.nH % m.G:
        raise LayoutError("query heads must be a multiple of KV heads")
    if lay.tp <= m.G and m.G % lay.tp:
        raise LayoutError("tp must divide the KV-head count")
    if lay.tp > m.G and (lay.tp % m.G or m.nH % lay.tp):
        raise LayoutError("with KV replication tp must be a multiple of the KV heads and divide the query heads")
    if m.I % lay.tp:
        raise LayoutError("tp must divide the MLP width")
    if lay.pp > m.L:
        raise LayoutError("pp must not exceed the layer count")
    if lay.pad == 0 and m.V % lay.tp:
        raise LayoutError("tp must divide the vocabulary when it is not padded")


def padded_vocab(lay: Layout) -> int:
    """Padded vocabulary Vp of a layout (equal to V when the pad multiple is 0)."""
    V = lay.model.V
    if lay.pad == 0:
        return V
    q = lay.tp * lay.pad
    return -(-V // q) * q


def stage_layers(lay: Layout, p: int) -> range:
    """Layers held by pipeline stage p: a contiguous range; the first L mod pp stages hold one more."""
    per, extra = divmod(lay.model.L, lay.pp)
    start = p * per + min(p, extra)
    return range(start, start + per + (1 if p < extra else 0))


def stage_of_layer(lay: Layout, layer: int) -> int:
    """The pipeline stage holding ``layer``."""
    for p in range(lay.pp):
        if layer in stage_layers(lay, p):
            return p
    raise IndexError(layer)


def kv_local(lay: Layout) -> int:
    """KV heads held by one TP rank (1 when KV heads are replicated, tp > kv_heads)."""
    return max(lay.model.G // lay.tp, 1)


def rank_of(lay: Layout, t: int, p: int) -> int:
    """Rank index inside the unit; TP is the fastest-varying coordinate."""
    return p * lay.tp + t


def _layer_specs(lay: Layout, layer: int) -> list:
    m, tp = lay.model, lay.tp
    H, hd = m.H, m.hd
    out = [TensorSpec("attn_norm", layer, (H,))]
    kvl = kv_local(lay)
    if lay.qkv == "interleaved":
        out.append(TensorSpec("qkv", layer, ((m.nH // tp + 2 * kvl) * hd, H)))
    else:
        out += [TensorSpec("q", layer, (m.nH // tp * hd, H)),
                TensorSpec("k", layer, (kvl * hd, H)),
                TensorSpec("v", layer, (kvl * hd, H))]
    out.append(TensorSpec("o", layer, (H, m.nH * hd // tp)))
    out.append(TensorSpec("mlp_norm", layer, (H,)))
    if lay.mlp == "block":
        out.append(TensorSpec("gate_up", layer, (2 * m.I // tp, H)))
    else:
        out += [TensorSpec("gate", layer, (m.I // tp, H)),
                TensorSpec("up", layer, (m.I // tp, H))]
    out.append(TensorSpec("down", layer, (H, m.I // tp)))
    return out


def rank_inventory(lay: Layout) -> list:
    """Per rank (in rank order), the ordered list of shard tensors it holds.

    Canonical order on rank (t, p): embedding if p == 0; then, for each local layer in order, attention
    norm, QKV, o, MLP norm, gate/up, down; then final norm and LM head if p == pp - 1.
    """
    check_layout(lay)
    m = lay.model
    vrows = padded_vocab(lay) // lay.tp
    ranks = []
    for p in range(lay.pp):
        for t in range(lay.tp):
            specs = []
            if p == 0:
                specs.append(TensorSpec("embed", -1, (vrows, m.H)))
            for layer in stage_layers(lay, p):
                specs += _layer_specs(lay, layer)
            if p == lay.pp - 1:
                specs.append(TensorSpec("final_norm", -1, (m.H,)))
                specs.append(TensorSpec("lm_head", -1, (vrows, m.H)))
            ranks.append(specs)
    return ranks


def groups(model: Model) -> list:
    """Independent tensor groups: the embedding, each layer, and the final group (final norm + LM head).
    The shards of one group are built from the logical tensors of that group only."""
    return ["embed"] + list(range(model.L)) + ["final"]


def group_of(spec: TensorSpec):
    if spec.kind == "embed":
        return "embed"
    if spec.kind in ("final_norm", "lm_head"):
        return "final"
    return spec.layer
