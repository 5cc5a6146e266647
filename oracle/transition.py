"""Transition DAG between two plans, and its critical-path cost (test infrastructure; see package header).

What is implemented, as this module reads section 6.1 (decomposition and DAG construction) and the
section 6 introduction (cost):
  * Per model-stage, four phases run in a fixed order: Split, Destroy, Extend, Merge. The common layout
    T_sub is the largest TP/PP layout that both the current and the target unit layouts divide into;
    current units are cut into T_sub units, surplus ones are released, missing ones are copied onto target
    GPUs, and the T_sub units are assembled into target units. A unit that is the only holder of its state
    is released only after the copy that needs it (an edge from that Extend to that Destroy).
  * Model-stages hand GPUs to each other through resource edges: an acquisition of GPUs another
    model-stage still holds waits for the Destroy that frees them. If that Destroy itself waits, directly
    or through other edges, on the acquisition, the plan has no deadlock-free order and is rejected.
    Releases are favoured, and equal cases are ordered generation, inference, training.
  * L_tran, the cost of the DAG's longest path, comes from the bytes moved, link bandwidth and
    communicator setup.

Readings (the paper gives no algorithm listing):
  * T_sub = (gcd(tp, tp*), gcd(pp, pp*)). Splitting a unit of layout (tp, pp) into T_sub units yields
    k = (tp/tps)(pp/pps) units; sub-unit (a, b), a < tp/tps, b < pp/pps, holds the unit's ranks
    (t, p) = (a*tps + t', b*pps + p') at its own rank (t', p'). Ranks are ordered r = p*tp + t.
  * The target of a model-stage is its layout (tp*, pp*, dp*) and its GPU set. A current T_sub unit is
    kept (no data moves) when all its GPUs lie in the target set, first fit in sub-unit order, up to the
    dp*(tp*/tps)(pp*/pps) T_sub units the target needs. All other sub-units are destroyed.
  * Missing T_sub units are extended onto the target GPUs no kept unit occupies, taken in ascending GPU id,
    tps*pps GPUs each in rank order. The i-th Extend copies from the first current sub-unit, scanning
    cyclically from position i, whose GPUs are disjoint from its own (an Extend targets a disjoint GPU set,
    section 5.2 (c)); none -> infeasible.
  * The T_sub units (kept ones first, then extended ones) are merged k* at a time into the dp* target
    units (no Merge when k* = 1). A merged unit's rank (t*, p*) is rank (t* mod tps, p* mod pps) of its
    sub-unit (t* div tps) + (p* div pps)(tp*/tps).
  * GPUs conflict only between model-stages of the same stage kind: those run concurrently and must hold
    disjoint GPU sets (section 4.2, Eq. (1)); model-stages of different kinds time-share GPUs.
  * Costs: Split = setup + (shard_sub - shard_cur) / bw(unit); Extend = setup + max over rank pairs of
    shard_sub / bw(pair); Merge = shard_target / hbm_bw; Destroy = 0. bw is the intra-node bandwidth when
    all GPUs involved share a node (gpu // gpus_per_node), else the inter-node bandwidth; shard = state
    bytes / GPUs of the unit. L_tran is the longest path (ready primitives run concurrently).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from math import gcd

SPLIT, DESTROY, EXTEND, MERGE = 0, 1, 2, 3


class Infeasible(Exception):
    """No deadlock-free transition DAG exists for this target plan under the rules above."""


@dataclass
class StageTransition:
    kind: int                 # 0 generation, 1 inference, 2 training
    tp: int
    pp: int
    dp: int
    gpus: list                # dp*tp*pp current GPU ids, unit-major, rank order
    tgt_tp: int
    tgt_pp: int
    tgt_dp: int
    tgt_gpus: list            # target GPU set (dp*tp*pp ids, any order)
    state_bytes: float        # logical state of one replica


@dataclass
class Links:
    gpus_per_node: int = 8
    intra_bw: float = 300e9
    inter_bw: float = 25e9
    hbm_bw: float = 5e12
    setup_s: float = 0.05


@dataclass
class Node:
    prim: int
    stage: int
    unit: int                 # SPLIT: current unit; DESTROY: current sub-unit; EXTEND: slot; MERGE: target unit
    src: int                  # EXTEND: source sub-unit; else -1
    gpus: list
    cost: float = 0.0
    start: float = 0.0
    finish: float = 0.0


@dataclass
class Dag:
    nodes: list = field(default_factory=list)
    edges: list = field(default_factory=list)      # (from, to, resource)
    target_units: list = field(default_factory=list)  # per stage: list of target unit GPU lists
    l_tran: float = 0.0

    @property
    def n_resource_edges(self):
        return sum(1 for e in self.edges if e[2])


def _split_gpus(gpus, tp, pp, tps, pps):
    """The T_sub sub-units of one unit (GPU lists in the sub-unit's own rank order)."""
    out = []
    for b in range(pp // pps):
        for a in range(tp // tps):
            sub = []
            for pq in range(pps):
                for tq in range(tps):
                    sub.append(gpus[(b * pps + pq) * tp + (a * tps + tq)])
            out.append(sub)
    return out


def _bw(links, gs):
    nodes = {g // links.gpus_per_node for g in gs}
    return links.intra_bw if len(nodes) == 1 else links.inter_bw


def _check(stages):
    for i, s in enumerate(stages):
        for name in ("tp", "pp", "dp", "tgt_tp", "tgt_pp", "tgt_dp"):
            if getattr(s, name) <= 0:
                raise ValueError(f"stage {i}: {name} must be positive")
        if len(s.gpus) != s.dp * s.tp * s.pp or len(set(s.gpus)) != len(s.gpus):
            raise ValueError(f"stage {i}: current GPU list must hold dp*tp*pp distinct ids")
        if len(s.tgt_gpus) != s.tgt_dp * s.tgt_tp * s.tgt_pp or len(set(s.tgt_gpus)) != len(s.tgt_gpus):
            raise ValueError(f"stage {i}: target GPU list must hold dp*tp*pp distinct ids")
    for i, a in enumerate(stages):
        for j, b in enumerate(stages[:i]):
            if a.kind == b.kind and (set(a.gpus) & set(b.gpus) or set(a.tgt_gpus) & set(b.tgt_gpus)):
                raise ValueError(f"stages {j} and {i} run concurrently but share GPUs")


def plan(stages, links: Links = Links()) -> Dag:
    """Build the global transition DAG and its critical-path cost. Raises Infeasible or ValueError."""
    _check(stages)
    dag = Dag()
    nodes, edges = dag.nodes, set()
    destroy_of_gpu = []          # per stage: gpu -> DESTROY node releasing it
    extends = []                 # (stage, node id)

    for si, s in enumerate(stages):
        tps, pps = gcd(s.tp, s.tgt_tp), gcd(s.pp, s.tgt_pp)
        n_sub = tps * pps
        k, ks = (s.tp // tps) * (s.pp // pps), (s.tgt_tp // tps) * (s.tgt_pp // pps)
        shard_cur, shard_sub = s.state_bytes / (s.tp * s.pp), s.state_bytes / n_sub
        unit_gpus = [s.gpus[u * s.tp * s.pp:(u + 1) * s.tp * s.pp] for u in range(s.dp)]

        # Split: current units -> T_sub units
        subs, split_of = [], []
        for u, ug in enumerate(unit_gpus):
            parts = _split_gpus(ug, s.tp, s.pp, tps, pps)
            sid = -1
            if k > 1:
                sid = len(nodes)
                nodes.append(Node(SPLIT, si, u, -1, list(ug),
                                  links.setup_s + (shard_sub - shard_cur) / _bw(links, ug)))
            for part in parts:
                subs.append(part)
                split_of.append(sid)

        # keep the sub-units that already sit inside the target GPU set
        tgt = set(s.tgt_gpus)
        need = s.tgt_dp * ks
        kept = []
        for j, part in enumerate(subs):
            if len(kept) < need and set(part) <= tgt:
                kept.append(j)
        kept_set = set(kept)

        # Destroy the rest
        dmap, dnode = {}, {}
        for j, part in enumerate(subs):
            if j in kept_set:
                continue
            did = len(nodes)
            nodes.append(Node(DESTROY, si, j, -1, list(part), 0.0))
            dnode[j] = did
            if split_of[j] >= 0:
                edges.add((split_of[j], did, 0))
            for g in part:
                dmap[g] = did
        destroy_of_gpu.append(dmap)

        # Extend the missing T_sub units onto the free target GPUs
        used = {g for j in kept for g in subs[j]}
        free = sorted(tgt - used)
        slots = []                       # (gpu list, provider node or -1, kept sub index or -1)
        for j in kept:
            slots.append((subs[j], split_of[j]))
        for i in range(need - len(kept)):
            slot = free[i * n_sub:(i + 1) * n_sub]
            src = -1
            for c in range(len(subs)):
                cand = (i + c) % len(subs)
                if not set(subs[cand]) & set(slot):
                    src = cand
                    break
            if src < 0:
                raise Infeasible(f"stage {si}: no replica disjoint from extend slot {i}")
            eid = len(nodes)
            cost = links.setup_s + max(shard_sub / _bw(links, (a, b)) for a, b in zip(subs[src], slot))
            nodes.append(Node(EXTEND, si, len(kept) + i, src, list(slot), cost))
            if split_of[src] >= 0:
                edges.add((split_of[src], eid, 0))
            if src in dnode:
                edges.add((eid, dnode[src], 0))          # destroyed only after it has been copied
            for g in slot:                               # release before acquire, same model-stage
                if g in dmap and dmap[g] != dnode.get(src):
                    edges.add((dmap[g], eid, 0))
            extends.append((si, eid))
            slots.append((slot, eid))

        # Merge k* T_sub units into each target unit
        units = []
        for u in range(s.tgt_dp):
            group = slots[u * ks:(u + 1) * ks]
            ug = [None] * (s.tgt_tp * s.tgt_pp)
            for p_ in range(s.tgt_pp):
                for t_ in range(s.tgt_tp):
                    sub = (p_ // pps) * (s.tgt_tp // tps) + t_ // tps
                    ug[p_ * s.tgt_tp + t_] = group[sub][0][(p_ % pps) * tps + t_ % tps]
            units.append(ug)
            if ks > 1:
                mid = len(nodes)
                nodes.append(Node(MERGE, si, u, -1, list(ug),
                                  (s.state_bytes / (s.tgt_tp * s.tgt_pp)) / links.hbm_bw))
                for _, prov in group:
                    if prov >= 0:
                        edges.add((prov, mid, 0))
        dag.target_units.append(units)

    # cross-model-stage resource edges: blocked acquisitions wait for the releasing Destroy
    succ = {}
    for a, b, _ in edges:
        succ.setdefault(a, set()).add(b)

    def reaches(a, b):
        stack, seen = [a], {a}
        while stack:
            x = stack.pop()
            if x == b:
                return True
            for y in succ.get(x, ()):
                if y not in seen:
                    seen.add(y)
                    stack.append(y)
        return False

    order = sorted(extends, key=lambda e: (stages[e[0]].kind, e[0], e[1]))
    for si, eid in order:
        for g in nodes[eid].gpus:
            for sj, other in enumerate(stages):
                if sj == si or other.kind != stages[si].kind or g not in set(other.gpus):
                    continue
                did = destroy_of_gpu[sj].get(g)
                if did is None:
                    raise Infeasible(f"stage {si} needs GPU {g}, which stage {sj} keeps")
                if (did, eid, 1) in edges:
                    continue
                if reaches(eid, did):
                    raise Infeasible(f"stage {si}: the Destroy releasing GPU {g} depends on the acquisition")
                edges.add((did, eid, 1))
                succ.setdefault(did, set()).add(eid)

    dag.edges = sorted(edges, key=lambda e: (e[1], e[0], e[2]))
    # ASAP schedule = critical path (nodes are created in a topological order except for resource
    # edges, so relax in a topological order computed explicitly)
    preds = {}
    for a, b, _ in dag.edges:
        preds.setdefault(b, []).append(a)
    indeg = {i: 0 for i in range(len(nodes))}
    for a, b, _ in dag.edges:
        indeg[b] += 1
    ready = sorted(i for i in indeg if indeg[i] == 0)
    topo = []
    while ready:
        x = ready.pop(0)
        topo.append(x)
        for y in sorted(succ.get(x, ())):
            indeg[y] -= 1
            if indeg[y] == 0:
                ready.append(y)
        ready.sort()
    if len(topo) != len(nodes):
        raise Infeasible("cycle in the transition DAG")
    for x in topo:
        n = nodes[x]
        n.start = max((nodes[p].finish for p in preds.get(x, [])), default=0.0)
        n.finish = n.start + n.cost
    dag.l_tran = max((n.finish for n in nodes), default=0.0)
    return dag
