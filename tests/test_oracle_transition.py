"""Pins of the oracle's transition-DAG planner (section 6.1) against facts that do not come from it.

* the paper's worked example (section 6.1): a (TP4, PP8) unit is split into four (TP4, PP2) units, two
  are destroyed and the remaining two are merged into the target (TP8, PP2);
* closed-form costs for single-primitive transitions;
* a GPU swap between two concurrently running model-stages has no deadlock-free order (infeasible), the
  same swap between model-stages of different stage kinds is feasible, a rotation through a free GPU is
  feasible with one resource-dependency edge;
* graph properties on random scenarios: every GPU handed between model-stages of one kind is released
  before it is acquired, every destroyed replica is copied before it is destroyed, the DAG is acyclic, and
  the target units hold exactly the target GPUs;
* brute force on tiny scenarios: the planner finds a DAG exactly when some order of the primitives
  satisfies every constraint.
"""
import itertools
import random

import pytest

from oracle.transition import DESTROY, EXTEND, MERGE, SPLIT, Infeasible, Links, StageTransition, plan

L = Links(gpus_per_node=8, intra_bw=100.0, inter_bw=10.0, hbm_bw=1000.0, setup_s=0.5)


def st(kind, tp, pp, dp, gpus, ttp, tpp, tdp, tg, state=800.0):
    return StageTransition(kind, tp, pp, dp, list(gpus), ttp, tpp, tdp, list(tg), state)


def test_paper_example_split_destroy_merge():
    s = st(1, 4, 8, 1, range(32), 8, 2, 1, range(16), state=3200.0)
    dag = plan([s], L)
    kinds = [n.prim for n in dag.nodes]
    assert kinds.count(SPLIT) == 1 and kinds.count(DESTROY) == 2 and kinds.count(EXTEND) == 0 \
        and kinds.count(MERGE) == 1
    split = next(n for n in dag.nodes if n.prim == SPLIT)
    destroyed = sorted(sorted(n.gpus) for n in dag.nodes if n.prim == DESTROY)
    assert destroyed == [list(range(16, 24)), list(range(24, 32))]
    (unit,) = dag.target_units[0]
    assert sorted(unit) == list(range(16)) and len(unit) == 16
    # Split: each GPU gathers the rest of its TP4 x PP2 shard (3200/8 - 3200/32 bytes); the 32-GPU unit
    # spans 4 nodes -> inter-node bandwidth
    assert split.cost == pytest.approx(0.5 + (3200 / 8 - 3200 / 32) / 10.0)
    merge = next(n for n in dag.nodes if n.prim == MERGE)
    assert merge.cost == pytest.approx((3200 / 16) / 1000.0)
    assert dag.l_tran == pytest.approx(split.cost + merge.cost)


def test_identity_and_dp_changes():
    assert plan([st(2, 2, 1, 2, range(4), 2, 1, 2, range(4))], L).nodes == []
    up = plan([st(2, 2, 1, 1, [0, 1], 2, 1, 2, [0, 1, 2, 3])], L)
    (e,) = up.nodes
    assert e.prim == EXTEND and e.gpus == [2, 3] and e.src == 0
    assert e.cost == pytest.approx(0.5 + (800 / 2) / 100.0) and up.l_tran == pytest.approx(e.cost)
    down = plan([st(2, 2, 1, 2, [0, 1, 2, 3], 2, 1, 1, [2, 3])], L)
    (d,) = down.nodes
    assert d.prim == DESTROY and d.gpus == [0, 1] and down.l_tran == 0.0
    far = plan([st(2, 1, 1, 1, [0], 1, 1, 2, [0, 9])], L)
    assert far.nodes[0].cost == pytest.approx(0.5 + 800 / 10.0)   # GPU 9 sits on another node


def test_swap_between_concurrent_stages_is_infeasible():
    a = st(2, 1, 1, 2, [0, 1], 1, 1, 2, [2, 3])
    b = st(2, 1, 1, 2, [2, 3], 1, 1, 2, [0, 1])
    with pytest.raises(Infeasible):
        plan([a, b], L)
    b.kind = 1                     # different stage kinds time-share GPUs: no conflict
    dag = plan([a, b], L)
    assert dag.n_resource_edges == 0


def test_rotation_through_a_free_gpu():
    a = st(2, 1, 1, 1, [0], 1, 1, 1, [1])
    b = st(2, 1, 1, 1, [1], 1, 1, 1, [2])
    dag = plan([a, b], L)
    assert dag.n_resource_edges == 1
    (res,) = [e for e in dag.edges if e[2]]
    assert dag.nodes[res[0]].prim == DESTROY and dag.nodes[res[0]].stage == 1 and dag.nodes[res[0]].gpus == [1]
    assert dag.nodes[res[1]].prim == EXTEND and dag.nodes[res[1]].stage == 0
    # a's Extend waits for b's copy then b's Destroy: critical path = two extends
    assert dag.l_tran == pytest.approx(2 * (0.5 + 800 / 100.0))


def _closure(dag):
    succ = {}
    for a, b, _ in dag.edges:
        succ.setdefault(a, set()).add(b)
    reach = {}
    for x in range(len(dag.nodes)):
        seen, stack = set(), [x]
        while stack:
            y = stack.pop()
            for z in succ.get(y, ()):
                if z not in seen:
                    seen.add(z)
                    stack.append(z)
        reach[x] = seen
    return reach


def random_scenario(rng, n_gpus=16):
    stages = []
    free = list(range(n_gpus))
    rng.shuffle(free)
    tfree = list(range(n_gpus))
    rng.shuffle(tfree)
    for si in range(rng.randint(1, 3)):
        kind = rng.randint(0, 2)
        opts = [(1, 1), (1, 2), (2, 1), (2, 2), (4, 1), (1, 4)]
        tp, pp = rng.choice(opts)
        ttp, tpp = rng.choice(opts)
        dp, tdp = rng.randint(1, 2), rng.randint(1, 2)
        same = [s for s in stages if s.kind == kind]
        cur_pool = [g for g in range(n_gpus) if all(g not in s.gpus for s in same)]
        tgt_pool = [g for g in range(n_gpus) if all(g not in s.tgt_gpus for s in same)]
        if len(cur_pool) < dp * tp * pp or len(tgt_pool) < tdp * ttp * tpp:
            continue
        rng.shuffle(cur_pool)
        rng.shuffle(tgt_pool)
        stages.append(st(kind, tp, pp, dp, cur_pool[:dp * tp * pp], ttp, tpp, tdp, tgt_pool[:tdp * ttp * tpp],
                         state=rng.choice([64.0, 512.0])))
    return stages


def test_graph_properties_on_random_scenarios():
    rng = random.Random(4)
    n_ok = n_inf = 0
    for _ in range(400):
        stages = random_scenario(rng)
        try:
            dag = plan(stages, L)
        except Infeasible:
            n_inf += 1
            continue
        n_ok += 1
        reach = _closure(dag)
        assert all(x not in reach[x] for x in reach)                       # acyclic
        for i, n in enumerate(dag.nodes):
            if n.prim == EXTEND:
                s = stages[n.stage]
                # every GPU it acquires from a same-kind model-stage is released first
                for j, m in enumerate(dag.nodes):
                    if m.prim == DESTROY and set(m.gpus) & set(n.gpus) and \
                            (m.stage == n.stage or stages[m.stage].kind == s.kind):
                        assert i in reach[j], "acquisition not ordered after the release"
                # the source is copied before it is destroyed
                for j, m in enumerate(dag.nodes):
                    if m.prim == DESTROY and m.stage == n.stage and m.unit == n.src:
                        assert j in reach[i]
        for si, s in enumerate(stages):
            units = dag.target_units[si]
            assert len(units) == s.tgt_dp and all(len(u) == s.tgt_tp * s.tgt_pp for u in units)
            assert sorted(g for u in units for g in u) == sorted(s.tgt_gpus)
        # ASAP schedule respects every edge; L_tran is the longest finish
        for a, b, _ in dag.edges:
            assert dag.nodes[b].start >= dag.nodes[a].finish - 1e-12
        assert dag.l_tran == pytest.approx(max((n.finish for n in dag.nodes), default=0.0))
    assert n_ok > 100 and n_inf > 5


def _brute_force_feasible(stages, dag_nodes_of):
    """Is there any order of the primitive set that respects: Split before the use of its sub-units,
    copy before destroy, merge after its providers, and exclusive GPUs per stage kind?"""
    nodes, hard = dag_nodes_of
    n = len(nodes)
    for order in itertools.permutations(range(n)):
        pos = {x: i for i, x in enumerate(order)}
        if any(pos[a] > pos[b] for a, b in hard):
            continue
        ok = True
        for i, e in enumerate(nodes):
            if e.prim != EXTEND:
                continue
            for j, d in enumerate(nodes):
                if d.prim == DESTROY and set(d.gpus) & set(e.gpus) and \
                        (d.stage == e.stage or stages[d.stage].kind == stages[e.stage].kind) and pos[j] > pos[i]:
                    ok = False
        if ok:
            return True
    return False


def test_brute_force_feasibility_tiny():
    rng = random.Random(11)
    checked = 0
    for _ in range(300):
        stages = random_scenario(rng, n_gpus=4)
        # the primitive set and its local (non-resource) edges, without the cross-stage rule
        try:
            dag = plan(stages, L)
            feasible = True
            local = [(a, b) for a, b, r in dag.edges if not r]
            nodes = dag.nodes
        except Infeasible as exc:
            feasible = False
            if "disjoint" in str(exc):
                continue
            # rebuild the primitive set with the cross-stage step disabled
            kinds = [s.kind for s in stages]
            for i, s in enumerate(stages):
                s.kind = 10 + i
            try:
                relaxed = plan(stages, L)
            finally:
                for s, k in zip(stages, kinds):
                    s.kind = k
            local = [(a, b) for a, b, r in relaxed.edges if not r]
            nodes = relaxed.nodes
        if len(nodes) > 8:
            continue
        assert _brute_force_feasible(stages, (nodes, local)) == feasible, stages
        checked += 1
    assert checked > 100
