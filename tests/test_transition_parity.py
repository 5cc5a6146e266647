"""The library's transition-DAG planner (C++, emu_dag_plan) against the oracle's (section 6.1):
identical primitives, edges, target units, costs and critical path on random multi-model-stage
scenarios, identical verdicts on infeasible plans, and planning time at 1,024 GPUs."""
import random
import time

import pytest

from oracle.transition import Infeasible, Links, plan
from paper_2609_34645_amd import emu
from tests.test_oracle_transition import L, random_scenario, st


def as_dicts(stages):
    return [dict(kind=s.kind, tp=s.tp, pp=s.pp, dp=s.dp, gpus=s.gpus, tgt_tp=s.tgt_tp, tgt_pp=s.tgt_pp,
                 tgt_dp=s.tgt_dp, tgt_gpus=s.tgt_gpus, state_bytes=s.state_bytes) for s in stages]


def lib_plan(stages, links=L):
    return emu.dag_plan(as_dicts(stages), links.gpus_per_node, links.intra_bw, links.inter_bw, links.hbm_bw,
                        links.setup_s)


def compare(stages, links=L):
    try:
        want = plan(stages, links)
    except Infeasible:
        with pytest.raises(emu.EmuError) as e:
            lib_plan(stages, links)
        assert e.value.code == emu.ERR_INFEASIBLE
        return False
    got = lib_plan(stages, links)
    assert len(got["nodes"]) == len(want.nodes)
    for g, w in zip(got["nodes"], want.nodes):
        assert (g["prim"], g["stage"], g["unit"], g["src"], g["gpus"]) == (w.prim, w.stage, w.unit, w.src, w.gpus)
        assert g["cost"] == w.cost and g["start"] == w.start and g["finish"] == w.finish
    assert got["edges"] == [tuple(e) for e in want.edges]
    assert got["target_units"] == want.target_units
    assert got["l_tran"] == want.l_tran and got["n_resource_edges"] == want.n_resource_edges
    return True


def test_paper_example_and_small_cases():
    assert compare([st(1, 4, 8, 1, range(32), 8, 2, 1, range(16), state=3200.0)])
    assert compare([st(2, 1, 1, 1, [0], 1, 1, 1, [1]), st(2, 1, 1, 1, [1], 1, 1, 1, [2])])
    assert not compare([st(2, 1, 1, 2, [0, 1], 1, 1, 2, [2, 3]), st(2, 1, 1, 2, [2, 3], 1, 1, 2, [0, 1])])


@pytest.mark.parametrize("seed", range(6))
def test_random_scenarios(seed):
    rng = random.Random(100 + seed)
    feasible = 0
    for _ in range(150):
        feasible += compare(random_scenario(rng, n_gpus=rng.choice([8, 16, 32])))
    assert feasible > 50


def test_invalid_input_rejected():
    with pytest.raises(emu.EmuError) as e:
        lib_plan([st(2, 1, 1, 2, [0, 0], 1, 1, 1, [0])])
    assert e.value.code == -11
    with pytest.raises(emu.EmuError) as e:      # two training stages holding one GPU
        lib_plan([st(2, 1, 1, 1, [0], 1, 1, 1, [0]), st(2, 1, 1, 1, [0], 1, 1, 1, [1])])
    assert e.value.code == -11


def ppo_1024():
    """Four model-stages on 1,024 GPUs (8 per node): rollout TP4 -> TP8, reward/reference PP2 -> PP4,
    actor training PP4 -> PP2 on fewer GPUs, critic training DP 64 -> 80 onto the GPUs the actor frees."""
    return [
        st(0, 4, 1, 128, range(512), 8, 1, 64, range(512), state=16e9),
        st(1, 4, 2, 32, range(512, 768), 4, 4, 16, range(512, 768), state=16e9),
        st(2, 4, 4, 32, range(512), 4, 2, 48, range(384), state=64e9),
        st(2, 4, 2, 64, range(512, 1024), 4, 2, 80, range(384, 1024), state=64e9),
    ]


def test_1024_gpu_scenario_and_planning_time():
    links = Links(gpus_per_node=8, intra_bw=300e9, inter_bw=25e9, hbm_bw=5e12, setup_s=0.05)
    stages = ppo_1024()
    assert compare(stages, links)
    got = lib_plan(stages, links)
    assert got["n_resource_edges"] > 0
    lib_ms = sorted(lib_plan(stages, links)["plan_ms"] for _ in range(20))[10]
    t = time.perf_counter()
    plan(stages, links)
    oracle_ms = (time.perf_counter() - t) * 1e3
    print(f"1024-GPU transition DAG: {len(got['nodes'])} primitives, {len(got['edges'])} edges "
          f"({got['n_resource_edges']} resource), L_tran {got['l_tran']:.3f} s; "
          f"planning {lib_ms:.3f} ms (library, median of 20) vs {oracle_ms:.1f} ms (oracle)")
    assert lib_ms < 200


def test_fuzz_malformed_and_random_inputs_same_verdict():
    """Random valid scenarios, about a third of them then malformed in one way (a zero or negative
    degree, a GPU list one id too long or too short, a repeated GPU id, a GPU shared with another
    model-stage of the same kind): the library never crashes, and its verdict (a DAG, EMU_ERR_ARG or
    EMU_ERR_INFEASIBLE) is the oracle's (a DAG, ValueError or Infeasible); where both plan, the DAGs are
    identical."""
    rng = random.Random(29)
    seen = {"ok": 0, "arg": 0, "infeasible": 0}
    for _ in range(600):
        stages = random_scenario(rng)
        if rng.random() < 0.35:
            s = rng.choice(stages)
            how = rng.randrange(4)
            if how == 0:
                setattr(s, rng.choice(["tp", "pp", "dp", "tgt_tp", "tgt_pp", "tgt_dp"]), rng.choice([0, -1]))
            elif how == 1:
                lst = rng.choice([s.gpus, s.tgt_gpus])
                if rng.random() < 0.5 or len(lst) < 2:
                    lst.append(99)
                else:
                    lst.pop()
            elif how == 2 and len(s.gpus) > 1:
                s.gpus[1] = s.gpus[0]
            else:
                other = st(s.kind, 1, 1, 1, [s.gpus[0]], 1, 1, 1, [50], state=64.0)
                stages.append(other)
        try:
            want = plan(stages, L)
            verdict = "ok"
        except ValueError:
            verdict = "arg"
        except Infeasible:
            verdict = "infeasible"
        try:
            got = lib_plan(stages)
            got_v = "ok"
        except emu.EmuError as e:
            got_v = {emu.STATUS_CODE["EMU_ERR_ARG"]: "arg", emu.ERR_INFEASIBLE: "infeasible"}[e.code]
        assert got_v == verdict, stages
        if verdict == "ok":
            assert got["l_tran"] == want.l_tran and len(got["nodes"]) == len(want.nodes)
        seen[verdict] += 1
    assert min(seen.values()) >= 20, seen


def test_negative_gpu_ids_rejected():
    with pytest.raises(emu.EmuError) as e:
        lib_plan([st(2, 1, 1, 1, [-3], 1, 1, 1, [0])])
    assert e.value.code == emu.STATUS_CODE["EMU_ERR_ARG"]
