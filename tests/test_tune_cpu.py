"""Configuration selection (paper_2007_00072_amd/tune.py) on the CPU: the
graph construction plus shortest path equal brute-force enumeration of
every attention grouping and every configuration of every stage."""
import itertools
import math
import random

import pytest

from paper_2007_00072_amd import tune


def brute_force(chains, costs):
    best = (math.inf, None, None)
    for p, stages in chains.items():
        options = [list(costs[st].items()) for st in stages]
        for combo in itertools.product(*options):
            t = sum(c[1] for c in combo)
            if t < best[0]:
                best = (t, p, {st: c[0] for st, c in zip(stages, combo)})
    return best


def random_case(rng):
    pre = [f"F{i}" for i in range(rng.randint(0, 3))]
    post = [f"G{i}" for i in range(rng.randint(0, 3))]
    mids = {1: ["a1", "a2", "a3"], 2: ["b1", "a3"], 3: ["c1"]}
    chains = {p: pre + m + post for p, m in mids.items()}
    costs = {}
    for stages in chains.values():
        for st in stages:
            if st not in costs:
                costs[st] = {(k,): rng.uniform(0.1, 10.0) for k in range(rng.randint(1, 4))}
    return chains, costs


@pytest.mark.parametrize("seed", range(40))
def test_selection_equals_brute_force(seed):
    rng = random.Random(seed)
    chains, costs = random_case(rng)
    t, p, cfgs = tune.select(chains, costs)
    bt, bp, bcfgs = brute_force(chains, costs)
    assert t == pytest.approx(bt, rel=1e-12)
    # the chosen stages are exactly one chain's, each at one of its configurations
    assert set(cfgs) == set(chains[p])
    assert sum(costs[st][c] for st, c in cfgs.items()) == pytest.approx(t, rel=1e-12)


def test_shared_points_are_merged():
    chains = {1: ["x", "a", "y"], 2: ["x", "b", "c", "y"]}
    costs = {s: {(0,): 1.0} for s in "xabcy"}
    n, edges, src, dst = tune.build_graph(chains, costs)
    # points: start, after x (shared), after a / after b / after c, before y (shared suffix), ends, sink
    starts = {u for u, v, w, pay in edges if pay[1] == "x"}
    assert starts == {src}
    y_from = {u for u, v, w, pay in edges if pay[1] == "y"}
    assert len(y_from) == 1


def test_shortest_path_rejects_negative_weights():
    with pytest.raises(ValueError):
        tune.shortest_path(2, [(0, 1, -1.0, None)], 0, 1)
    assert tune.shortest_path(3, [(0, 1, 1.0, "e")], 0, 2) == (math.inf, [])


def test_saved_plans_are_well_formed():
    # every plan shipped with the package names a known workload and only
    # valid configurations (what plan_create accepts)
    import glob
    import json
    import os
    from paper_2007_00072_amd.inputs import WORKLOADS
    plans = glob.glob(os.path.join(os.path.dirname(tune.__file__), "plans", "*.json"))
    assert len(plans) >= 2
    for path in plans:
        plan = json.load(open(path))
        assert plan["workload"] in WORKLOADS, path
        assert os.path.basename(path) == plan["workload"] + ".json"
        assert 0 <= int(plan["attn_path"]) <= 3 and int(plan.get("qkv_fusion", 0)) in (0, 1, 2)
        assert plan["entries"]
        for e in plan["entries"]:
            assert 0 <= e["tile_cfg"] <= 25 and 1 <= e["splits"] <= 64, (path, e)
            assert e["M"] > 0 and e["N"] > 0 and e["K"] > 0 and e["batch"] >= 1


def layout_case(rng):
    # chains keyed by (attention grouping, layout combination): layout
    # choices rename the stages whose time they change, as the tuner does
    pre = ["F1", "F2"]
    groupings = {1: ["a1", "a2"], 2: ["b1"], 3: ["c1"]}
    layouts = [{"d": 1, "f": 2}, {"d": 0, "f": 2}, {"d": 0, "f": 1}]
    chains = {}
    for p, mid in groupings.items():
        for li, lay in enumerate(layouts):
            stages = pre + [f"LN [{lay['f']},{lay['d']}]", "W", f"Wd [{lay['d']}]"] + mid + ["G", f"fin [{lay['f']}]"]
            chains[(p, li)] = stages
    costs = {}
    for stages in chains.values():
        for st in stages:
            if st not in costs:
                costs[st] = {(k,): rng.uniform(0.1, 10.0) for k in range(rng.randint(1, 3))}
    return chains, costs


@pytest.mark.parametrize("seed", range(30))
def test_layout_selection_equals_brute_force(seed):
    rng = random.Random(1000 + seed)
    chains, costs = layout_case(rng)
    t, key, cfgs = tune.select(chains, costs)
    bt, bkey, _ = brute_force(chains, costs)
    assert t == pytest.approx(bt, rel=1e-12)
    assert set(cfgs) == set(chains[key])


def test_layout_options_and_stage_names():
    lanes, combos = tune.layout_options(1024, "f16", 4096)
    assert lanes == [64, 32, 16]
    # column-split form with and without dO^T, row form without it; dH^T on or off
    assert len(combos) == 6
    assert {(c["ln_bwd_form"], c["dO_transposed"]) for c in combos} == {(2, 1), (2, 0), (1, 0)}
    assert all(c["dO_transposed"] == 0 for c in combos if c["ln_bwd_form"] == 1)
    lanes, combos = tune.layout_options(32, "f32", 64)
    assert lanes == [64] and combos == [{"ln_bwd_form": 1, "dO_transposed": 0, "dH_transposed": 0}]
    lay = {"ln_bwd_form": 2, "dO_transposed": 1, "dH_transposed": 0, "ln_lanes": 64}
    assert tune.stage_name("B4 linear2_dw", lay) == "B4 linear2_dw [dO_transposed=1]"
    # Linear-2 dX takes the activation backward into its epilogue only when
    # dH is not written transposed: its stage depends on that choice
    assert tune.stage_name("B3 linear2_dx", lay) == "B3 linear2_dx [dH_transposed=0]"
    assert tune.stage_name("B6 linear1_dx", lay) == "B6 linear1_dx"


def test_canonical_labels_fold_epilogue_operators():
    # a fused launch and the unfused pair land on one stage
    assert tune.canonical("F7+8 linear1_bias_act") == tune.canonical("F7 linear1") == "F7 linear1"
    assert tune.canonical("F8 bias_act") == "F7 linear1"
    assert tune.canonical("B3+5 linear2_dx_act_bwd") == tune.canonical("B5 act_bwd") == "B3 linear2_dx"
    assert tune.canonical("B4 linear2_dw") == "B4 linear2_dw"
