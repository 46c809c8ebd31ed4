"""Configuration selection for one encoder layer (Sec. "Configuration
Selection"), re-targeted to this library's knobs.

The paper benchmarks every configuration of every operator, builds a
directed acyclic graph whose nodes are the data layouts between operators
and whose edges are operators weighted by their fastest configuration for
that pair of layouts, runs a single-source shortest path from the input to
the output, and saves the path to a configuration file used when training
starts.  Forward and backward passes are optimised separately.

Here the knobs a caller can change are each contraction's kernel, tile and
split factor (plan entries, ``lib.Plan``), the grouping of the attention-score
steps (``attn_path``: separate launches, scores kept on chip, or scores with
the next contraction in the same launch), and the fused operators' layout
and reduction choices (``lib.LayoutChoice``): whether the LayerNorm-2
backward and the activation backward also write their output transposed
for the weight-gradient contraction that reads it (which then reads it
contiguous along the tokens: a different contraction, with its own
candidates), the LayerNorm backward's reduction form, and the lanes per
row of the LayerNorm kernels.  The graph's nodes are the points between
consecutive operators; each attention grouping and each layout combination
is an alternative chain of operators between shared points (a stage whose
time depends on the layout appears once per layout as its own stage).
Timings come from the library's per-launch events.  A contraction shape
that occurs at several points of a pass is one decision: its candidates are
timed over all its occurrences together, and its node sits at the first
occurrence.

Usage (on the GPU):
    python -m paper_2007_00072_amd.tune --workload bert_large_f16 --out plan.json
"""
from __future__ import annotations

import argparse
import heapq
import json
import math
import time
from collections import OrderedDict, defaultdict
from typing import Dict, List, Sequence, Tuple

TILE_CFGS = list(range(26))
# A measured difference smaller than the run-to-run spread of these timings
# does not move a contraction off the library's own choice.
KEEP_BUILTIN = 0.97
SPLITS = (1, 2, 4)
ATTN_PATHS = (1, 2, 3)   # 1 separate, 2 scores on chip, 3 scores + next contraction
SWEEP_PATH = 3           # the grouping under which contraction candidates are swept


# --------------------------------------------------------------- the graph
def shortest_path(n_nodes: int, edges: Sequence[Tuple[int, int, float, object]], src: int, dst: int):
    """Dijkstra on a graph with non-negative weights.  Returns (cost,
    [edge payloads along the path]); (inf, []) if dst is unreachable."""
    adj = defaultdict(list)
    for u, v, w, pay in edges:
        if w < 0:
            raise ValueError("negative edge weight")
        adj[u].append((v, w, pay))
    dist = [math.inf] * n_nodes
    back = [None] * n_nodes
    dist[src] = 0.0
    heap = [(0.0, src)]
    while heap:
        d, u = heapq.heappop(heap)
        if d > dist[u]:
            continue
        for v, w, pay in adj[u]:
            if d + w < dist[v]:
                dist[v] = d + w
                back[v] = (u, pay)
                heapq.heappush(heap, (dist[v], v))
    if math.isinf(dist[dst]):
        return math.inf, []
    path, v = [], dst
    while v != src:
        u, pay = back[v]
        path.append(pay)
        v = u
    return dist[dst], path[::-1]


def build_graph(chains: Dict[int, List[str]], costs: Dict[str, Dict[object, float]]):
    """Graph of one pass: `chains` maps each attention grouping to its list
    of operator stages (the stages outside the attention block are shared
    by every chain and appear in each list in order); `costs[stage]` maps
    each configuration of a stage to its time (a stage with one fixed
    configuration has one entry).  Nodes are the points between stages:
    shared points are shared by all chains, points inside a grouping's
    private stretch belong to that grouping.  Each configuration of a stage
    is one edge.  Returns (n_nodes, edges, src, dst); an edge payload is
    (path, stage, configuration)."""
    ids = {}

    def node(key):
        if key not in ids:
            ids[key] = len(ids)
        return ids[key]

    edges = []
    for path, stages in chains.items():
        for i, st in enumerate(stages):
            before = _point_key(chains, path, stages, i)
            after = _point_key(chains, path, stages, i + 1)
            for cfg, t in costs[st].items():
                edges.append((node(before), node(after), t, (path, st, cfg)))
    src = node(("pt", ()))
    dst = node(("end",))
    for path, stages in chains.items():
        edges.append((node(_point_key(chains, path, stages, len(stages))), dst, 0.0, (path, None, None)))
    return len(ids), edges, src, dst


def _shared_prefix(chains, prefix) -> bool:
    return all(list(s[: len(prefix)]) == list(prefix) for s in chains.values())


def _point_key(chains, path, stages, i):
    """Key of the point after the first i stages of a chain (a layout
    between two operators): shared by every chain when the stages before it
    are the same in every chain, or when the stages after it are; otherwise
    the chain's own."""
    prefix, suffix = list(stages[:i]), list(stages[i:])
    if _shared_prefix(chains, prefix):
        return ("pt", tuple(prefix))
    if all(list(s[len(s) - len(suffix):]) == suffix for s in chains.values()) and suffix:
        return ("sfx", tuple(suffix))
    if not suffix:
        return ("tail", path)
    return ("pt", path, tuple(prefix))


def select(chains: Dict[int, List[str]], costs: Dict[str, Dict[object, float]]):
    """Shortest path of one pass: (time, attention grouping, {stage: config})."""
    n, edges, src, dst = build_graph(chains, costs)
    t, path = shortest_path(n, edges, src, dst)
    if not path:
        raise RuntimeError("no configuration reaches the output")
    cfgs = {st: cfg for _, st, cfg in path if st is not None}
    # shared stages' edges exist once per chain; the grouping is the chain
    # whose stages the path took
    grouping = next(p for p, stages in chains.items() if set(stages) == set(cfgs) and len(stages) == len(cfgs))
    return t, grouping, cfgs


# ------------------------------------------------------------ measurement
class _Layer:
    """A BERT-style layer with seeded inputs; fwd+bwd runs with per-launch timing."""

    def __init__(self, workload: str, shape=None, **desc_over):
        import torch
        from .inputs import WORKLOADS, make_activation, make_params
        from .runner import EncoderLayer, desc_for
        self.torch = torch
        wl = WORKLOADS[workload]
        if shape is not None:
            wl = wl.with_(shape=shape)
        self.wl = wl
        self.layer = EncoderLayer(desc_for(wl, 0, **desc_over), make_params(wl), "cuda")
        self.x = make_activation(wl, 0).to("cuda")
        self.dy = make_activation(wl, 1).to("cuda")

    def use(self, entries=(), attn_path: int = 0, layout=None):
        """Runs the layer with this plan from now on (nothing: built-in choices)."""
        from . import lib
        lib.set_plan(self.layer.desc, lib.Plan(entries, attn_path, layout)
                     if (entries or attn_path or layout) else None)

    def step(self):
        self.layer.forward(self.x)
        self.layer.backward(self.x, self.dy)

    def timed(self, reps: int) -> Dict[str, float]:
        """Mean ms per launch label (an operator's extra launches, e.g. a
        split-k reduce, are added to it) over `reps` steps.  Labels are
        canonical (see CANON, FOLD): a contraction with an operator in its
        epilogue and the same contraction followed by that operator's own
        launch are one stage."""
        from . import lib
        self.step()
        self.torch.cuda.synchronize()
        lib.dm_trace_enable(True)
        for _ in range(reps):
            self.step()
        self.torch.cuda.synchronize()
        recs = lib.trace_records()
        lib.dm_trace_enable(False)
        tot = defaultdict(float)
        for lab, _sub, ms in recs:
            tot[canonical(lab)] += ms
        return {k: v / reps for k, v in tot.items()}

    def launches(self):
        """(label, ContractChoice) of every contraction one step launches."""
        from . import lib
        lib.dm_trace_enable(True)
        lib.plan_log(True)
        self.step()
        self.torch.cuda.synchronize()
        recs = lib.plan_log_read()
        lib.plan_log(False)
        lib.dm_trace_enable(False)
        return [(canonical(r.label.decode()), r) for r in recs]


# Contractions that take an element-wise operator into their epilogue where
# their kernel allows: the fused launch's label and the operator's own
# launch (when the kernel cannot take it) both map to the contraction's
# stage, so every configuration of the contraction is timed with the
# operator's cost included.
CANON = {"F7+8 linear1_bias_act": "F7 linear1", "B3+5 linear2_dx_act_bwd": "B3 linear2_dx"}
FOLD = {"F8 bias_act": "F7 linear1", "B5 act_bwd": "B3 linear2_dx"}


def canonical(label: str) -> str:
    label = CANON.get(label, label)
    return FOLD.get(label, label)


def _is_fwd(label: str) -> bool:
    return label.startswith("F")


# Stages whose time depends on a layout choice, and the fields it depends on
# (the stage appears once per value of those fields in the graph).
LAYOUT_STAGES = {
    "F6 bdrln1": ("ln_lanes",), "F10 bdrln2": ("ln_lanes",),
    "B1-2 ln2_bwd": ("ln_bwd_form", "dO_transposed", "ln_lanes"), "B8-10 ln1_bwd": ("ln_bwd_form", "ln_lanes"),
    "B4 linear2_dw": ("dO_transposed",), "B3 linear2_dx": ("dH_transposed",), "B7 linear1_dw": ("dH_transposed",),
    "B colsum finish": ("ln_bwd_form", "dH_transposed"),
}


def layout_options(I: int, dtype: str, T: int):
    """(forward lane counts, backward layout combinations) a layer of width
    I in storage type dtype can take; every combination is complete
    (ln_lanes filled in later from the forward's choice)."""
    sixteen = dtype != "f32"
    split_ok = sixteen and I % 64 == 0 and 320 <= I <= 1024
    lanes = [64, 32, 16] if 256 < I <= 1024 else [64]
    combos = []
    for form in ([2, 1] if split_ok else [1]):
        for dot in ([1, 0] if form == 2 else [0]):
            for dht in ([0, 1] if sixteen and T % 8 == 0 else [0]):
                combos.append({"ln_bwd_form": form, "dO_transposed": dot, "dH_transposed": dht})
    return lanes, combos


def stage_name(label: str, layout: dict) -> str:
    fields = LAYOUT_STAGES.get(label)
    if not fields:
        return label
    return label + " [" + ",".join(f"{f}={layout[f]}" for f in fields) + "]"


def tune(workload: str, reps: int = 3, log=print, shape=None, tile_cfgs=TILE_CFGS, splits=SPLITS):
    """Measure and select; returns the plan as a dict (see load_plan).
    shape: run the workload's layer at other sizes; tile_cfgs / splits: the
    candidates tried for every contraction."""
    from . import lib
    L = _Layer(workload, shape)
    L.use()
    t0 = time.time()
    for _ in range(5):  # clocks and caches settle before anything is timed
        L.step()
    L.torch.cuda.synchronize()
    s = L.wl.shape
    lanes_opts, combos = layout_options(s.I, L.wl.dtype, s.B * s.J)
    # forward: each lane count (the LayerNorm forward's reduction width)
    lane_times = {}
    for ln in lanes_opts:
        L.use((), 0, {"ln_lanes": ln})
        tm = L.timed(reps)
        lane_times[ln] = tm.get("F6 bdrln1", 0.0) + tm.get("F10 bdrln2", 0.0)
    lanes = min(lane_times, key=lane_times.get)
    for c in combos:
        c["ln_lanes"] = lanes
    fwd_layout = dict(combos[0])
    # every (attention grouping, layout combination): per-stage times and
    # the contractions each stage launches
    runs = {}
    for p in ATTN_PATHS:
        for li, lay in enumerate(combos):
            L.use((), p, lay)
            tm = L.timed(reps)
            runs[(p, li)] = (tm, L.launches())
    builtin_layout = {"ln_bwd_form": -1, "dO_transposed": -1, "dH_transposed": -1, "ln_lanes": -1}
    L.use()
    base = L.timed(reps)
    # stage names per run, fixed-cost stage times (averaged over the runs
    # that have the stage), and where each contraction shape occurs
    # (contractions are swept where they run under the library's own
    # grouping; those of the other groupings keep their measured time)
    chains_f, chains_b = {}, {}
    fixed = defaultdict(list)
    where: Dict[tuple, List[str]] = OrderedDict()
    occurs_in: Dict[tuple, int] = {}
    label_key = {}
    # a contraction shape is swept under the first layout where it occurs;
    # a layout-dependent stage of it under another layout (e.g. Linear-2 dX
    # when dH is written transposed and the activation backward runs on its
    # own) keeps its measured time
    for (p, li), (tm, launches) in runs.items():
        if p == SWEEP_PATH:
            for lab, r in launches:
                occurs_in.setdefault(r.key(), li)
    for (p, li), (tm, launches) in runs.items():
        lay = combos[li]
        names = {lab: stage_name(lab, lay) for lab in tm}
        if p == SWEEP_PATH:
            for lab, r in launches:
                if occurs_in[r.key()] != li and stage_name(lab, lay) not in label_key:
                    continue
                st = names.get(lab, stage_name(lab, lay))
                label_key[st] = r.key()
                where.setdefault(r.key(), [])
                if st not in where[r.key()]:
                    where[r.key()].append(st)
    for (p, li), (tm, launches) in runs.items():
        lay = combos[li]
        names = {lab: stage_name(lab, lay) for lab in tm}
        for lab, t in tm.items():
            if names[lab] not in label_key:
                fixed[names[lab]].append(t)
        fwd = [names[l] for l in tm if _is_fwd(l)]
        bwd = [names[l] for l in tm if not _is_fwd(l)]
        if li == 0:
            chains_f[p] = fwd
        chains_b[(p, li)] = bwd
    # candidates of every contraction shape, timed over all its occurrences
    # under a layout where it occurs
    shape_costs: Dict[tuple, Dict[tuple, float]] = {}
    for key, sts in where.items():
        lay = combos[occurs_in[key]]
        seen = {}
        for cfg in tile_cfgs:
            for sp in splits:
                e = lib.ContractChoice(*key, cfg, sp)
                L.use([e], 0, lay)
                ran = {(r.tile_cfg, r.splits) for lab, r in L.launches() if r.key() == key}
                if len(ran) != 1:
                    continue
                eff = ran.pop()
                if eff in seen:
                    continue
                tm = L.timed(reps)
                names = {lab: stage_name(lab, lay) for lab in tm}
                seen[eff] = sum(t for lab, t in tm.items() if names[lab] in sts)
        L.use((), 0, lay)
        builtin = next(((r.tile_cfg, r.splits) for lab, r in L.launches() if r.key() == key), None)
        if builtin in seen:
            seen[builtin] *= KEEP_BUILTIN
        shape_costs[key] = seen
        best = min(seen.items(), key=lambda kv: kv[1])
        log(f"  {sts}: {len(seen)} configurations, best {best[0]} {best[1] * 1e3:.1f} us (built-in {builtin})")
    L.use()

    def costs_for(chains):
        # a contraction shape carries its candidates at its first stage of a
        # chain; its later stages in the same chain cost nothing more
        costs, firsts, laters = {}, set(), set()
        for stages in chains.values():
            seen_keys = set()
            for st in stages:
                k = label_key.get(st)
                if k in shape_costs:
                    (laters if k in seen_keys else firsts).add(st)
                    seen_keys.add(k)
        if firsts & laters:
            raise RuntimeError(f"stages both first and repeated: {sorted(firsts & laters)}")
        for stages in chains.values():
            for st in stages:
                if st in firsts:
                    costs[st] = {("cfg",) + c: t for c, t in shape_costs[label_key[st]].items()}
                elif st in laters:
                    costs[st] = {("same",): 0.0}
                else:
                    costs[st] = {("fixed",): sum(fixed[st]) / len(fixed[st])}
        return costs

    result = {"workload": workload, "passes": {}}
    chosen = {}
    # one grouping knob and one layout serve both passes: per grouping, the
    # forward's best and the backward's best over the layouts; the grouping
    # with the lower total wins
    cf, cb = costs_for(chains_f), costs_for(chains_b)
    totals = {}
    for p in ATTN_PATHS:
        tf, _, cfg_f = select({p: chains_f[p]}, cf)
        tb, key_b, cfg_b = select({k: v for k, v in chains_b.items() if k[0] == p}, cb)
        totals[p] = (tf + tb, tf, tb, key_b[1], cfg_f, cfg_b)
    attn_path = min(totals, key=lambda q: totals[q][0])
    _, tf, tb, li, cfg_f, cfg_b = totals[attn_path]
    layout = dict(combos[li])
    for pass_name, t, cfgs in (("forward", tf, cfg_f), ("backward", tb, cfg_b)):
        for st, c in cfgs.items():
            if c[0] == "cfg" and st in label_key:
                chosen[label_key[st]] = c[1:]
        result["passes"][pass_name] = {"predicted_ms": t, "attn_path": attn_path,
                                        "stages": {st: list(c) for st, c in cfgs.items()}}
    # the backward's best time under each layout (this grouping): the
    # measured value of each layout choice
    result["layout_table"] = []
    for k in sorted(k for k in chains_b if k[0] == attn_path):
        t, _, _ = select({k: chains_b[k]}, cb)
        result["layout_table"].append(dict(combos[k[1]], backward_ms=round(t, 4)))
    result["lane_table"] = {str(k): round(v, 4) for k, v in lane_times.items()}
    entries = []
    for key, (cfg, sp) in chosen.items():
        e = lib.ContractChoice(*key, cfg, sp)
        e.label = ",".join(where[key]).encode()[:47]
        entries.append(e)
    result["attn_path"] = attn_path
    result["layout"] = layout
    result["entries"] = [dict(M=e.M, N=e.N, K=e.K, batch=e.batch, dtype=e.dtype, a_kcontig=e.a_kcontig,
                              b_kcontig=e.b_kcontig, tile_cfg=e.tile_cfg, splits=e.splits,
                              label=e.label.decode()) for e in entries]
    result["builtin_ms"] = sum(base.values())
    # Q/K/V projection grouping (Sec. "Algebraic Fusion"), a property of the
    # layer: the grouping with the least projection time over both passes
    table = fusion_table(workload, reps, shape)
    result["qkv_fusion_table"] = table
    result["qkv_fusion"] = min(table, key=lambda f: table[f]["forward"] + table[f]["backward"])
    L.use(entries, attn_path, layout)
    result["planned_ms"] = sum(L.timed(reps).values())
    L.use()
    result["tuning_seconds"] = round(time.time() - t0, 1)
    return result


FUSIONS = {0: "QKV fused", 1: "QK fused", 2: "unfused"}


def fusion_table(workload: str, reps: int = 3, shape=None):
    """Forward (Q/K/V projections) and backward (their dX and dW) time in
    ms of each projection grouping, built-in configurations (the analogue
    of the paper's algebraic-fusion table)."""
    out = {}
    for f in FUSIONS:
        L = _Layer(workload, shape, qkv_fusion=f)
        for _ in range(10):
            L.step()
        tm = L.timed(max(reps, 10))
        # backward: dX and dW of the projections (the encoder launches the
        # first group's dW together with the output projection's dW)
        out[f] = {"forward": tm.get("F1 qkv", 0.0),
                  "backward": tm.get("B18 qkv_dx", 0.0) + tm.get("B19 qkv_dw", 0.0) +
                  tm.get("B12+19 out_dw+qkv_dw", 0.0)}
        del L
    return out


def load_plan(path: str):
    """The plan a tuning run saved: (its dict, a lib.Plan to name in a
    descriptor)."""
    from . import lib
    with open(path) as f:
        plan = json.load(f)
    entries = [lib.ContractChoice(e["M"], e["N"], e["K"], e["batch"], e["dtype"], e["a_kcontig"], e["b_kcontig"],
                                  e["tile_cfg"], e["splits"]) for e in plan["entries"]]
    return plan, lib.Plan(entries, int(plan["attn_path"]), plan.get("layout"))


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="bert_large_f16")
    ap.add_argument("--reps", type=int, default=3)
    ap.add_argument("--out", default=None)
    ap.add_argument("--fusion-table", action="store_true", help="only time the Q/K/V projection groupings")
    a = ap.parse_args()
    if a.fusion_table:
        t = fusion_table(a.workload, a.reps)
        print("grouping      forward us  backward us")
        for f, r in t.items():
            print(f"{FUSIONS[f]:12s} {r['forward'] * 1e3:10.1f} {r['backward'] * 1e3:12.1f}", flush=True)
        return 0
    if not a.out:
        ap.error("--out is required")
    res = tune(a.workload, a.reps, log=lambda s: print(s, flush=True))
    with open(a.out, "w") as f:
        json.dump(res, f, indent=1)
    print(f"built-in {res['builtin_ms']:.3f} ms, planned {res['planned_ms']:.3f} ms (sum of launches), "
          f"attn_path {res['attn_path']}, layout {res['layout']}, {len(res['entries'])} entries, "
          f"{res['tuning_seconds']} s", flush=True)
    return 0


if __name__ == "__main__":
    raise SystemExit(main())
