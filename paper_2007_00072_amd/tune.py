"""Configuration selection for one encoder layer (Sec. "Configuration
Selection"), re-targeted to this library's knobs.

The paper benchmarks every configuration of every operator, builds a
directed acyclic graph whose nodes are the data layouts between operators
and whose edges are operators weighted by their fastest configuration for
that pair of layouts, runs a single-source shortest path from the input to
the output, and saves the path to a configuration file used when training
starts.  Forward and backward passes are optimised separately.

Here the knobs a caller can change are each contraction's kernel, tile and
split factor (plan entries, ``lib.Plan``) and the grouping of the attention-score
steps (``attn_path``: separate launches, scores kept on chip, or scores with
the next contraction in the same launch).  The tensors between operators
keep one layout whatever the configuration, so the graph's layout nodes are
the points between consecutive operators; the attention-score groupings are
alternative chains of operators between the same two points.  Timings come
from the library's per-launch events.  A contraction shape that occurs at
several points of a pass is one decision: its candidates are timed over all
its occurrences together, and its node sits at the first occurrence.

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

TILE_CFGS = list(range(20))
# A measured difference smaller than the run-to-run spread of these timings
# does not move a contraction off the library's own choice.
KEEP_BUILTIN = 0.97
SPLITS = (1, 2, 4)
ATTN_PATHS = (1, 2, 3)   # 1 separate, 2 scores on chip, 3 scores + next contraction


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

    def use(self, entries=(), attn_path: int = 0):
        """Runs the layer with this plan from now on (nothing: built-in choices)."""
        from . import lib
        lib.set_plan(self.layer.desc, lib.Plan(entries, attn_path) if (entries or attn_path) else None)

    def step(self):
        self.layer.forward(self.x)
        self.layer.backward(self.x, self.dy)

    def timed(self, reps: int) -> Dict[str, float]:
        """Mean ms per launch label (an operator's extra launches, e.g. a
        split-k reduce, are added to it) over `reps` steps."""
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
            tot[lab] += ms
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
        return [(r.label.decode(), r) for r in recs]


def _is_fwd(label: str) -> bool:
    return label.startswith("F")


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
    # attention groupings: which labels each produces, and their times
    grouping_times, grouping_labels = {}, {}
    for p in ATTN_PATHS:
        L.use((), p)
        tm = L.timed(reps)
        grouping_times[p] = tm
        grouping_labels[p] = list(tm.keys())
    L.use()
    base = L.timed(reps)
    launches = L.launches()
    # contraction shapes and the labels at which each occurs
    where: Dict[tuple, List[str]] = OrderedDict()
    choice_of = {}
    for lab, r in launches:
        where.setdefault(r.key(), [])
        if lab not in where[r.key()]:
            where[r.key()].append(lab)
        choice_of[r.key()] = r
    # candidates of every contraction shape, timed over all its occurrences
    shape_costs: Dict[tuple, Dict[tuple, float]] = {}
    for key, labs in where.items():
        seen = {}
        for cfg in tile_cfgs:
            for sp in splits:
                e = lib.ContractChoice(*key, cfg, sp)
                L.use([e], 0)
                ran = {(r.tile_cfg, r.splits) for lab, r in L.launches() if r.key() == key}
                if len(ran) != 1:
                    continue
                eff = ran.pop()
                if eff in seen:
                    continue
                tm = L.timed(reps)
                seen[eff] = sum(tm.get(lab, 0.0) for lab in labs)
        builtin = (choice_of[key].tile_cfg, choice_of[key].splits)
        if builtin in seen:
            seen[builtin] *= KEEP_BUILTIN
        shape_costs[key] = seen
        best = min(seen.items(), key=lambda kv: kv[1])
        log(f"  {labs}: {len(seen)} configurations, best {best[0]} {best[1] * 1e3:.1f} us "
            f"(built-in {(choice_of[key].tile_cfg, choice_of[key].splits)} "
            f"{sum(base.get(l, 0.0) for l in labs) * 1e3:.1f} us)")
    L.use()
    # one graph per pass; contraction stages carry their shape's candidates
    # at the first occurrence, later occurrences cost nothing
    label_key = {}
    for key, labs in where.items():
        for lab in labs:
            label_key[lab] = key
    first = {labs[0] for labs in where.values()}
    result = {"workload": workload, "passes": {}}
    chosen = {}
    attn_total = {p: 0.0 for p in ATTN_PATHS}
    per_pass = {}
    for pass_name, in_pass in (("forward", _is_fwd), ("backward", lambda l: not _is_fwd(l))):
        chains, costs = {}, {}
        for p in ATTN_PATHS:
            stages = [l for l in grouping_labels[p] if in_pass(l)]
            chains[p] = stages
            for st in stages:
                if st in label_key and label_key[st] in shape_costs:
                    # a shape's occurrence inside one grouping only is timed per grouping
                    if st in first:
                        costs[st] = {("cfg",) + c: t for c, t in shape_costs[label_key[st]].items()}
                    else:
                        costs[st] = {("same",): 0.0}
                else:
                    costs[st] = {("fixed", p): grouping_times[p][st]}
        t, grouping, cfgs = select(chains, costs)
        per_pass[pass_name] = (t, grouping, cfgs)
        for st, c in cfgs.items():
            if c[0] == "cfg" and st in label_key:
                chosen[label_key[st]] = c[1:]
        result["passes"][pass_name] = {"predicted_ms": t, "attn_path": grouping,
                                        "stages": {st: list(c) for st, c in cfgs.items()}}
        for p in ATTN_PATHS:
            sub = {p: chains[p]}
            try:
                attn_total[p] += select(sub, costs)[0]
            except RuntimeError:
                attn_total[p] = math.inf
    # one grouping knob serves both passes: the one with the lower total
    groupings = {v[1] for v in per_pass.values()}
    attn_path = groupings.pop() if len(groupings) == 1 else min(attn_total, key=attn_total.get)
    entries = []
    for key, (cfg, sp) in chosen.items():
        e = lib.ContractChoice(*key, cfg, sp)
        e.label = ",".join(where[key]).encode()[:47]
        entries.append(e)
    result["attn_path"] = attn_path
    result["entries"] = [dict(M=e.M, N=e.N, K=e.K, batch=e.batch, dtype=e.dtype, a_kcontig=e.a_kcontig,
                              b_kcontig=e.b_kcontig, tile_cfg=e.tile_cfg, splits=e.splits,
                              label=e.label.decode()) for e in entries]
    result["builtin_ms"] = sum(base.values())
    # Q/K/V projection grouping (Sec. "Algebraic Fusion"), a property of the
    # layer: the grouping with the least projection time over both passes
    table = fusion_table(workload, reps, shape)
    result["qkv_fusion_table"] = table
    result["qkv_fusion"] = min(table, key=lambda f: table[f]["forward"] + table[f]["backward"])
    L.use(entries, attn_path)
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
    return plan, lib.Plan(entries, int(plan["attn_path"]))


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
          f"attn_path {res['attn_path']}, {len(res['entries'])} entries, {res['tuning_seconds']} s", flush=True)
    return 0


if __name__ == "__main__":
    raise SystemExit(main())
