#!/usr/bin/env python
"""Benchmark: forward + backward of the paper's hot path on one MI355X,
through the library's C ABI.  Default workload: one BERT-large post-LN
encoder layer (fp16, B=8, L=512, I=1024, H=16, P=64, FFN 4096, three
dropouts p=0.1).  --workload picks another: bert_base_bf16 (B=96, L=128),
bert_large_stack24_bf16 (24 layers, B=4, L=512, forward through all then
backward through all), mha_large_f16 (multi-head self-attention alone,
[I][B][J] layout), tiny_f32.

Prints one JSON line: ms per fwd+bwd step (inputs resident in HBM; with
--graph also the time of replaying the step captured as one HIP graph),
the roofline position of the dominant kernel (per-launch durations
measured with HIP events on the launch stream), the aggregate HBM rate of
the fused memory-bound operators, the data-movement reduction against the
operators one by one, the CPU oracle timed on a bounded sample, and the
paper's own speedups (other hardware) as context.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--graph] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "BERT-large layer fwd+bwd ms/iter; fused-kernel HBM GB/s vs peak"


def csrc_hash() -> str:
    h = hashlib.sha256()
    d = os.path.join(ROOT, "paper_2007_00072_amd", "csrc")
    for f in sorted(os.listdir(d)):
        h.update(f.encode())
        h.update(open(os.path.join(d, f), "rb").read())
    return h.hexdigest()[:16]


def traffic_for(label: str):
    """HBM bytes per launch of `label` from the committed counter summary, if
    it was taken on the current kernel sources."""
    p = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(p):
        return None
    try:
        t = json.load(open(p))
    except ValueError:
        return None
    e = t.get("kernels", {}).get(label)
    if not e or t.get("csrc_sha") != csrc_hash():
        return None
    return e.get("bytes_per_launch")


def host_cpu() -> dict:
    """The host the oracle runs on: CPU model, cores this process may use."""
    model = ""
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                model = ln.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:
        cores = os.cpu_count() or 1
    return {"cpu_model": model, "cores_available": cores, "OMP_NUM_THREADS": os.environ.get("OMP_NUM_THREADS")}


def cpu_baseline(wl, sample_b: int):
    """The oracle (float64, numpy) on the first `sample_b` sequences of the
    batch, forward + backward, scaled to ms per full step (per layer for a
    stack, times its layer count)."""
    from oracle import layer as OL
    from paper_2007_00072_amd.inputs import make_activation, make_params

    s = wl.shape
    params = {n: t.double().numpy() for n, t in make_params(wl).items()}
    x = make_activation(wl, 0).double().numpy()
    dy = make_activation(wl, 1).double().numpy()
    cut = (lambda a: a[:, :sample_b]) if wl.layout == "ibj" else (lambda a: a[:sample_b])
    x, dy = cut(x), cut(dy)
    cfg = OL.Config(B=sample_b, J=s.J, K=s.K, H=s.H, P=s.P, W=s.W, I=s.I, F=s.F, p_attn=wl.p_attn,
                    p_attn_out=wl.p_attn_out, p_ffn_out=wl.p_ffn_out, seed=wl.seed, eps=1e-12,
                    store_dtype=wl.dtype)
    t0 = time.perf_counter()
    if wl.kind == "mha":
        xi = x if wl.layout == "ibj" else x.transpose(2, 0, 1)
        di = dy if wl.layout == "ibj" else dy.transpose(2, 0, 1)
        _, cache = OL.mha_forward_ibj(xi, xi, xi, params, cfg)
        OL.mha_backward_ibj(di, cache, params, cfg)
    else:
        _, cache = OL.encoder_forward(x, params, cfg)
        OL.encoder_backward(dy, cache, params, cfg)
    dt = time.perf_counter() - t0
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = 1
    scale = s.B / sample_b * wl.n_layers
    whole = scale == 1
    what = "layer" if wl.kind == "encoder" else "attention"
    sample = (f"one full fwd+bwd step ({s.B} sequences)" if whole else
              f"first {sample_b} of {s.B} sequences of one {what}, fwd+bwd, scaled x{scale:g}"
              + (f" ({wl.n_layers} layers)" if wl.n_layers > 1 else ""))
    out = {"value": round(dt * 1e3 * scale, 1),
           "unit": "ms/iter" if whole else "ms/iter (extrapolated from sample)",
           "cores": threads, "kind": "oracle",
           "sample": sample + f"; float64 numpy, BLAS threads={threads}, element-wise steps single-threaded",
           "sample_seconds": round(dt, 2)}
    out.update(host_cpu())
    return out


PAPER_CONTEXT = {
    "encoder_layer": "1.30x forward+backward over PyTorch (7.01 ms against 9.14 ms), BERT-large layer, "
                     "B=8, L=512, one NVIDIA V100 16 GB, CUDA 10.1, fp16 data with fp32 accumulation "
                     "(Sec. End-to-End Performance, Table 5)",
    "full_bert": "1.19x end-to-end BERT-large pretraining over NVIDIA's BERT implementation, "
                 "128 V100 GPUs (Sec. End-to-End Performance; Supplement, End-to-end training)",
    "data_movement_reduction": "22.91% against the standard implementation, V100 (Sec. End-to-End Performance, "
                               "from Table 3's I/O columns)",
    "note": "context only: other hardware and other fusion; not the target",
}


def describe(wl) -> str:
    s = wl.shape
    if wl.kind == "mha":
        return (f"{wl.name}: multi-head self-attention fwd+bwd (fused Q/K/V, output bias), layout {wl.layout}, "
                f"B={s.B}, J=K={s.J}, I={s.I}, H={s.H}, P=W={s.P}, attention-probability dropout p={wl.p_attn}, "
                f"{wl.dtype}")
    layers = f"{wl.n_layers} encoder layers" if wl.n_layers > 1 else "encoder layer"
    return (f"{wl.name}: post-LN {layers} fwd+bwd, B={s.B}, L={s.J}, I={s.I}, H={s.H}, P={s.P}, FFN={s.F}, "
            f"GELU, dropout p={wl.p_attn} x3, {wl.dtype}")


def copy_rate_gbs(torch, dev, reps: int = 10) -> float:
    """HBM rate of a plain device-to-device copy of 1 GiB (read + write
    bytes over time), the practical ceiling beside the 8 TB/s peak."""
    n = 1 << 28
    src = torch.empty(n, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    rate = 2.0 * 4 * n * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del src, dst
    return rate


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="bert_large_f16")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample", type=int, default=0, help="sequences in the CPU-oracle sample (0: the whole batch)")
    ap.add_argument("--kernels-json", default=None, help="write the per-kernel table here")
    ap.add_argument("--graph", action="store_true",
                    help="also time replays of the step captured as one HIP graph (reported beside the "
                         "launch-by-launch time, after checking that a replay writes what an eager step writes)")
    ap.add_argument("--plan", default=None,
                    help="configuration plan written by paper_2007_00072_amd.tune (default: the built-in choices)")
    a = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if a.gpus != 1 or world != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1",
                          "n_gpus": a.gpus}))
        return 2

    import torch
    from paper_2007_00072_amd import dataflow, lib
    from paper_2007_00072_amd.inputs import WORKLOADS, make_activation, make_params
    from paper_2007_00072_amd.runner import EncoderLayer, desc_for

    wl = WORKLOADS[a.workload]
    s = wl.shape
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    plan_name, plan, cplan = "built-in", {}, None
    if a.plan:
        from paper_2007_00072_amd.tune import load_plan
        plan, cplan = load_plan(a.plan)
        if plan.get("workload") != wl.name:
            print(json.dumps({"error": f"plan {a.plan} was tuned for {plan.get('workload')}, not {wl.name}"}))
            return 2
        plan_name = os.path.basename(a.plan)
    outputs = []        # tensors a step writes (checked against a graph replay)
    grads = []          # parameter-gradient dicts
    if wl.kind == "mha":
        from paper_2007_00072_amd.runner import MultiHeadAttention
        att = MultiHeadAttention(desc_for(wl, self_attention=True, plan=cplan), make_params(wl), dev)
        x = make_activation(wl, 0).to(dev)
        dy = make_activation(wl, 1).to(dev)
        y, dx = torch.empty_like(x), torch.empty_like(x)
        outputs, grads = [y, dx], [att.grads]

        def step():
            att.forward(x, out=y)
            att.backward(x, dy, dq=dx)
        work = dataflow.mha(s, wl.dtype, wl.layout)
    else:
        desc_kw = dict(qkv_fusion=int(plan.get("qkv_fusion", 0)), plan=cplan)
        layers = []
        for li in range(wl.n_layers):
            layers.append(EncoderLayer(desc_for(wl, li, **desc_kw), make_params(wl, layer=li), dev,
                                       workspace=layers[0].ws if layers else None))
        x = make_activation(wl, 0).to(dev)
        dy = make_activation(wl, 1).to(dev)
        acts = [x] + [torch.empty_like(x) for _ in layers]
        dacts = [torch.empty_like(x) for _ in layers] + [dy]
        outputs, grads = [acts[-1], dacts[0]], [L.grads for L in layers]

        def step():
            for li, L in enumerate(layers):
                L.forward(acts[li], acts[li + 1])
            for li in reversed(range(len(layers))):
                layers[li].backward(acts[li], dacts[li + 1], dacts[li])
        work = dataflow.encoder_layer(s, wl.dtype)

    for _ in range(a.warmup):
        step()
    torch.cuda.synchronize()
    st = torch.cuda.current_stream()

    def timed(run):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        e0.record(st)
        for _ in range(a.steps):
            run()
        e1.record(st)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / a.steps, time.perf_counter() - t0

    ms, wall = timed(step)
    graph_ms, graph_check = None, None
    if a.graph:
        # the whole step (every launch of forward and backward) captured once
        # and replayed; the library issues no allocation, copy or
        # synchronisation inside a step, so capture records its kernels only
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        torch.cuda.synchronize()
        for _ in range(a.warmup):
            graph.replay()
        graph_ms, _ = timed(graph.replay)
        # a replay writes exactly what an eager step writes
        graph.replay()
        torch.cuda.synchronize()
        og = [t.clone() for t in outputs]
        gg = [{n: t.clone() for n, t in g.items()} for g in grads]
        step()
        torch.cuda.synchronize()
        same = all(torch.equal(a, b) for a, b in zip(og, outputs)) and \
            all(torch.equal(g0[n], g1[n]) for g0, g1 in zip(gg, grads) for n in g0)
        graph_check = "replay bit-identical to an eager step" if same else "MISMATCH"
        if not same:
            print(json.dumps({"error": "graph replay differs from the eager step"}))
            return 1

    # per-launch durations: the library brackets each launch with events on this stream
    lib.dm_trace_enable(True)
    for _ in range(a.steps):
        step()
    torch.cuda.synchronize()
    recs = lib.trace_records()
    lib.dm_trace_enable(False)
    per, order = {}, []
    for lab, sub, t in recs:
        key = (lab, sub)
        if key not in per:
            per[key] = []
            order.append(key)
        per[key].append(t)
    table = []
    for key in order:
        lab, sub = key
        ts = per[key]
        w = work.get(lab) if not sub else None
        avg = sum(ts) / len(ts)
        row = {"kernel": lab + (" " + sub if sub else ""), "op": lab, "us": round(avg * 1e3, 2),
               "launches_per_step": len(ts) / a.steps}
        if w is not None:
            row.update(bound=w.bound, gflop=round(w.flop / 1e9, 4), mbytes=round(w.bytes / 1e6, 3))
            if avg > 0:
                row["tflops"] = round(w.flop / (avg * 1e-3) / 1e12, 1)
                row["gbs"] = round(w.bytes / (avg * 1e-3) / 1e9, 1)
        table.append(row)
    step_us = lambda rows: sum(r["us"] * r["launches_per_step"] for r in rows)
    traced_ms = step_us(table) / 1e3
    # dominant kernel: the single launch with the largest time per step
    dom = max((r for r in table if "bound" in r), key=lambda r: r["us"] * r["launches_per_step"])
    dw = work[dom["op"]]
    dom_s = dom["us"] * 1e-6
    if dw.bound == "mfma":
        achieved = dw.flop / dom_s / 1e12
        peak = dataflow.MFMA_PEAK_TFLOPS[wl.dtype]
        unit = "TFLOP/s"
    else:
        achieved = dw.bytes / dom_s / 1e9
        peak = dataflow.HBM_PEAK_GBS
        unit = "GB/s"
    copy_gbs = copy_rate_gbs(torch, dev)
    roof = {"bound": dw.bound, "kernel": dom["kernel"], "achieved": round(achieved, 1), "peak": peak,
            "unit": unit, "frac": round(achieved / peak, 4), "traffic": traffic_for(dom["kernel"]),
            "per_launch_us": dom["us"], "copy_GBs": round(copy_gbs, 1),
            "frac_of_copy": round(achieved / copy_gbs, 4) if unit == "GB/s" else None,
            "algorithmic_per_launch": dw.flop if dw.bound == "mfma" else dw.bytes}
    # operator classes; second launches (reduce / finish) count with their operator
    is_fused = lambda r: work.get(r["op"]) is not None and work[r["op"]].cls == "fused"
    is_contr = lambda r: work.get(r["op"]) is not None and work[r["op"]].cls == "contraction"
    fused = [r for r in table if is_fused(r)]
    fb = sum(work[r["op"]].bytes * r["launches_per_step"] for r in fused if r["op"] == r["kernel"])
    ft = step_us(fused) * 1e-6
    fused_summary = {"GB/s": round(fb / ft / 1e9, 1), "frac_of_peak": round(fb / ft / 1e9 / dataflow.HBM_PEAK_GBS, 4),
                     "us_per_step": round(ft * 1e6, 1), "mbytes_per_step": round(fb / 1e6, 2)}
    contraction = [r for r in table if is_contr(r)]
    cf = sum(work[r["op"]].flop * r["launches_per_step"] for r in contraction if r["op"] == r["kernel"])
    ct = step_us(contraction) * 1e-6
    mf = [r for r in contraction if work[r["op"]].bound == "mfma"]
    mff = sum(work[r["op"]].flop * r["launches_per_step"] for r in mf if r["op"] == r["kernel"])
    mft = step_us(mf) * 1e-6

    out = {
        "metric": METRIC, "value": round(ms, 4), "unit": "ms", "n_gpus": 1, "steps": a.steps,
        "warmup": a.warmup, "ms_per_step": round(ms, 4), "higher_is_better": False, "scaling": "weak",
        "vs_baseline": None, "dtype": wl.dtype, "data": "synthetic (seeded N(0,1) inputs, N(0,0.02) weights)",
        "config": {"workload": describe(wl), "global_batch": s.B, "seq_len": s.J, "layers": wl.n_layers,
                   "parallelism": "single GPU", "plan": plan_name},
        "roofline": roof,
        "fused_hbm": fused_summary,
        "contractions": {"tflops_all": round(cf / ct / 1e12, 1), "us_per_step": round(ct * 1e6, 1),
                         "mfma_bound_tflops": round(mff / mft / 1e12, 1),
                         "mfma_bound_frac": round(mff / mft / 1e12 / dataflow.MFMA_PEAK_TFLOPS[wl.dtype], 4)},
        "graph_ms_per_step": round(graph_ms, 4) if graph_ms is not None else None,
        "graph_check": graph_check,
        "traced_ms_per_step": round(traced_ms, 4),
        "wall_s": round(wall, 3),
        "paper_context": PAPER_CONTEXT,
    }
    if wl.kind == "encoder":
        # the fused step's algorithmic elements against the same layer's
        # operators one by one (every input read, every output and stored
        # dropout mask written), per layer
        ops = {r["op"] for r in table}
        path = ("keys" if "B13-17 score_bwd_keys" in ops else
                "scores_next" if "F2-4 qkt_softmax_gamma" in ops else
                "scores" if "F2-3 qkt_softmax" in ops else "separate")
        out["data_movement"] = dict(dataflow.data_movement(s, wl.dtype, path,
                                                           epilogue={k for k in dataflow.EPILOGUE if k in ops},
                                                           folded="B20 qkv_bias_grad" not in ops),
                                    per="layer fwd+bwd", paper="22.91% (V100; see paper_context)")
    if a.kernels_json:
        # the launch records of one step in issue order (a label recurs where
        # an operator launches the same kernel pair twice)
        per_step = len(recs) // a.steps
        sequence = [lab + (" " + sub if sub else "") for lab, sub, _ in recs[:per_step]]
        with open(a.kernels_json, "w") as f:
            json.dump({"workload": wl.name, "ms_per_step": ms, "kernels": table, "sequence": sequence}, f, indent=1)
    if not a.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, a.cpu_sample or s.B)
    print(json.dumps(out))
    return 0


if __name__ == "__main__":
    sys.exit(main())
