"""HBM traffic of every launch of the encoder layer from rocprofv3 counters.

Two passes over the same program, one counter each (FETCH_SIZE, then
WRITE_SIZE, KiB per dispatch), each followed by a plain device-to-device
copy of known size that calibrates the counter:

    rocprofv3 --pmc FETCH_SIZE -f csv -d OUT/fetch -o run -- python3 paper_2007_00072_amd/traffic.py run \\
        --kernels-json OUT/seq.json
    rocprofv3 --pmc WRITE_SIZE -f csv -d OUT/write -o run -- python3 paper_2007_00072_amd/traffic.py run
    python3 paper_2007_00072_amd/traffic.py summarize --fetch OUT/fetch/.../run_counter_collection.csv \\
        --write OUT/write/.../run_counter_collection.csv --kernels OUT/seq.json --out profiles/traffic

`run` executes warm-up steps, one step whose launches the library labels
(the dispatch order is the same in every step), then the copy.  `summarize`
maps the last step's library dispatches to the launch labels, scales each
counter by (copy bytes / counter reading of the copy), and writes
`<out>.json` (bytes per launch, with the hash of the kernel sources it was
taken on) and `<out>.md`.
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
COPY_BYTES = 512 << 20


def csrc_hash() -> str:
    h = hashlib.sha256()
    d = os.path.join(ROOT, "paper_2007_00072_amd", "csrc")
    # kernel and host sources only: build leftovers in the folder change nothing
    for f in sorted(x for x in os.listdir(d) if x.endswith((".hip", ".hpp", ".h"))):
        h.update(f.encode())
        h.update(open(os.path.join(d, f), "rb").read())
    return h.hexdigest()[:16]


def run(a) -> None:
    sys.path.insert(0, ROOT)
    import torch
    from paper_2007_00072_amd import lib
    from paper_2007_00072_amd.inputs import WORKLOADS, make_activation, make_params
    from paper_2007_00072_amd.runner import EncoderLayer, desc_for

    wl = WORKLOADS[a.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    layer = EncoderLayer(desc_for(wl), make_params(wl), dev)
    x = make_activation(wl, 0).to(dev)
    dy = make_activation(wl, 1).to(dev)
    y, dx = torch.empty_like(x), torch.empty_like(x)
    src = torch.ones(COPY_BYTES // 2, dtype=torch.float16, device=dev)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(a.warmup):
        layer.forward(x, y)
        layer.backward(x, dy, dx)
    torch.cuda.synchronize()
    lib.dm_trace_enable(True)
    layer.forward(x, y)
    layer.backward(x, dy, dx)
    torch.cuda.synchronize()
    seq = [lab + (" " + sub if sub else "") for lab, sub, _ in lib.trace_records()]
    lib.dm_trace_enable(False)
    dst.copy_(src)
    torch.cuda.synchronize()
    print(f"traffic run: {a.workload}, {a.warmup + 1} steps of {len(seq)} launches, then a {COPY_BYTES} B copy",
          flush=True)
    if a.kernels_json:
        with open(a.kernels_json, "w") as f:
            json.dump({"workload": wl.name, "sequence": seq, "copy_bytes": COPY_BYTES}, f, indent=1)


def _read(path):
    rows = list(csv.DictReader(open(path)))
    out = []
    for r in rows:
        out.append((int(r["Dispatch_Id"]), r["Kernel_Name"], float(r["Counter_Value"])))
    out.sort()
    return out


def _per_launch(rows, seq):
    lib = [r for r in rows if "dm::" in r[1] or "_ZN2dm" in r[1]]
    n = len(seq)
    if len(lib) % n:
        raise SystemExit(f"{len(lib)} library dispatches are not a whole number of {n}-launch steps")
    last = lib[-n:]
    copy = [r for r in rows if r[0] > last[-1][0]]
    if not copy:
        raise SystemExit("no copy dispatch after the last step")
    return [r[2] for r in last], copy[-1][2]


def summarize(a) -> None:
    sys.path.insert(0, ROOT)
    from paper_2007_00072_amd import dataflow
    from paper_2007_00072_amd.inputs import WORKLOADS

    info = json.load(open(a.kernels))
    seq, copy_bytes = info["sequence"], info["copy_bytes"]
    fetch, fcopy = _per_launch(_read(a.fetch), seq)
    write, wcopy = _per_launch(_read(a.write), seq)
    kf, kw = copy_bytes / (fcopy * 1024.0), copy_bytes / (wcopy * 1024.0)
    wl = WORKLOADS[info["workload"]]
    work = dataflow.encoder_layer(wl.shape, wl.dtype)
    kern = {}
    lines = [f"# HBM traffic per launch: {wl.name}", ""]
    if a.command:
        lines += ["Commands:", "", "```", a.command, "```", ""]
    lines += [f"Calibration: a {copy_bytes} B device copy reads {fcopy:.0f} KiB (FETCH_SIZE) and writes "
              f"{wcopy:.0f} KiB (WRITE_SIZE); factors {kf:.4f} (fetch) and {kw:.4f} (write) turn counter KiB "
              f"into bytes.", "",
              "| launch | fetch MB | write MB | traffic MB | algorithmic MB | traffic / algorithmic |",
              "|---|---|---|---|---|---|"]
    tot_t = tot_a = 0.0
    for lab, f, w in zip(seq, fetch, write):
        fb, wb = f * 1024.0 * kf, w * 1024.0 * kw
        alg = work[lab].bytes if lab in work else None
        kern[lab] = {"fetch_bytes": round(fb), "write_bytes": round(wb), "bytes_per_launch": round(fb + wb),
                     "algorithmic_bytes": alg}
        tot_t += fb + wb
        tot_a += alg or 0.0
        ratio = f"{(fb + wb) / alg:.2f}" if alg else "-"
        lines.append(f"| {lab} | {fb / 1e6:.2f} | {wb / 1e6:.2f} | {(fb + wb) / 1e6:.2f} | "
                     f"{(alg or 0) / 1e6:.2f} | {ratio} |")
    lines += ["", f"Step total: {tot_t / 1e6:.1f} MB measured, {tot_a / 1e6:.1f} MB algorithmic.", ""]
    with open(a.out + ".json", "w") as f:
        json.dump({"workload": wl.name, "csrc_sha": csrc_hash(), "calibration": {"fetch": kf, "write": kw},
                   "kernels": kern}, f, indent=1)
    with open(a.out + ".md", "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def main() -> None:
    ap = argparse.ArgumentParser()
    sp = ap.add_subparsers(dest="cmd", required=True)
    r = sp.add_parser("run")
    r.add_argument("--workload", default="bert_large_f16")
    r.add_argument("--warmup", type=int, default=2)
    r.add_argument("--kernels-json", default=None)
    s = sp.add_parser("summarize")
    s.add_argument("--fetch", required=True)
    s.add_argument("--write", required=True)
    s.add_argument("--kernels", required=True)
    s.add_argument("--out", required=True)
    s.add_argument("--command", default="")
    a = ap.parse_args()
    run(a) if a.cmd == "run" else summarize(a)


if __name__ == "__main__":
    main()
