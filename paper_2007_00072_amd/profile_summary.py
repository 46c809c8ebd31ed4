"""Per-operator summary of a rocprofv3 kernel trace of bench.py.

    rocprofv3 --kernel-trace --stats -f csv -d OUT -o bench -- python bench.py ... --kernels-json K.json
    python -m paper_2007_00072_amd.profile_summary --trace OUT/.../bench_kernel_trace.csv \\
        --stats OUT/.../bench_kernel_stats.csv --kernels K.json --out profiles/NAME.md

The library's dispatches repeat with the same sequence every step, so the
n-th dispatch of a step belongs to the n-th launch that the library's own
event timing recorded (bench's --kernels-json "sequence").  The summary puts
rocprofv3's per-dispatch durations next to the event-timed ones.
"""
from __future__ import annotations

import argparse
import csv
import json
import os
import re


def short_name(sym: str) -> str:
    m = re.search(r"gemm_mfmaI(DF16_|DF16b)Li(\d+)ELi(\d+)ELi(\d)ELi(\d)ELi(\d)ELb(\d)ELb(\d)", sym)
    if m:
        dt = "f16" if m.group(1) == "DF16_" else "bf16"
        mode = lambda b: "k" if b == "1" else "o"
        return f"gemm_mfma<{dt},{m.group(2)}x{m.group(3)},waves {m.group(4)}x{m.group(5)},A:{mode(m.group(7))},B:{mode(m.group(8))}>"
    m = re.search(r"gemm_dmaI(DF16_|DF16b)Li(\d+)ELi(\d+)ELi(\d)ELi(\d)ELb(\d)ELb(\d)", sym)
    if m:
        dt = "f16" if m.group(1) == "DF16_" else "bf16"
        mode = lambda b: "k" if b == "1" else "o"
        return f"gemm_dma<{dt},{m.group(2)}x{m.group(3)},waves {m.group(4)}x{m.group(5)},A:{mode(m.group(6))},B:{mode(m.group(7))}>"
    m = re.search(r"gemm_lean(_pair)?I(DF16_|DF16b)Li(\d+)ELi(\d+)ELi(\d)ELi(\d)ELi(\d+)ELi(\d)ELb(\d)ELb(\d)"
                  r"((?:EL[ib]\d+)*)E", sym)
    if m:
        dt = "f16" if m.group(2) == "DF16_" else "bf16"
        mode = lambda b: "k" if b == "1" else "o"
        # the remaining template arguments: lean (k groups, row sums, k-loop
        # schedule, activation step) or pair (row sums)
        rest = re.findall(r"EL([ib])(\d+)", m.group(11))
        names = ("row sums",) if m.group(1) else ("k groups", "row sums", "schedule", "act")
        extra = "" if m.group(8) == "4" else f",{m.group(8)} stages"
        for (kind, val), nm in zip(rest, names):
            if nm == "k groups" and val != "1":
                extra += f",k groups {val}"
            elif nm == "row sums" and val == "1":
                extra += ",row sums"
            elif nm == "schedule" and val in ("1", "2"):
                extra += ",interleaved" if val == "1" else ",ping-pong"
            elif nm == "act" and val != "0":
                extra += f",act {val}"
        return (f"gemm_lean{m.group(1) or ''}<{dt},{m.group(3)}x{m.group(4)},waves {m.group(5)}x{m.group(6)},"
                f"bk {m.group(7)},A:{mode(m.group(9))},B:{mode(m.group(10))}{extra}>")
    m = re.search(r"gemm_(x32|big)I(DF16_|DF16b)", sym)
    if m:
        return f"gemm_{m.group(1)}<{'f16' if m.group(2) == 'DF16_' else 'bf16'}>"
    m = re.search(r"attn_fused_kI(DF16_|DF16b)Li(\d+)ELi(\d)ELi(\d)ELb(\d)(?:ELi(\d))?", sym)
    if m:
        dt = "f16" if m.group(1) == "DF16_" else "bf16"
        nxt = f",next {32 * int(m.group(6))}" if m.group(6) and m.group(6) != "0" else ""
        return f"attn_fused_k<{dt},{'bwd' if m.group(5) == '1' else 'fwd'},D {16 * int(m.group(4))}{nxt}>"
    m = re.search(r"_ZN2dm12_GLOBAL__N_1\d+(\w+?)I", sym)
    if m:
        return m.group(1)
    m = re.search(r"dm::\(anonymous namespace\)::(\w+)", sym)
    return m.group(1) if m else sym[:60]


def main() -> None:
    ap = argparse.ArgumentParser()
    ap.add_argument("--trace", required=True)
    ap.add_argument("--stats", default=None)
    ap.add_argument("--kernels", required=True)
    ap.add_argument("--out", required=True)
    ap.add_argument("--command", default="")
    a = ap.parse_args()

    seq_info = json.load(open(a.kernels))
    seq = seq_info.get("sequence") or [r["kernel"] for r in seq_info["kernels"]]
    ev = {r["kernel"]: r["us"] for r in seq_info["kernels"]}
    rows = list(csv.DictReader(open(a.trace)))
    lib = [r for r in rows if "dm::" in r["Kernel_Name"] or "_ZN2dm" in r["Kernel_Name"]]
    # host submission order: the backward issues some launches on a second
    # stream, so start times may interleave differently from step to step
    key = "Correlation_Id" if lib and "Correlation_Id" in lib[0] else "Dispatch_Id"
    lib.sort(key=lambda r: int(r[key]))
    streams = {(r.get("Queue_Id"), r.get("Stream_Id")) for r in lib}
    n = len(seq)
    if len(lib) % n:
        raise SystemExit(f"{len(lib)} library dispatches are not a whole number of {n}-launch steps")
    steps = len(lib) // n
    lines = [f"# rocprofv3 kernel trace: {seq_info['workload']}", ""]
    if a.command:
        lines += ["Command:", "", "```", a.command, "```", ""]
    lines += [f"{steps} steps x {n} launches; per-launch averages over all steps.", "",
              "| # | operator launch | kernel | rocprofv3 avg (us) | event avg (us) |",
              "|---|---|---|---|---|"]
    total = 0.0
    for p in range(n):
        ds = [(int(lib[s * n + p]["End_Timestamp"]) - int(lib[s * n + p]["Start_Timestamp"])) / 1e3
              for s in range(steps)]
        names = {lib[s * n + p]["Kernel_Name"] for s in range(steps)}
        if len(names) != 1:
            raise SystemExit(f"launch {p} maps to several kernels: {names}")
        avg = sum(ds) / len(ds)
        total += avg
        lines.append(f"| {p} | {seq[p]} | `{short_name(names.pop())}` | {avg:.1f} | {ev[seq[p]]:.1f} |")
    lines += ["", f"Sum of per-launch averages: {total / 1e3:.3f} ms per step "
                  f"(bench event timing of the whole step: {seq_info['ms_per_step']:.3f} ms)."]
    if len(streams) > 1:
        lines += ["Launches ran on more than one stream and overlap, so their sum exceeds the step time."]
    lines += [""]
    if a.stats and os.path.exists(a.stats):
        st = list(csv.DictReader(open(a.stats)))
        st.sort(key=lambda r: -float(r["TotalDurationNs"]))
        lines += ["rocprofv3 --stats (per kernel symbol, all dispatches of the run):", "",
                  "| kernel | calls | avg (us) | % |", "|---|---|---|---|"]
        for r in st[:25]:
            lines.append(f"| `{short_name(r['Name'])}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                         f"{float(r['Percentage']):.2f} |")
    with open(a.out, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


if __name__ == "__main__":
    main()
