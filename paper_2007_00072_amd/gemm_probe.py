"""Contraction kernel sweep on one GPU: where a contraction's time goes.

    python -m paper_2007_00072_amd.gemm_probe --out profiles/contraction_sweep_f16.md

For output shapes of the encoder layer's contractions (4096 tokens at
BERT-large width: 4096 x 4096, the fused Q/K/V projection's 4096 x 3072
and 4096 x 1024), times the library's lean kernels (`contract` with a
fixed tile configuration) as the contraction length K grows, so the cost
per k-step (the slope) separates from the fixed cost of launch, prologue
and output stores (the intercept), next to torch.matmul on the same
operands (the vendor BLAS of this PyTorch build, for reference only) and
to a plain fill of the output (its store cost alone).  Also times a plain
device copy of 1 GiB (the practical HBM ceiling).  Event timing on the
current stream, operands resident on the GPU, fp16 storage, fp32
accumulation.
"""
from __future__ import annotations

import argparse
import json
import sys

import torch

from . import lib

PEAK_TFLOPS = 2516.6   # dense fp16 MFMA


def _time(fn, iters=30, warm=5):
    for _ in range(warm):
        fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(iters):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / iters * 1e3


def _slope(ks, us):
    n = len(ks)
    mk, mu = sum(ks) / n, sum(us) / n
    b = sum((k - mk) * (u - mu) for k, u in zip(ks, us)) / sum((k - mk) ** 2 for k in ks)
    return b, mu - b * mk


def sweep(dev):
    rows = []
    ks = (512, 1024, 2048, 4096)
    for M, N, cfgs in ((4096, 4096, (13, 20, 23, 24)), (4096, 3072, (23, 25)), (4096, 1024, (15, 18, 22))):
        C = torch.empty((M, N), device=dev, dtype=torch.float16)
        fill = _time(lambda: C.fill_(1.0))
        res = {"M": M, "N": N, "fill_us": fill, "cfg": {}}
        blas = []
        per = {c: [] for c in cfgs}
        for K in ks:
            A = torch.randn((M, K), device=dev).half()
            B = torch.randn((N, K), device=dev).half()
            blas.append(_time(lambda: torch.matmul(A, B.t(), out=C)))
            for c in cfgs:
                per[c].append(_time(lambda: lib.contract(lib.DM_F16, 1, M, N, K, 1.0, A, 0, M * K, B, 1, N * K, None,
                                                         C, 0, M * N, c, 1, None, 0)))
            del A, B
        res["ks"] = list(ks)
        res["blas_us"] = blas
        for c in cfgs:
            res["cfg"][c] = per[c]
        rows.append(res)
    src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    copy_us = _time(lambda: dst.copy_(src), iters=10)
    return rows, 2.0 * (1 << 30) / copy_us / 1e3


def write(rows, copy_gbs, path, command):
    out = ["# Contraction sweep: fixed cost and cost per k-step (fp16)", "", "Command:", "", "```", command, "```", "",
           "Lean kernels of the library (`contract`, fixed tile configuration, unsplit) against the contraction "
           "length K at fixed output M x N; slope and intercept of a least-squares line through the four K.  "
           "`torch.matmul` (this PyTorch build's BLAS) on the same operands for reference.  `fill` is a plain "
           "fill of the output tensor.", "",
           f"Plain 1 GiB device copy: {copy_gbs:.0f} GB/s (bytes read + written).", ""]
    names = {13: "256x256, 8 waves", 20: "256x256, 4 waves, interleaved", 23: "256x256, 8 waves, ping-pong",
             24: "256x256, 8 waves, ping-pong, 5 stages", 25: "256x192, 8 waves, ping-pong",
             15: "128x128, 8 waves", 18: "128x128, 4 waves",
             22: "128x128, 4 waves, interleaved"}
    for r in rows:
        M, N, ks = r["M"], r["N"], r["ks"]
        out += [f"## M = {M}, N = {N} (output fill {r['fill_us']:.1f} us)", "",
                "| kernel | " + " | ".join(f"K={k} (us)" for k in ks) + " | us per 1024 of K | TFLOP/s per k-step "
                "| fixed (us) |", "|---|" + "---|" * (len(ks) + 3)]
        series = [(f"cfg {c} ({names.get(c, '')})", v) for c, v in r["cfg"].items()] + [("torch.matmul", r["blas_us"])]
        for name, us in series:
            b, a = _slope(ks, us)
            tf = 2.0 * M * N / (b * 1e-6) / 1e12
            out.append(f"| {name} | " + " | ".join(f"{u:.1f}" for u in us) +
                       f" | {b * 1024:.1f} | {tf:.0f} ({tf / PEAK_TFLOPS:.2f} of peak) | {a:.1f} |")
        out.append("")
    with open(path, "w") as f:
        f.write("\n".join(out))


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", default=None, help="markdown summary to write")
    ap.add_argument("--json", default=None)
    a = ap.parse_args()
    if not torch.cuda.is_available():
        print("needs a GPU", file=sys.stderr)
        return 1
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    rows, copy_gbs = sweep(dev)
    print(json.dumps({"rows": rows, "copy_GBs": copy_gbs}))
    if a.json:
        with open(a.json, "w") as f:
            json.dump({"rows": rows, "copy_GBs": copy_gbs}, f, indent=1)
    if a.out:
        write(rows, copy_gbs, a.out, "python3 -m paper_2007_00072_amd.gemm_probe --out profiles/contraction_sweep_f16.md")
    return 0


if __name__ == "__main__":
    sys.exit(main())
