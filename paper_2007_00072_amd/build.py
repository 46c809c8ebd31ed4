"""Builds libdmtx.so (the HIP kernels and the C ABI) for gfx950, in-tree.

    python -m paper_2007_00072_amd.build [--jobs N]

Each .hip source is compiled separately with hipcc and the objects are
linked into paper_2007_00072_amd/libdmtx.so, which exports exactly the C
functions that include/dmtx.h declares (a linker version script keeps
everything else local).
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import os
import re
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libdmtx.so")
SOURCES = ["gemm.hip", "fused.hip", "attn.hip", "abi.hip", "layer.hip", "noalloc.hip"]
HEADER = os.path.join(ROOT, "include", "dmtx.h")

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
    # packed fp32 instructions stay off (hipcc -O3 would otherwise form them)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I" + os.path.join(ROOT, "include"),
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def _deps_mtime(src: str) -> float:
    """Newest modification time of a source and the headers it may include."""
    paths = [os.path.join(CSRC, src), HEADER] + [os.path.join(CSRC, f) for f in os.listdir(CSRC)
                                                  if f.endswith(".hpp")]
    return max(os.path.getmtime(p) for p in paths)


def _compile(src: str, incremental: bool = False) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    if incremental and os.path.exists(obj) and os.path.getmtime(obj) > _deps_mtime(src):
        return obj
    cmd = [hipcc(), *HIPCC_FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile of {src} failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    errs = [ln for ln in r.stderr.splitlines()
            if "warning" in ln and "packed-fp32-ops" not in ln and "recognized feature" not in ln]
    if errs:
        sys.stderr.write("\n".join(errs) + "\n")
    return obj


def abi_names(header: str = HEADER) -> list:
    """Names of the functions the C header declares (declarations start at
    column 0 with a return type; comments and typedefs are skipped)."""
    text = re.sub(r"/\*.*?\*/", "", open(header).read(), flags=re.S)
    names = []
    for ln in text.splitlines():
        m = re.match(r"^(?:const\s+)?(?:int|int32_t|size_t|void|char)\s*\**\s*(\w+)\s*\(", ln)
        if m:
            names.append(m.group(1))
    return names


def build(jobs: int = 4, verbose: bool = False, incremental: bool = False) -> str:
    """Compiles every source (incremental: only those whose object is older
    than the source or a header) and links the library."""
    os.makedirs(BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(lambda s: _compile(s, incremental), SOURCES))
    tmp = LIB + ".tmp"
    vscript = os.path.join(BUILD, "exports.map")
    with open(vscript, "w") as f:
        f.write("{\n  global:\n" + "".join(f"    {n};\n" for n in abi_names()) + "  local: *;\n};\n")
    cmd = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", "-Wl,--version-script=" + vscript, "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
    return LIB


# Host-side AddressSanitizer + UndefinedBehaviorSanitizer build of the
# same sources, for checking the host code (argument validation, workspace
# carving, plan objects) on a machine without a GPU.  The sanitizers apply
# to host code only; device code is compiled unoptimised (its kernels are
# never launched from this build).  Load it with the sanitizer runtime
# preloaded (hostsan_runtime()) and DMTX_LIB pointing at it.
HOSTSAN_DIR = os.path.join(BUILD, "hostsan")
HOSTSAN_LIB = os.path.join(HOSTSAN_DIR, "libdmtx_hostsan.so")
HOSTSAN_FLAGS = [
    "--offload-arch=gfx950", "-g", "-std=c++17", "-fPIC", "-fno-omit-frame-pointer",
    "-Xarch_host", "-O1", "-Xarch_device", "-O0",
    "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
    "-Xarch_host", "-fno-sanitize-recover=all",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I" + os.path.join(ROOT, "include"),
]


def hostsan_runtime() -> str:
    """Path of clang's shared ASan runtime (which carries UBSan too)."""
    out = subprocess.run([hipcc(), "--offload-host-only", "-print-file-name=libclang_rt.asan-x86_64.so"],
                         capture_output=True, text=True).stdout.strip()
    if out and os.path.isabs(out) and os.path.exists(out):
        return out
    llvm = os.path.join(os.path.dirname(os.path.dirname(os.path.realpath(hipcc()))), "lib", "llvm", "lib", "clang")
    for ver in sorted(os.listdir(llvm)) if os.path.isdir(llvm) else []:
        cand = os.path.join(llvm, ver, "lib", "linux", "libclang_rt.asan-x86_64.so")
        if os.path.exists(cand):
            return cand
    raise RuntimeError("clang's shared ASan runtime not found")


def hostsan_stale() -> bool:
    if not os.path.exists(HOSTSAN_LIB):
        return True
    t = os.path.getmtime(HOSTSAN_LIB)
    return any(_deps_mtime(src) > t for src in SOURCES)


def build_hostsan(jobs: int = 4, verbose: bool = False) -> str:
    """Builds the host-sanitized library (every source, then the link)."""
    os.makedirs(HOSTSAN_DIR, exist_ok=True)

    def one(src):
        obj = os.path.join(HOSTSAN_DIR, os.path.splitext(src)[0] + ".o")
        cmd = [hipcc(), *HOSTSAN_FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"sanitized compile of {src} failed:\n{' '.join(cmd)}\n{r.stderr}")
        return obj

    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(one, SOURCES))
    tmp = HOSTSAN_LIB + ".tmp"
    cmd = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", "-shared-libsan",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"sanitized link failed:\n{' '.join(cmd)}\n{r.stderr}")
    os.replace(tmp, HOSTSAN_LIB)
    if verbose:
        print("built", HOSTSAN_LIB)
    return HOSTSAN_LIB


def main() -> None:
    ap = argparse.ArgumentParser()
    ap.add_argument("--jobs", type=int, default=min(4, os.cpu_count() or 1))
    ap.add_argument("--incremental", action="store_true", help="recompile only sources newer than their objects")
    ap.add_argument("--hostsan", action="store_true", help="also build the host-sanitized library")
    a = ap.parse_args()
    build(a.jobs, verbose=True, incremental=a.incremental)
    if a.hostsan:
        build_hostsan(a.jobs, verbose=True)


if __name__ == "__main__":
    main()
