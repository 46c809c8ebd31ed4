"""The C ABI's host code under AddressSanitizer and UndefinedBehaviorSanitizer.

A second build of the library (host code instrumented, device code never
launched) is loaded into a child interpreter with clang's ASan runtime
preloaded, and the CPU validation tests of test_abi_cpu.py run against it:
every rejected descriptor, null or misaligned pointer, short workspace,
plan object and saved-tensor view goes through the instrumented host code.
Any out-of-bounds access, use after free or undefined behaviour aborts the
child (recovery is off), which fails this test.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def hostsan_lib():
    from paper_2007_00072_amd import build
    try:
        build.hipcc()
    except RuntimeError:
        pytest.skip("hipcc not available")
    if build.hostsan_stale():
        build.build_hostsan(jobs=min(8, os.cpu_count() or 1))
    return build.HOSTSAN_LIB, build.hostsan_runtime()


def test_validation_layer_clean_under_asan_ubsan(hostsan_lib):
    lib_path, runtime = hostsan_lib
    env = dict(os.environ)
    env.update({
        "DMTX_LIB": lib_path,
        "LD_PRELOAD": runtime,
        # the interpreter itself is not instrumented: its allocations at exit
        # are not this library's leaks
        "ASAN_OPTIONS": "detect_leaks=0:halt_on_error=1:abort_on_error=0",
        "UBSAN_OPTIONS": "print_stacktrace=1:halt_on_error=1",
        "PYTHONDONTWRITEBYTECODE": "1",
    })
    # the export-table checks read the product library's symbol table, which
    # the unversioned sanitized build does not reproduce
    cmd = [sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
           os.path.join(ROOT, "tests", "test_abi_cpu.py"), "-k", "not exports"]
    r = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert "ERROR: AddressSanitizer" not in out, out[-4000:]
    assert "runtime error:" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert " passed" in out and " failed" not in out, out[-2000:]


def test_sanitized_build_is_the_one_loaded(hostsan_lib):
    lib_path, runtime = hostsan_lib
    env = dict(os.environ, DMTX_LIB=lib_path, LD_PRELOAD=runtime, ASAN_OPTIONS="detect_leaks=0")
    code = ("from paper_2007_00072_amd import lib as L\n"
            "print(L.LIB_PATH)\n"
            "print([ln.split()[-1] for ln in open('/proc/self/maps') if 'libdmtx' in ln][:1])\n")
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-2000:]
    assert lib_path in r.stdout and "libdmtx_hostsan.so" in r.stdout, r.stdout
