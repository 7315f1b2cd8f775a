"""The host side of the C ABI under AddressSanitizer and UndefinedBehaviorSanitizer: the
argument checks, size queries and workspace layout of fp_api.cpp are rebuilt with both
sanitizers on the host pass only (no device code is instrumented), linked with the
library's kernel objects, and the ABI tests run against that build in a fresh process with
the sanitizer runtime preloaded.  Any report fails the test."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2502_20766_amd")
OUT = os.path.join(PKG, "_build", "asan")


def _tool(name):
    for cand in (os.path.join("/opt/rocm/bin", name), os.path.join("/opt/rocm/llvm/bin", name)):
        if os.path.exists(cand):
            return cand
    return None


def _asan_runtime():
    clang = _tool("amdclang++") or "/opt/rocm/lib/llvm/bin/clang++"
    r = subprocess.run([clang, "-print-file-name=libclang_rt.asan-x86_64.so"],
                       capture_output=True, text=True)
    path = r.stdout.strip()
    return path if r.returncode == 0 and os.path.isabs(path) and os.path.exists(path) else None


def _build_sanitized():
    from paper_2502_20766_amd import _build
    hipcc = _tool("hipcc")
    objs = [os.path.join(PKG, "_build", os.path.splitext(s)[0] + ".o")
            for s in _build.SOURCES if s.endswith(".hip")]
    if not all(os.path.exists(o) for o in objs):
        _build.build()
    os.makedirs(OUT, exist_ok=True)
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
    api_o = os.path.join(OUT, "fp_api.o")
    lib = os.path.join(OUT, "libflexprefill.so")
    cmds = [[hipcc, "-x", "hip", "-O1", "-g", "-std=c++17", "-fPIC", f"--offload-arch={_build.ARCH}",
             "-Wall", "-Werror", *san, "-c", os.path.join(PKG, "csrc", "fp_api.cpp"), "-o", api_o],
            [hipcc, f"--offload-arch={_build.ARCH}", "-shared", "-fPIC", *san, "-shared-libasan",
             api_o, *objs, "-o", lib]]
    for c in cmds:
        r = subprocess.run(c, capture_output=True, text=True)
        assert r.returncode == 0, r.stdout + r.stderr
    return lib


def test_abi_tests_clean_under_address_sanitizer():
    runtime = _asan_runtime()
    if runtime is None or _tool("hipcc") is None:
        pytest.skip("hipcc or the clang AddressSanitizer runtime is not available")
    lib = _build_sanitized()
    env = dict(os.environ, FLEXPREFILL_LIB=lib, LD_PRELOAD=runtime,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi.py")],
                       capture_output=True, text=True, env=env, cwd=ROOT, timeout=600)
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert " passed" in out
