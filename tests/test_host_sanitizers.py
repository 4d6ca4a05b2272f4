"""The C ABI's host code under AddressSanitizer and UndefinedBehaviorSanitizer.

api.cpp (argument validation, workspace planning, launch set-up) is compiled
with both sanitizers on its host side only and linked with the library's
kernel objects; the ABI host tests then run against that library in a child
process with the sanitizer runtime preloaded. Every entry point they call
returns before any HIP call, so this runs without a GPU. Any sanitizer
report fails the test.
"""
import glob
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2609_40335_amd")
OBJS = [os.path.join(PKG, "_build", f"{n}.o") for n in ("embed", "gemm", "gram", "misc", "vector")]


def _hipcc():
    for c in ("/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    return None


def _asan_runtime():
    found = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return found[-1] if found else None


def test_abi_host_code_is_sanitizer_clean(tmp_path):
    hipcc, rt = _hipcc(), _asan_runtime()
    if hipcc is None or rt is None:
        pytest.skip("needs hipcc and clang's AddressSanitizer runtime")
    if not all(os.path.exists(o) for o in OBJS):
        pytest.skip("kernel objects not built (python -m paper_2609_40335_amd.build)")
    # Sanitizers on the host side only; device code is built as usual.
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-fno-gpu-sanitize"]
    obj = str(tmp_path / "api_san.o")
    lib = str(tmp_path / "libdpghost_san.so")
    cc = [hipcc, "-x", "hip", "--offload-arch=gfx950", "-std=c++17", "-fPIC", "-O1", "-g",
          "-fno-omit-frame-pointer", "-I", os.path.join(ROOT, "include"),
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", *san,
          "-c", os.path.join(PKG, "csrc", "api.cpp"), "-o", obj]
    r = subprocess.run(cc, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    ld = [hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", *san, "-shared-libasan",
          "-o", lib, obj, *OBJS]
    r = subprocess.run(ld, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    logs = tmp_path / "reports"
    logs.mkdir()
    env = dict(os.environ)
    env.update({
        "DPGHOST_LIBRARY": lib,
        "LD_PRELOAD": rt,
        # Python and torch are not instrumented: only this library's own
        # accesses are checked, and leaks at interpreter exit are not ours.
        "ASAN_OPTIONS": f"detect_leaks=0:verify_asan_link_order=0:alloc_dealloc_mismatch=0:"
                        f"log_path={logs}/asan",
        "UBSAN_OPTIONS": f"halt_on_error=1:print_stacktrace=1:log_path={logs}/ubsan",
    })
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi_host.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    reports = sorted(logs.iterdir())
    text = "".join(p.read_text()[:4000] for p in reports)
    assert not reports, text
    assert r.returncode == 0, (r.stdout + r.stderr)[-4000:]
