"""AddressSanitizer and UndefinedBehaviorSanitizer over the host runtime.

The runtime (runtime.cpp, prof.cpp) is compiled again with both sanitizers
on its host code only (hipcc, each -fsanitize= after -Xarch_host), linked
with the kernel objects of the normal build and a C++ driver
(host_sanitize_driver.cpp) that exercises every host-only path of the C ABI:
network validation, the partitioner, the planner in every mode and lane
count, bindings and their alignment checks, the per-task state machine and
schedule traces.  No call of the driver enqueues device work, so it runs
without a GPU.  Needs the in-tree build (its kernel objects) and hipcc."""
import glob
import os
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2004_09910_amd")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CLANG = "/opt/rocm/llvm/bin/clang++"
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer"]


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout[-3000:]}\n{r.stderr[-3000:]}"
    return r


def test_host_runtime_under_asan_and_ubsan():
    kernels = sorted(glob.glob(os.path.join(PKG, "_build", "*.hip.o")))
    if not (os.path.exists(HIPCC) and os.path.exists(CLANG) and kernels):
        pytest.skip("needs hipcc, clang++ and the in-tree build's kernel objects")
    inc = ["-I" + os.path.join(ROOT, "include"), "-I" + os.path.join(PKG, "csrc")]
    with tempfile.TemporaryDirectory() as tmp:
        objs = []
        for src in ("runtime.cpp", "prof.cpp"):
            o = os.path.join(tmp, src + ".o")
            _run([HIPCC, "-x", "hip", "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
                  "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"] + SAN + inc +
                 ["-c", os.path.join(PKG, "csrc", src), "-o", o])
            objs.append(o)
        drv = os.path.join(tmp, "driver.o")
        _run([CLANG, "-O1", "-g", "-std=c++17", "-fsanitize=address,undefined",
              "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer"] + inc +
             ["-c", os.path.join(ROOT, "tests", "host_sanitize_driver.cpp"), "-o", drv])
        exe = os.path.join(tmp, "driver")
        _run([CLANG, "-fsanitize=address,undefined", drv] + objs + kernels +
             ["-L/opt/rocm/lib", "-lamdhip64", "-lrocprofiler-sdk-roctx",
              "-Wl,-rpath,/opt/rocm/lib", "-o", exe])
        env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
                   UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
        r = _run([exe], env=env, timeout=300)
        assert "host driver: ok" in r.stdout
