"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

* The launch planner (``csrc/cardan_planner.cpp``) is built with g++
  ``-fsanitize=address,undefined`` together with ``tests/host/planner_sweep.cpp``,
  which checks the plan invariants (workspace layout, counter offsets shared
  across batches, ranks and forms, split coverage, the gate/up item mapping
  being a bijection) over the named workload shapes and random shapes of the
  supported domain.
* The C ABI's host code (``csrc/cardan_api.hip`` plus the planner) is built
  with the sanitizers on its host side only, with the kernel launchers
  replaced by ``tests/host/kernel_stubs.cpp``, and ``tests/test_abi_cpu.py``
  runs against that library in a child process with the sanitizer runtime
  preloaded.
"""

import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_21137_amd", "csrc")
HOST = os.path.join(ROOT, "tests", "host")
ROCM = "/opt/rocm"
HIPCC = os.path.join(ROCM, "bin", "hipcc")
CLANGXX = os.path.join(ROCM, "lib", "llvm", "bin", "clang++")


def _run(cmd, **kw):
    res = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert res.returncode == 0, f"{' '.join(cmd)}\n{res.stdout[-4000:]}\n{res.stderr[-4000:]}"
    return res


def test_planner_sweep_under_sanitizers(tmp_path):
    exe = str(tmp_path / "planner_sweep")
    _run(["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
          "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"),
          os.path.join(HOST, "planner_sweep.cpp"), os.path.join(CSRC, "cardan_planner.cpp"), "-o", exe])
    res = _run([exe, "150"], env={**os.environ, "ASAN_OPTIONS": "detect_leaks=1"})
    assert " 0 failures" in res.stdout, res.stdout


def _asan_runtime():
    hits = sorted(glob.glob(os.path.join(ROCM, "lib", "llvm", "lib", "clang", "*", "lib", "linux",
                                         "libclang_rt.asan-x86_64.so")))
    return hits[-1] if hits else None


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
def test_abi_validation_under_sanitizers(tmp_path):
    rt = _asan_runtime()
    if rt is None:
        pytest.skip("clang AddressSanitizer runtime not found")
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
    inc = ["-I", os.path.join(ROOT, "include")]
    api = str(tmp_path / "api.o")
    _run([HIPCC, "-O1", "-g", "-std=c++17", "-fPIC", "--offload-arch=gfx950", *san, *inc, "-c",
          os.path.join(CSRC, "cardan_api.hip"), "-o", api])
    host = ["-x", "c++", "-O1", "-g", "-std=c++17", "-fPIC", "-fsanitize=address,undefined",
            "-fno-sanitize-recover=all", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROCM, "include"), *inc]
    objs = [api]
    for src in (os.path.join(CSRC, "cardan_planner.cpp"), os.path.join(HOST, "kernel_stubs.cpp")):
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        _run([CLANGXX, *host, "-c", src, "-o", obj])
        objs.append(obj)
    lib = str(tmp_path / "libcardan_asan.so")
    _run([HIPCC, "-shared", "-fPIC", "--offload-arch=gfx950", "-Xarch_host", "-fsanitize=address",
          "-Xarch_host", "-fsanitize=undefined", "-shared-libsan", *objs, "-o", lib])
    env = {**os.environ, "CARDAN_LIB": lib, "LD_PRELOAD": rt,
           "ASAN_OPTIONS": "detect_leaks=0:halt_on_error=1", "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}
    res = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                          os.path.join(ROOT, "tests", "test_abi_cpu.py")],
                         capture_output=True, text=True, env=env, cwd=ROOT)
    out = res.stdout + res.stderr
    assert res.returncode == 0, out[-6000:]
    assert " passed" in res.stdout and " failed" not in res.stdout and " skipped" not in res.stdout, out[-3000:]
    assert "ERROR: AddressSanitizer" not in out and "runtime error:" not in out, out[-6000:]
