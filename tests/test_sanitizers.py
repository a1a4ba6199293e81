"""CPU sanitizer runs (AddressSanitizer + UndefinedBehaviorSanitizer); no GPU.

* The library's host-only code (argument validation, the split-KV planner
  and the plan-table packing, ``csrc/host_plan.cpp``) is built with
  ``g++ -fsanitize=address,undefined`` together with a checker
  (``tests/sanitize/host_plan_check.cpp``) that runs it over random,
  malformed and extreme batches and checks the plan's invariants (unit
  counts, packed plan-table fields, the XCD swizzle, the makespan model
  against brute-force dealing).
* The library (host code instrumented, the gfx950 device code as always)
  and the oracle are built against ROCm clang's shared sanitizer runtime,
  and the C-ABI tests and every oracle pin run in one process with that
  runtime preloaded; a planted heap overflow in a throwaway library shows
  that the runtime is live.
"""
import glob
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2501_12162_amd", "csrc")
INCLUDE = os.path.join(ROOT, "include")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]


def _runtime():
    rt = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return rt[-1] if rt else None


def test_host_plan_code_under_asan_ubsan(tmp_path):
    if shutil.which("g++") is None:
        pytest.skip("g++ not available")
    exe = str(tmp_path / "host_plan_check")
    subprocess.run(["g++", "-std=c++17", *SAN, "-I", INCLUDE, "-I", CSRC, os.path.join(CSRC, "host_plan.cpp"),
                    os.path.join(ROOT, "tests", "sanitize", "host_plan_check.cpp"), "-o", exe], check=True)
    r = subprocess.run([exe], capture_output=True, text=True, env=dict(os.environ, ASAN_OPTIONS="abort_on_error=1"))
    assert r.returncode == 0, r.stdout + r.stderr
    assert "host plan checks passed" in r.stdout


@pytest.fixture(scope="module")
def instrumented(tmp_path_factory):
    rt = _runtime()
    clang = "/opt/rocm/llvm/bin/clang"
    if rt is None or not os.path.exists(clang):
        pytest.skip("ROCm clang sanitizer runtime not available")
    from paper_2501_12162_amd.build import hipcc, sources
    d = tmp_path_factory.mktemp("sanitized")
    lib = str(d / "libadaserve.so")
    # host code instrumented; each sanitizer flag applies to the host pass only
    # (the device code keeps the library's own -O3: its inline asm needs it)
    host = []
    for f in SAN[:-1] + ["-shared-libsan"]:
        host += ["-Xarch_host", f]
    subprocess.run([hipcc(), "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
                    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", *host,
                    "-I", INCLUDE, "-I", CSRC, *sources(), "-o", lib], check=True, capture_output=True)
    orc = str(d / "liboracle.so")
    subprocess.run([clang, "-std=c11", "-fPIC", "-shared", "-fopenmp", *SAN, "-shared-libsan",
                    os.path.join(ROOT, "oracle", "oracle.c"), "-o", orc, "-lm",
                    "-Wl,-rpath,/opt/rocm/llvm/lib"], check=True)
    bad_c = d / "bad.c"
    bad_c.write_text("#include <stdlib.h>\nint poke(int n) { int *a = malloc(4 * n); int s = a[n]; "
                     "free(a); return s; }\n")
    bad = str(d / "libbad.so")
    subprocess.run([clang, "-fPIC", "-shared", *SAN, "-shared-libsan", str(bad_c), "-o", bad], check=True)
    env = dict(os.environ, LD_PRELOAD=rt, ADASERVE_LIBRARY=lib, ADASERVE_ORACLE_LIB=orc,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    return env, bad


def test_sanitizer_runtime_is_live(instrumented):
    env, bad = instrumented
    r = subprocess.run([sys.executable, "-c", "import ctypes; ctypes.CDLL(%r).poke(4)" % bad],
                       capture_output=True, text=True, env=env)
    assert r.returncode != 0 and "heap-buffer-overflow" in r.stderr


def test_abi_and_oracle_pins_under_asan_ubsan(instrumented):
    env, _ = instrumented
    probe = ("import oracle, paper_2501_12162_amd as ada; oracle._load(); ada.load_library(); "
             "print(open('/proc/self/maps').read())")
    maps = subprocess.run([sys.executable, "-c", probe], capture_output=True, text=True, env=env, cwd=ROOT)
    assert maps.returncode == 0, maps.stderr
    for path in (env["ADASERVE_LIBRARY"], env["ADASERVE_ORACLE_LIB"], env["LD_PRELOAD"]):
        assert os.path.realpath(path) in maps.stdout or path in maps.stdout, path
    tests = ["tests/test_abi.py"] + sorted(os.path.relpath(p, ROOT) for p in
                                           glob.glob(os.path.join(ROOT, "tests", "test_oracle_*.py")))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", *tests],
                       capture_output=True, text=True, env=env, cwd=ROOT)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert " passed" in r.stdout
