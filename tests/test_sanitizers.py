"""AddressSanitizer + UndefinedBehaviorSanitizer builds of the host code (CPU only).

* The oracle, built with gcc -fsanitize=address,undefined (no recovery), runs its own pin
  tests (tests/test_oracle_pins.py): every training mode, merge, forward, cost, gradient and
  trace path of the C code.
* The HIP library, its host code built with clang's -fsanitize=address,undefined (device code
  unoptimised: it is loaded, never launched here), runs the host-side ABI tests
  (tests/test_abi.py): configuration checks, parameter counts, the data split, argument
  validation and the error paths of pnn_init.

Each runs in a child process with the sanitizer runtime preloaded (Python itself is not
instrumented; leak detection is off because the interpreter keeps its allocations to the end)
and must end with status 0, no sanitizer report, and the instrumented library mapped.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

DRIVER = r"""
import sys
sys.path.insert(0, {root!r})
{setup}
import pytest
rc = pytest.main(["-q", "-x", "-p", "no:cacheprovider", {tests!r}])
maps = open("/proc/self/maps").read()
assert {lib!r} in maps, "the instrumented library was not loaded"
sys.exit(rc)
"""


def _run(tmp_path, setup, tests, lib, preload):
    drv = tmp_path / "driver.py"
    drv.write_text(DRIVER.format(root=ROOT, setup=setup, tests=tests, lib=lib))
    env = dict(os.environ, LD_PRELOAD=preload, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([sys.executable, str(drv)], cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out and "runtime error:" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert " passed" in out, out[-2000:]


def _gcc_runtime(name):
    p = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return p if os.path.isabs(p) and os.path.exists(p) else None


@pytest.mark.skipif(shutil.which("gcc") is None or _gcc_runtime("libasan.so") is None, reason="gcc's ASan runtime")
def test_oracle_under_asan_ubsan(tmp_path):
    lib = str(tmp_path / "liboracle_asan.so")
    subprocess.check_call(["gcc", "-O1", "-g", "-fno-omit-frame-pointer", "-std=c11", "-fPIC", "-shared",
                           "-ffp-contract=off", "-fno-fast-math", "-Wall",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                           "-o", lib, os.path.join(ROOT, "oracle", "pnn_oracle.c"), "-lm", "-lpthread"])
    setup = f"from oracle import oracle as O\nO._LIB_PATH = {lib!r}"
    _run(tmp_path, setup, os.path.join(ROOT, "tests", "test_oracle_pins.py"), lib, _gcc_runtime("libasan.so"))


def _clang_asan_runtime():
    base = "/opt/rocm/lib/llvm/lib/clang"
    if not os.path.isdir(base):
        return None
    for v in sorted(os.listdir(base), reverse=True):
        p = os.path.join(base, v, "lib", "linux", "libclang_rt.asan-x86_64.so")
        if os.path.exists(p):
            return p
    return None


@pytest.mark.skipif(not os.path.exists(HIPCC) or _clang_asan_runtime() is None, reason="hipcc and clang's ASan runtime")
def test_host_library_under_asan_ubsan(tmp_path):
    lib = str(tmp_path / "libpnn_asan.so")
    subprocess.check_call([HIPCC, "--offload-arch=gfx950", "-O1", "-Xarch_device", "-O0", "-std=c++17", "-fPIC", "-shared",
                           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-Xarch_host", "-fno-sanitize-recover=all",
                           "-Xarch_host", "-fno-omit-frame-pointer",
                           "-o", lib, os.path.join(ROOT, "paper_2304_09590_amd", "csrc", "pnn.hip")],
                          stdout=subprocess.DEVNULL, stderr=subprocess.DEVNULL)
    setup = f"from paper_2304_09590_amd import pnn\npnn.LIB_PATH = {lib!r}"
    _run(tmp_path, setup, os.path.join(ROOT, "tests", "test_abi.py"), lib, _clang_asan_runtime())
