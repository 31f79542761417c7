"""The library's host code under AddressSanitizer and
UndefinedBehaviorSanitizer, on the CPU: tests/asan/abi_host_driver.c calls
every workspace query over a grid of extents (up to INT64_MAX, so every
overflow guard is exercised) and every entry point with arguments that must
be rejected before any HIP call.  The HIP sources are built with the
sanitizers on the host side only (no GPU code is instrumented and nothing is
launched)."""
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

from conftest import ROOT

CSRC = os.path.join(ROOT, "paper_2402_09900_amd", "csrc")
INC = os.path.join(ROOT, "include")
CLANG = "/opt/rocm/llvm/bin/clang"
SAN_HOST = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-omit-frame-pointer"]


def _have_toolchain():
    return os.path.exists(CLANG) and subprocess.run(["which", "hipcc"], capture_output=True).returncode == 0


@pytest.mark.skipif(not _have_toolchain(), reason="hipcc / ROCm clang not installed")
def test_host_code_is_clean_under_asan_and_ubsan(tmp_path):
    srcs = sorted(f for f in os.listdir(CSRC) if f.endswith(".hip"))

    def compile_one(f):
        cmd = ["hipcc", "-c", "-O1", "-g", "-std=c++17", "--offload-arch=gfx950",
               "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"] + SAN_HOST + \
              ["-I", INC, os.path.join(CSRC, f), "-o", str(tmp_path / (f + ".o"))]
        return subprocess.run(cmd, capture_output=True, text=True)

    with ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        for res in ex.map(compile_one, srcs):
            assert res.returncode == 0, res.stderr[-2000:]
    drv_o = str(tmp_path / "driver.o")
    subprocess.run([CLANG, "-O1", "-g", "-fsanitize=address,undefined", "-fno-omit-frame-pointer", "-I", INC,
                    "-c", os.path.join(ROOT, "tests", "asan", "abi_host_driver.c"), "-o", drv_o], check=True)
    exe = str(tmp_path / "driver")
    subprocess.run([CLANG + "++", "--hip-link", "--offload-arch=gfx950", "-fsanitize=address,undefined", "-o", exe,
                    drv_o] + [str(tmp_path / (f + ".o")) for f in srcs] +
                   ["-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib"], check=True)
    env = dict(os.environ, UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", ASAN_OPTIONS="detect_leaks=1")
    res = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    assert res.returncode == 0, res.stdout + res.stderr[-3000:]
    assert "runtime error" not in res.stderr and "AddressSanitizer" not in res.stderr, res.stderr[-3000:]
    assert "validation done" in res.stdout
