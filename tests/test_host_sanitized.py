"""The host runtime under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

tests/host/runtime_host_check.cpp compiles the runtime source with its kernel
launchers replaced by recorders that check every workspace range a forward
touches (inside the workspace, clear of its guard areas) and the index
invariants the kernels rely on, over the probe's workloads, their variants and
seeded random shapes at several compute-unit counts, plus the config checks on
values that would overflow.  Only host code is instrumented (the sanitizer
flags apply to the host pass); nothing runs on a GPU."""
from __future__ import annotations

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "host", "runtime_host_check.cpp")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=undefined"]


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
def test_runtime_host_logic_under_sanitizers(tmp_path):
    obj, exe = tmp_path / "check.o", tmp_path / "check"
    common = ["--offload-arch=gfx950", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer"]
    subprocess.run([HIPCC, "-x", "hip", *common, *SAN, "-c", SRC, "-o", str(obj)], check=True,
                   capture_output=True, text=True, timeout=600)
    subprocess.run([HIPCC, "--offload-arch=gfx950", *SAN, str(obj), "-o", str(exe)], check=True,
                   capture_output=True, text=True, timeout=600)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    res = subprocess.run([str(exe), "300"], capture_output=True, text=True, timeout=600, env=env)
    assert res.returncode == 0, (res.stdout + res.stderr)[-4000:]
    assert " 0 failures" in res.stdout, res.stdout
    assert "runtime error" not in res.stderr and "AddressSanitizer" not in res.stderr, res.stderr[-4000:]
