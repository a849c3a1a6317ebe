"""Build ``libsp_probe.so`` (gfx950 HIP kernels + C ABI) in the package directory."""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libsp_probe.so")
SOURCES = ["attention.hip", "merge.hip", "gemm.hip", "rowops.hip", "runtime.hip", "measure.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared", "-fvisibility=hidden",
    # packed fp32 instructions are kept out of every kernel
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # matrix-core accumulators in ordinary VGPRs: the attention state is rescaled
    # and masked by VALU code, and AGPR accumulators cost a copy each way
    "-mllvm", "-amdgpu-mfma-vgpr-form",
]


def build(verbose: bool = False, extra=None) -> str:
    """Compile every HIP source into LIB (always recompiles; one hipcc process
    per source, in parallel, then one link); returns the path."""
    import concurrent.futures
    import tempfile
    noise = "is not a recognized feature for this target"

    def run(cmd):
        if verbose:
            print(" ".join(cmd), flush=True)
        res = subprocess.run(cmd, capture_output=True, text=True)
        msgs = "\n".join(l for l in (res.stdout + res.stderr).splitlines() if noise not in l)
        if res.returncode != 0:
            raise RuntimeError(f"hipcc failed ({res.returncode}):\n{msgs}")
        if verbose and msgs.strip():
            print(msgs, file=sys.stderr)

    with tempfile.TemporaryDirectory(prefix="sp_probe_build_") as tmpdir:
        objs = [os.path.join(tmpdir, s.replace(".hip", ".o")) for s in SOURCES]
        cflags = [f for f in FLAGS if f != "-shared"]
        cmds = [[HIPCC, *cflags, *(extra or []), "-c", "-o", o, os.path.join(CSRC, s)]
                for s, o in zip(SOURCES, objs)]
        workers = min(len(cmds), max(1, (os.cpu_count() or 1)))
        with concurrent.futures.ThreadPoolExecutor(max_workers=workers) as ex:
            list(ex.map(run, cmds))
        tmp = LIB + ".tmp"
        run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs])
        os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True, extra=sys.argv[1:])
