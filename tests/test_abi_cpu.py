"""Host-side checks of the C-ABI library: it loads, exports every function the
header declares, and its host logic (config checks, workspace sizing, status
strings) behaves, without any compute call (CPU only)."""
from __future__ import annotations

import ctypes
import os
import re

import pytest

from paper_2608_28099_amd import binding, configs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sp_probe.h")

pytestmark = pytest.mark.skipif(not os.path.exists(binding.LIB_PATH),
                                reason="libsp_probe.so not built (run __graft_entry__.build())")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sp_probe_\w+)\s*\(", text)))


def test_header_declares_the_binding_exports():
    assert declared_functions() == sorted(binding.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = binding.load()
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_only_abi_symbols_are_exported():
    import subprocess
    out = subprocess.run(["nm", "-D", "--defined-only", binding.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = sorted(l.split()[-1] for l in out.splitlines() if " T " in l)
    assert exported == declared_functions()


def test_status_strings():
    for st, name in binding.STATUS.items():
        assert binding.sp_probe_status_string(st).startswith(name)
    assert binding.sp_probe_status_string(12345) == "unknown status"


def test_struct_layouts_match_the_c_compiler(tmp_path):
    """ctypes mirrors of the four ABI structs have the sizes and field offsets
    gcc gives the header's declarations."""
    import shutil
    import subprocess
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    structs = {"sp_probe_config": binding.sp_probe_config, "sp_kv_cache": binding.sp_kv_cache,
               "sp_probe_weights": binding.sp_probe_weights, "sp_probe_fusion": binding.sp_probe_fusion}
    lines = ['#include <stdio.h>', '#include <stddef.h>', f'#include "{HEADER}"', "int main(void) {"]
    for name, cls in structs.items():
        lines.append(f'  printf("{name} %zu\\n", sizeof({name}));')
        for field, _ in cls._fields_:
            lines.append(f'  printf("{name}.{field} %zu\\n", offsetof({name}, {field}));')
    lines.append("  return 0; }")
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", "-o", str(exe), str(src)], check=True)
    out = dict(l.split() for l in subprocess.run([str(exe)], capture_output=True, text=True,
                                                 check=True).stdout.splitlines())
    for name, cls in structs.items():
        assert int(out[name]) == ctypes.sizeof(cls), name
        for field, _ in cls._fields_:
            assert int(out[f"{name}.{field}"]) == getattr(cls, field).offset, (name, field)


@pytest.mark.parametrize("name", sorted(configs.WORKLOADS))
def test_workspace_sizing(name):
    w = configs.WORKLOADS[name]
    cfg = binding.make_config(w)
    n = binding.sp_probe_workspace_bytes(cfg)
    M = w.batch * w.k
    e = 2 if w.dtype == "bf16" else 4
    # at least the activations: attention output, a, w, s, y
    floor = M * (w.n_q_heads * w.head_dim * e + w.hidden * (4 + e + 4) + w.intermediate * e)
    assert n >= floor
    assert n < 64 << 30


def test_invalid_configs_are_rejected_without_a_device():
    w = configs.SMALL_BF16
    bad = [dict(head_dim=96), dict(n_kv_heads=3), dict(k=0), dict(k=65), dict(n_classes=0),
           dict(hidden=500), dict(intermediate=100), dict(split_len=300), dict(split_len=128),
           dict(max_batch=0), dict(dtype=7), dict(flags=8),
           dict(max_batch=1 << 20),  # projection operands past 32-bit byte offsets
           dict(max_tasks=65), dict(max_tasks=-1), dict(max_tasks=64, k=17),
           dict(flags=4, pool=1)]     # last-row-only needs LAST pooling
    for kw in bad:
        cfg = binding.make_config(w)
        for k, v in kw.items():
            setattr(cfg, k, v)
        assert binding.sp_probe_workspace_bytes(cfg) == 0, kw
        h = ctypes.c_void_p()
        st = binding.load().sp_probe_init(ctypes.byref(cfg), ctypes.byref(h))
        assert st in (-1, -2), (kw, st)
        assert h.value is None


def test_null_arguments():
    lib = binding.load()
    assert lib.sp_probe_init(None, None) == -1
    assert lib.sp_probe_forward(None, None, None, None, None, None, None, None) == -1
    assert lib.sp_probe_forward_recursive(None, None, None, None, None, None, None, None, None, None) == -1
    assert lib.sp_probe_plan_recursive(None, 1, None, None, None, None) == -1
    assert lib.sp_probe_destroy(None) == 0
    assert lib.sp_probe_tap_bytes(None, 0, 1) == 0
    assert lib.sp_probe_check_device_error(None, None) == -1


def test_workspace_grows_with_tasks():
    w = configs.QWEN9B_BF16
    one = binding.sp_probe_workspace_bytes(binding.make_config(w))
    four = binding.sp_probe_workspace_bytes(binding.make_config(w, max_tasks=4))
    pruned = binding.sp_probe_workspace_bytes(binding.make_config(w, max_tasks=4, flags=binding.SP_FLAG_LAST_ROW_ONLY))
    assert four > 3 * one // 2 and 0 < pruned


def test_bench_refuses_more_than_one_gpu():
    """bench.py measures one GPU; --gpus N > 1 exits with status 2 and says why,
    before anything touches a device."""
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    res = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120)
    assert res.returncode == 2
    assert "one GPU" in res.stderr and not res.stdout.strip()
