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


def _split_rule(n_max, batch, n_kv, groups, waves, cus, hd=128):
    """The documented split rule, restated: splits sized so that the grid at the
    full batch and length fills one round of resident workgroups (cus x the
    workgroups a compute unit holds), capped at a third of the longest sequence,
    rounded up to 256 tokens, at least 1024."""
    per_cu = min(3, (12 if hd == 128 else 20) // waves)
    slots = cus * max(per_cu, 1)
    want = -(-(n_max * batch * n_kv * groups) // slots)
    third = (n_max + 2) // 3
    return max(1024, -(-min(want, third) // 256) * 256)


@pytest.mark.parametrize("cus", [64, 128, 256, 304, 512])
def test_split_plan_follows_the_compute_unit_count(cus):
    """The host plan reads the compute-unit count (a small batch of the long
    context: the one-round rule binds, not the third-of-a-sequence cap)."""
    w = configs.WORKLOADS["long_9b_bf16"]
    cfg = binding.make_config(w, max_batch=4)
    plan = binding.sp_probe_plan_config(cfg, cus)
    rows = w.k * w.n_q_heads // w.n_kv_heads
    assert plan["rows_per_kv_head"] == rows and plan["query_groups"] == 1
    sl = _split_rule(w.max_seq_len(), 4, w.n_kv_heads, 1, 4, cus)
    assert plan["split_len"] == sl
    assert plan["max_splits"] == -(-w.max_seq_len() // sl)


def test_split_plan_differs_across_compute_unit_counts_and_matches_workspace_bytes():
    w = configs.WORKLOADS["long_9b_bf16"]
    cfg = binding.make_config(w, max_batch=4)
    a, b = binding.sp_probe_plan_config(cfg, 128), binding.sp_probe_plan_config(cfg, 256)
    assert a["split_len"] > b["split_len"]   # half the compute units: longer splits
    assert a["max_splits"] < b["max_splits"]
    # more splits, more partials in the workspace
    assert b["workspace_bytes"] > a["workspace_bytes"]
    # with no device the sizing assumes 256 compute units
    assert binding.sp_probe_workspace_bytes(cfg) == b["workspace_bytes"]


def test_plan_config_rejects_bad_arguments():
    w = configs.SMALL_BF16
    cfg = binding.make_config(w)
    lib = binding.load()
    z = ctypes.c_int32()
    assert lib.sp_probe_plan_config(ctypes.byref(cfg), 0, None, None, None, None, None) == -1
    assert lib.sp_probe_plan_config(ctypes.byref(cfg), 1 << 20, None, None, None, None, None) == -1
    assert lib.sp_probe_plan_config(None, 256, ctypes.byref(z), None, None, None, None) == -1
    cfg.head_dim = 96
    assert lib.sp_probe_plan_config(ctypes.byref(cfg), 256, None, None, None, None, None) == -2


def test_packed_image_size():
    """The fp16 image holds a 256-byte header and the seven matrices, each
    segment rounded up to 256 bytes; none for fp32 configs."""
    w = configs.WORKLOADS["9b_bf16"]
    cfg = binding.make_config(w)
    d, hd, I = w.hidden, w.head_dim, w.intermediate
    segs = [(w.n_q_heads + 2 * w.n_kv_heads) * hd * d, d * w.n_q_heads * hd, I * d, I * d, d * I]
    assert binding.sp_probe_packed_bytes(cfg) == 256 + sum(-(-2 * n // 256) * 256 for n in segs)
    assert binding.sp_probe_packed_bytes(binding.make_config(configs.TINY_F32)) == 0
    lib = binding.load()
    wt = binding.sp_probe_weights()
    # host checks before any device is needed
    assert lib.sp_probe_pack_weights(ctypes.byref(binding.make_config(configs.TINY_F32)), ctypes.byref(wt),
                                     None, 0, None) == -2
    assert lib.sp_probe_pack_weights(ctypes.byref(cfg), ctypes.byref(wt), None, 0, None) == -1


def test_sp1_trainable_tensors_are_table_1s_count():
    """Table 1 (PII detection, 9B base, d = 4096): SP-1 with a one-logit linear head
    trains 8.2K numbers, 50x fewer than MultiMax's 412K.  The trainable inputs the
    C ABI takes are the soft prompt [k][d], w_cls [C][d] and the optional b_cls [C];
    drawn for k = 1, C = 1 at d = 4096 they hold 8,192 numbers (8,193 with the
    bias); every other tensor of the call is the frozen head.  Sec. 1's k = 5 soft
    vectors at the stated d = 3584 are 17,920, the quoted figure of about 18K."""
    from paper_2608_28099_amd import inputs

    hdr = open(os.path.join(ROOT, "include", "sp_probe.h")).read()
    assert "soft_prompt device [k][d]" in hdr and "w_cls[C][d], b_cls[C]" in hdr
    names = ("soft_prompt", "w_cls", "b_cls")
    w = configs.QWEN9B_BF16.replace(name="sp1_c1", k=1, n_classes=1, cls_bias=False)
    assert w.hidden == 4096
    p = inputs.params(w, "cpu", only=names)
    shapes = {n: tuple(t.shape) for n, t in p.items() if t is not None}
    assert shapes == {"soft_prompt": (1, 4096), "w_cls": (1, 4096)}
    n = sum(t.numel() for t in p.values() if t is not None)
    assert n == 8192 and f"{n / 1000:.1f}K" == "8.2K"
    pb = inputs.params(w.replace(cls_bias=True), "cpu", only=names)
    nb = sum(t.numel() for t in pb.values() if t is not None)
    assert nb == 8193 and f"{nb / 1000:.1f}K" == "8.2K"
    assert round(412_000 / n) == 50
    p5 = inputs.params(w.replace(k=5, hidden=3584), "cpu", only=("soft_prompt",))
    assert p5["soft_prompt"].numel() == 17920 and round(p5["soft_prompt"].numel(), -3) == 18000
