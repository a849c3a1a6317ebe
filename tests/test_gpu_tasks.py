"""GPU parity of the multi-task one-pass forward (several soft prompts and
classifiers on one cache, Sec. 3.3) and of the last-row-only execution
(SP_FLAG_LAST_ROW_ONLY: under LAST pooling only the last soft row of each task
runs past the attention) against the fp64 oracle, through the C ABI."""
from __future__ import annotations

import os

import numpy as np
import pytest
import torch

from oracle import probe as oracle
from paper_2608_28099_amd import binding, configs, inputs
from tests import helpers as H

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    binding.load()
    return torch.device("cuda:0")


def announce(msg):
    print(msg, flush=True)


def case(w, dev, n_tasks):
    lens = inputs.seq_lens(w)
    kv = inputs.kv_cache(w, lens, "cpu")
    params = inputs.params(w, "cpu")
    tasks = inputs.task_params(w, n_tasks, "cpu")
    kv_d, p_d = H.to_device(kv, params, dev)
    t_d = {k: (None if v is None else v.to(dev)) for k, v in tasks.items()}
    return kv, params, tasks, kv_d, p_d, t_d


def oracle_tasks(w, kv, params, tasks, idx=None):
    idx = range(w.batch) if idx is None else idx
    W = H.oracle_weights(params)
    kvs = [tuple(t.double().cpu().numpy() for t in kv.logical_kv(b)) for b in idx]
    f = lambda t: None if t is None else t.double().cpu().numpy()
    return oracle.probe_batch_tasks(kvs, f(tasks["soft_prompts"]), f(tasks["w_cls"]), f(tasks["b_cls"]),
                                    W, H.head_shape(w))


def run_tasks(probe, kv_d, p_d, t_d, n):
    return probe.forward_multi(kv_d, p_d, t_d["soft_prompts"][:n].contiguous(), t_d["w_cls"][:n].contiguous(),
                               None if t_d["b_cls"] is None else t_d["b_cls"][:n].contiguous())


TASK_CASES = [
    (configs.TINY_RAGGED_F32, 2, 0),
    (configs.SMALL_BF16, 3, 0),
    (configs.SMALL_G5_BF16, 4, 0),                                   # mean pooling, bias
    (configs.SMALL_BF16, 3, binding.SP_FLAG_LAST_ROW_ONLY),
    (configs.SMALL_BF16.replace(name="small_bf16_k17", k=17, seed=80), 2, binding.SP_FLAG_LAST_ROW_ONLY),
    (configs.TINY_RAGGED_F32, 2, binding.SP_FLAG_LAST_ROW_ONLY),
    # 64 sequences x 8 KV heads x 2 tasks of k = 48: the merge takes blocks of 32
    # soft rows (two per task, the second partial); 384 query rows per KV head
    (configs.Workload(name="tasks_merge_blocks", dtype="bf16", batch=64, k=48, hidden=256, n_q_heads=32,
                      n_kv_heads=8, head_dim=128, intermediate=128, n_classes=2,
                      seq_len=("uniform", 1, 64), kv_std=1.0, weight_std=0.05, seed=43), 2, 0),
]


@pytest.mark.parametrize("w,T,flags", TASK_CASES, ids=lambda x: getattr(x, "name", str(x)))
def test_tasks_match_oracle(w, T, flags, dev):
    """Every task of a T-task call, and the calls with fewer tasks on the same handle."""
    announce(f"[tasks] {w.name} T={T} flags={flags}")
    kv, params, tasks, kv_d, p_d, t_d = case(w, dev, T)
    probe = binding.Probe(w, flags=flags, max_tasks=T)
    ref = oracle_tasks(w, kv, params, tasks)
    for n in (T, 1):
        got = run_tasks(probe, kv_d, p_d, t_d, n).cpu().numpy()
        assert got.shape == (w.batch, n, w.n_classes)
        for t in range(n):
            err = H.check_logits(got[:, t], ref[:, t], w.dtype, f"{w.name} T={n} task {t}")
        announce(f"[tasks] {w.name} T={n}: max err {err:.3e}")
    # the one-task entry point on the same handle is task 0
    one = probe.forward(kv_d, p_d).cpu().numpy()
    H.check_logits(one, ref[:, 0], w.dtype, f"{w.name} single")
    probe.close()


@pytest.mark.parametrize("k", [1, 5, 16])
def test_last_row_only_matches_full_forward(k, dev):
    """Same logits as the full one-pass forward within the bf16 bar, for SP-1
    (where nothing is pruned), SP-5 and SP-16, and both against the oracle."""
    w = configs.SMALL_BF16.replace(name=f"small_last_k{k}", k=k, seed=90 + k)
    kv, params, tasks, kv_d, p_d, t_d = case(w, dev, 1)
    full = binding.Probe(w)
    pruned = binding.Probe(w, flags=binding.SP_FLAG_LAST_ROW_ONLY)
    assert pruned.plan(w.batch)["rows_per_kv_head"] == w.group
    a = full.forward(kv_d, p_d).cpu().numpy()
    b = pruned.forward(kv_d, p_d).cpu().numpy()
    ref = np.stack([o["logits"] for o in H.oracle_outputs(w, kv, params, range(w.batch))])
    H.check_logits(a, ref, w.dtype, "full")
    H.check_logits(b, ref, w.dtype, "last row only")
    assert np.max(np.abs(a - b)) < 5e-3
    full.close()
    pruned.close()


def test_last_row_only_taps(dev):
    """The pruned forward's attention output and residuals are the oracle's last soft row."""
    w = configs.SMALL_BF16
    kv, params, tasks, kv_d, p_d, t_d = case(w, dev, 1)
    probe = binding.Probe(w, flags=binding.SP_FLAG_LAST_ROW_ONLY)
    probe.forward(kv_d, p_d)
    B, d = w.batch, w.hidden
    o = probe.tap(binding.SP_TAP_ATTN, B, dev).view(torch.float16).cpu().double().numpy()[: B * w.n_q_heads * w.head_dim]
    y = probe.tap(binding.SP_TAP_Y, B, dev).view(torch.float32).cpu().double().numpy()[: B * d]
    probe.close()
    outs = H.oracle_outputs(w, kv, params, range(B))
    o = o.reshape(B, -1)
    y = y.reshape(B, d)
    for b in range(B):
        for got, ref, what in ((o[b], outs[b]["o"][-1], "o"), (y[b], outs[b]["y"][-1], "y")):
            e = np.max(np.abs(got - ref)) / np.max(np.abs(ref))
            assert e <= 1e-2, f"{what} b={b}: relative error {e:.3e}"


def test_task_count_errors(dev):
    w = configs.SMALL_BF16
    kv, params, tasks, kv_d, p_d, t_d = case(w, dev, 2)
    probe = binding.Probe(w, max_tasks=2)
    out = torch.full((w.batch, 3, w.n_classes), 7.0, device=dev)
    stream = torch.cuda.current_stream().cuda_stream
    wt = binding.make_weights(dict(p_d, w_cls=t_d["w_cls"]))
    for n in (0, 3, -1):
        st = binding.sp_probe_forward_multi(probe.h, binding.make_kv(kv_d), kv_d.seq_lens.data_ptr(),
                                            kv_d.block_table.data_ptr(), n, t_d["soft_prompts"].data_ptr(),
                                            wt, out.data_ptr(), stream)
        assert st == -1, (n, st)
    torch.cuda.synchronize()
    assert torch.all(out == 7.0)
    probe.close()


FULL = [(configs.LONG_9B_BF16, 4, binding.SP_FLAG_LAST_ROW_ONLY), (configs.LONG_9B_BF16, 1, binding.SP_FLAG_LAST_ROW_ONLY),
        (configs.QWEN27B_BF16, 1, binding.SP_FLAG_LAST_ROW_ONLY), (configs.QWEN9B_BF16, 3, 0)]


@pytest.mark.slow
@pytest.mark.parametrize("w,T,flags", FULL, ids=lambda x: getattr(x, "name", str(x)))
def test_tasks_full_size_sampled_sequences(w, T, flags, dev):
    announce(f"[tasks full] {w.name} T={T} flags={flags}: generating on the GPU")
    lens = inputs.seq_lens(w)
    kv = inputs.kv_cache(w, lens, dev)
    params = inputs.params(w, dev)
    tasks = inputs.task_params(w, T, dev)
    probe = binding.Probe(w, flags=flags, max_tasks=T)
    got = probe.forward_multi(kv, params, tasks["soft_prompts"], tasks["w_cls"], tasks["b_cls"]).cpu().numpy()
    torch.cuda.synchronize()
    announce(f"[tasks full] {w.name}: forward done")
    rng = np.random.default_rng(300 + w.seed)
    pick = sorted({int(np.argmin(lens)), int(np.argmax(lens)), *rng.choice(w.batch, 1, replace=False).tolist()})
    if os.environ.get("SP_FULL_SAMPLES"):
        pick = pick[: int(os.environ["SP_FULL_SAMPLES"])]
    ref = oracle_tasks(w, kv, params, tasks, pick)
    for i, b in enumerate(pick):
        for t in range(T):
            err = H.check_logits(got[b:b + 1, t], ref[i:i + 1, t], w.dtype, f"{w.name} b={b} task {t}")
        announce(f"[tasks full] {w.name}: b={b} N={lens[b]} max err {err:.3e}")
    probe.close()
    del kv, params
    torch.cuda.empty_cache()


LIMIT_CASES = [
    # k = 64 soft rows (the largest k) x 16 tasks = 1024 rows per sequence (the
    # largest tasks x k), 64 classes (the largest classifier), one query head per
    # KV head, an empty context next to a ragged one
    (configs.Workload(name="limit_k64_t16_c64", dtype="bf16", batch=2, k=64, hidden=256, n_q_heads=2,
                      n_kv_heads=2, head_dim=128, intermediate=128, n_classes=64,
                      seq_len=("list", (0, 333)), kv_std=1.0, weight_std=0.05, seed=61), 16, 0),
    # 64 tasks (the largest task count) of k = 16 with four query heads per KV
    # head: 4096 query rows per KV head in one call, head_dim 64
    (configs.Workload(name="limit_t64_g4_hd64", dtype="bf16", batch=2, k=16, hidden=256, n_q_heads=8,
                      n_kv_heads=2, head_dim=64, intermediate=128, n_classes=2,
                      seq_len=("list", (257, 40)), kv_std=1.0, weight_std=0.05, seed=62), 64, 0),
    # the same 64 tasks with only each task's last row past the attention
    (configs.Workload(name="limit_t64_last", dtype="bf16", batch=2, k=16, hidden=256, n_q_heads=8,
                      n_kv_heads=2, head_dim=64, intermediate=128, n_classes=2,
                      seq_len=("list", (257, 40)), kv_std=1.0, weight_std=0.05, seed=63), 64,
     binding.SP_FLAG_LAST_ROW_ONLY),
    # the fp32 path at its cap of 64 query rows per KV head (4 tasks x k 8 x 2)
    (configs.Workload(name="limit_f32_rows64", dtype="f32", batch=3, k=8, hidden=128, n_q_heads=4,
                      n_kv_heads=2, head_dim=64, intermediate=64, n_classes=3,
                      seq_len=("list", (1, 64, 190)), kv_std=1.0, weight_std=0.1, seed=64), 4, 0),
]


@pytest.mark.parametrize("w,T,flags", LIMIT_CASES, ids=lambda x: getattr(x, "name", str(x)))
def test_largest_row_counts(w, T, flags, dev):
    """The largest k, task count, tasks x k, class count and fp32 row count the
    library accepts, every task against the oracle."""
    announce(f"[limits] {w.name} T={T} flags={flags}")
    kv, params, tasks, kv_d, p_d, t_d = case(w, dev, T)
    probe = binding.Probe(w, flags=flags, max_tasks=T)
    try:
        got = run_tasks(probe, kv_d, p_d, t_d, T).cpu().numpy()
        ref = oracle_tasks(w, kv, params, tasks)
        assert got.shape == (w.batch, T, w.n_classes)
        err = max(H.check_logits(got[:, t], ref[:, t], w.dtype, f"{w.name} task {t}") for t in range(T))
        announce(f"[limits] {w.name}: max err {err:.3e}")
    finally:
        probe.close()
