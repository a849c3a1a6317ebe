"""Seeded random configurations against the fp64 oracle, through the C ABI.

Each case draws a head shape (head_dim 64/128, 1-4 KV heads, 1-8 query heads per
KV head, k soft rows 1-64), widths, pooling, bias, storage dtype, a ragged batch
(empty, one-token and tail-ending contexts), a cache layout (16/32/64-token
pages or contiguous storage), an automatic or fixed split length, and a mode:
one task, several tasks in one call, last-row-only, or the recursive form.  The
cases together reach attention workgroups of 1 to 12 waves, one or several
query groups and splits, every merge block shape, and the GEMM tile fallbacks
of narrow widths."""
from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import probe as oracle
from paper_2608_28099_amd import binding, configs, inputs
from tests import helpers as H

pytestmark = pytest.mark.gpu

N_CASES = 32


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    binding.load()
    return torch.device("cuda:0")


def draw(i: int):
    """Case i: (workload, mode, tasks, split_len), from a generator seeded by i."""
    rng = np.random.default_rng(7000 + i)
    dtype = "f32" if rng.random() < 0.2 else "bf16"
    hd = int(rng.choice([64, 128]))
    n_kv = int(rng.choice([1, 2, 4]))
    g = int(rng.choice([1, 2, 3, 4, 5, 8]))
    mode = str(rng.choice(["one", "tasks", "last", "recursive"], p=[0.4, 0.2, 0.2, 0.2]))
    tasks = int(rng.integers(2, 5)) if mode in ("tasks", "last") and rng.random() < 0.7 else 1
    k = int(rng.choice([1, 2, 3, 5, 8, 13, 16, 24, 32, 48, 64]))
    if dtype == "f32":
        k = max(1, min(k, 64 // (g * tasks)))    # the fp32 path holds <= 64 rows per KV head
    mult = 32 if dtype == "bf16" else 4
    hidden = int(rng.choice([64, 128, 256, 320]))
    inter = int(rng.choice([64, 96, 160, 256]))
    hidden, inter = -(-hidden // mult) * mult, -(-inter // mult) * mult
    batch = int(rng.integers(1, 7))
    lens = [int(x) for x in rng.choice([0, 1, 31, 32, 33, 255, 257, 511, 700], size=batch)]
    lens = [int(rng.integers(0, 800)) if rng.random() < 0.3 else n for n in lens]
    layout = str(rng.choice(["paged", "contiguous"], p=[0.75, 0.25]))
    block = int(rng.choice([16, 32, 64]))
    pool = "mean" if mode not in ("last", "recursive") and rng.random() < 0.3 else "last"
    w = configs.Workload(
        name=f"rand{i}_{dtype}_hd{hd}_kv{n_kv}_g{g}_k{k}_{mode}{tasks}", dtype=dtype, batch=batch, k=k,
        hidden=hidden, n_q_heads=n_kv * g, n_kv_heads=n_kv, head_dim=hd, intermediate=inter,
        n_classes=int(rng.choice([1, 2, 5])), seq_len=("list", tuple(lens)), layout=layout,
        block_size=block, kv_std=1.0, weight_std=0.05, soft_std=0.5, pool=pool,
        cls_bias=bool(rng.random() < 0.5), seed=9000 + i)
    split_len = 256 if rng.random() < 0.5 else 0
    return w, mode, tasks, split_len


@pytest.mark.parametrize("i", range(N_CASES), ids=lambda i: f"case{i}")
def test_random_configuration(i, dev):
    w, mode, T, split_len = draw(i)
    print(f"[random] {w.name} lens={w.seq_len[1]} layout={w.layout}/{w.block_size} split={split_len}",
          flush=True)
    lens = inputs.seq_lens(w)
    kv = inputs.kv_cache(w, lens, "cpu")
    params = inputs.params(w, "cpu")
    kv_d, p_d = H.to_device(kv, params, dev)
    flags = binding.SP_FLAG_LAST_ROW_ONLY if mode == "last" else 0
    probe = binding.Probe(w, split_len=split_len, flags=flags, max_tasks=T)
    try:
        if mode == "recursive":
            fusion = inputs.fusion_params(w, "cpu")
            f_d = {name: v.to(dev) for name, v in fusion.items()}
            got = probe.forward_recursive(kv_d, p_d, f_d).cpu().numpy()
            ref = np.stack([o["logits"] for o in
                            H.oracle_outputs_recursive(w, kv, params, fusion, range(w.batch))])
            H.check_logits(got, ref, w.dtype, w.name)
        elif mode in ("tasks", "last"):
            tasks = inputs.task_params(w, T, "cpu")
            t_d = {name: (None if v is None else v.to(dev)) for name, v in tasks.items()}
            got = probe.forward_multi(kv_d, p_d, t_d["soft_prompts"], t_d["w_cls"], t_d["b_cls"]).cpu().numpy()
            kvs = [tuple(t.double().cpu().numpy() for t in kv.logical_kv(b)) for b in range(w.batch)]
            f = lambda t: None if t is None else t.double().cpu().numpy()
            ref = oracle.probe_batch_tasks(kvs, f(tasks["soft_prompts"]), f(tasks["w_cls"]), f(tasks["b_cls"]),
                                           H.oracle_weights(params), H.head_shape(w))
            for t in range(T):
                H.check_logits(got[:, t], ref[:, t], w.dtype, f"{w.name} task {t}")
        else:
            got = probe.forward(kv_d, p_d).cpu().numpy()
            ref = np.stack([o["logits"] for o in H.oracle_outputs(w, kv, params, range(w.batch))])
            H.check_logits(got, ref, w.dtype, w.name)
    finally:
        probe.close()
