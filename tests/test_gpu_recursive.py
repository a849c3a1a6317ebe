"""GPU parity of the recursive SP-k forward (MTP input fusion, Sec. 3.1, chained
over k steps, Sec. 3.2) against the fp64 oracle, through the C ABI.

Small workloads: every sequence and logit, and every step's fused row, residuals
and attention output.  Full-size workloads in the benchmark's launch
configuration: sampled sequences.  Bitwise invariances, the read-only cache,
host-side errors and profiling as for the one-pass forward.
"""
from __future__ import annotations

import os

import numpy as np
import pytest
import torch

from paper_2608_28099_amd import binding, configs, inputs
from tests import helpers as H

pytestmark = pytest.mark.gpu

SMALL = [configs.TINY_F32_SP2, configs.TINY_RAGGED_F32_SP5, configs.SMALL_BF16_SP5,
         configs.SMALL_BF16_SP1, configs.SMALL_G5_BF16_SP2]


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    binding.load()
    return torch.device("cuda:0")


def announce(msg):
    print(msg, flush=True)


def case(w, dev, layout=None, block_size=None):
    lens = inputs.seq_lens(w)
    kv = inputs.kv_cache(w, lens, "cpu", layout=layout, block_size=block_size)
    params = inputs.params(w, "cpu")
    fusion = inputs.fusion_params(w, "cpu")
    kv_d, p_d = H.to_device(kv, params, dev)
    f_d = {k: v.to(dev) for k, v in fusion.items()}
    return kv, params, fusion, kv_d, p_d, f_d


def oracle_logits(w, kv, params, fusion, idx=None):
    idx = range(w.batch) if idx is None else idx
    return np.stack([o["logits"] for o in H.oracle_outputs_recursive(w, kv, params, fusion, idx)])


@pytest.mark.parametrize("w", SMALL, ids=lambda w: w.name)
def test_small_recursive_logits_match_oracle(w, dev):
    announce(f"[recursive] {w.name}")
    kv, params, fusion, kv_d, p_d, f_d = case(w, dev)
    probe = binding.Probe(w)
    got = probe.forward_recursive(kv_d, p_d, f_d).cpu().numpy()
    err = H.check_logits(got, oracle_logits(w, kv, params, fusion), w.dtype, w.name)
    announce(f"[recursive] {w.name}: max err {err:.3e}")
    probe.close()


@pytest.mark.parametrize("w", SMALL, ids=lambda w: w.name)
def test_small_recursive_steps_match_oracle(w, dev):
    """Every step: the fused row x_t, the attention output, the residuals a_t, y_t."""
    announce(f"[recursive taps] {w.name}")
    kv, params, fusion, kv_d, p_d, f_d = case(w, dev)
    probe = binding.Probe(w)
    probe.forward_recursive(kv_d, p_d, f_d)
    B, k, d = w.batch, w.k, w.hidden
    act = torch.float16 if w.dtype == "bf16" else torch.float32
    taps = {name: probe.tap(t, B, dev).view(dt).cpu().double().numpy().reshape(B, k, -1)
            for name, t, dt in (("x", binding.SP_TAP_X, torch.float32), ("o", binding.SP_TAP_ATTN, act),
                                ("a", binding.SP_TAP_A, torch.float32), ("y", binding.SP_TAP_Y, torch.float32))}
    probe.close()
    outs = H.oracle_outputs_recursive(w, kv, params, fusion, range(B))
    rel = 1e-4 if w.dtype == "f32" else 1e-2
    for b in range(B):
        for name, got in taps.items():
            ref = outs[b][name]
            e = np.max(np.abs(got[b] - ref)) / max(np.max(np.abs(ref)), 1e-30)
            assert e <= rel, f"{w.name} {name} b={b}: relative error {e:.3e}"


@pytest.mark.parametrize("k", [3, 17])
def test_recursive_splits_and_step_counts(k, dev):
    """Several attention splits per sequence (split_len 256), k crossing a 16-row
    boundary, head_dim 64 and 128, both dtypes."""
    for dtype in ("bf16", "f32"):
        for hd in (64, 128):
            w = configs.Workload(name=f"rec_splits_{dtype}_{hd}_k{k}", dtype=dtype, batch=3, k=k,
                                 hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=hd, intermediate=320,
                                 n_classes=2, seq_len=("list", (700, 256, 1)), kv_std=1.0,
                                 weight_std=0.05, seed=70 + k)
            kv, params, fusion, kv_d, p_d, f_d = case(w, dev)
            probe = binding.Probe(w, split_len=256)
            assert probe.plan_recursive(w.batch)["max_splits"] == 3
            got = probe.forward_recursive(kv_d, p_d, f_d).cpu().numpy()
            H.check_logits(got, oracle_logits(w, kv, params, fusion), w.dtype, w.name)
            probe.close()


def test_one_pass_and_recursive_share_a_handle(dev):
    """Both forwards on one handle, interleaved: each keeps matching the oracle
    and repeats bit for bit."""
    w = configs.SMALL_BF16_SP5
    kv, params, fusion, kv_d, p_d, f_d = case(w, dev)
    probe = binding.Probe(w)
    rec0 = probe.forward_recursive(kv_d, p_d, f_d).clone()
    one0 = probe.forward(kv_d, p_d).clone()
    rec1 = probe.forward_recursive(kv_d, p_d, f_d).clone()
    one1 = probe.forward(kv_d, p_d).clone()
    assert torch.equal(rec0, rec1) and torch.equal(one0, one1)
    H.check_logits(rec1.cpu().numpy(), oracle_logits(w, kv, params, fusion), w.dtype, "recursive")
    ref_one = np.stack([o["logits"] for o in H.oracle_outputs(w, kv, params, range(w.batch))])
    H.check_logits(one1.cpu().numpy(), ref_one, w.dtype, "one-pass")
    probe.close()


def test_recursive_invariances_are_bitwise(dev):
    w = configs.SMALL_BF16_SP5
    kv, params, fusion, kv_d, p_d, f_d = case(w, dev)
    probe = binding.Probe(w)
    base = probe.forward_recursive(kv_d, p_d, f_d).clone()
    for layout, bs, seed in (("paged", 32, 6), ("contiguous", None, 0)):
        kv2 = inputs.repack(kv, layout, bs, perm_seed=seed)
        kv2_d, _ = H.to_device(kv2, params, dev)
        out = probe.forward_recursive(kv2_d, p_d, f_d)
        assert torch.equal(out, base), f"{layout} bs={bs} differs"
    perm = [3, 0, 4, 2, 1]
    kvp = inputs.permute_batch(kv_d, perm)
    fp = dict(f_d, hidden_last=f_d["hidden_last"][perm].contiguous())
    out = probe.forward_recursive(kvp, p_d, fp)
    assert torch.equal(out, base[perm]), "batch permutation changes the logits"
    probe.close()


def test_recursive_does_not_write_the_cache(dev):
    w = configs.TINY_RAGGED_F32_SP5
    kv, params, fusion, kv_d, p_d, f_d = case(w, dev)
    before = kv_d.pool.clone()
    bt_before = kv_d.block_table.clone()
    probe = binding.Probe(w)
    probe.forward_recursive(kv_d, p_d, f_d)
    torch.cuda.synchronize()
    assert torch.equal(kv_d.pool.view(torch.int32), before.view(torch.int32))
    assert torch.equal(kv_d.block_table, bt_before)
    probe.close()


def test_recursive_host_errors(dev):
    w = configs.SMALL_BF16_SP5
    kv, params, fusion, kv_d, p_d, f_d = case(w, dev)
    probe = binding.Probe(w)
    sentinel = torch.full((w.batch, w.n_classes), 123.0, device=dev)
    stream = torch.cuda.current_stream().cuda_stream
    wt = binding.make_weights(p_d)
    fu = binding.make_fusion(f_d)
    kvc = binding.make_kv(kv_d)
    hl = f_d["hidden_last"].data_ptr()

    def call(kvx=kvc, hidden=hl, fusion=fu):
        return binding.sp_probe_forward_recursive(probe.h, kvx, kv_d.seq_lens.data_ptr(),
                                                  kv_d.block_table.data_ptr(),
                                                  p_d["soft_prompt"].data_ptr(), hidden, fusion, wt,
                                                  sentinel.data_ptr(), stream)

    assert call(kvx=binding.make_kv(kv_d, 0)) == 0            # empty batch: no-op
    assert call(kvx=binding.make_kv(kv_d, w.batch + 1)) == -6
    assert call(hidden=None) == -1
    assert call(hidden=hl + 2) == -1                           # misaligned
    assert call(fusion=binding.make_fusion(dict(f_d, w_fc=None))) == -1
    torch.cuda.synchronize()
    assert torch.all(sentinel == 123.0), "logits written despite an error"
    probe.close()


def test_recursive_profile_reports_every_stage(dev):
    w = configs.SMALL_BF16_SP5
    kv, params, fusion, kv_d, p_d, f_d = case(w, dev)
    probe = binding.Probe(w, flags=binding.SP_FLAG_PROFILE)
    for _ in range(3):
        probe.forward_recursive(kv_d, p_d, f_d)
    stages, n = probe.profile_read()
    assert n == 3
    assert all(v > 0 for v in stages.values()), stages
    probe.forward(kv_d, p_d)
    probe.forward_recursive(kv_d, p_d, f_d)
    stages, n = probe.profile_read()
    assert n == 2
    probe.close()


FULL = [configs.QWEN9B_BF16_SP5, configs.QWEN27B_BF16_SP2, configs.LONG_9B_BF16_SP5]


@pytest.mark.slow
@pytest.mark.parametrize("w", FULL, ids=lambda w: w.name)
def test_recursive_full_size_sampled_sequences(w, dev):
    announce(f"[recursive full] {w.name}: generating on the GPU")
    lens = inputs.seq_lens(w)
    kv = inputs.kv_cache(w, lens, dev)
    params = inputs.params(w, dev)
    fusion = inputs.fusion_params(w, dev)
    probe = binding.Probe(w)
    announce(f"[recursive full] {w.name}: plan {probe.plan_recursive(w.batch)}")
    got = probe.forward_recursive(kv, params, fusion).cpu().numpy()
    torch.cuda.synchronize()
    announce(f"[recursive full] {w.name}: forward done")
    rng = np.random.default_rng(200 + w.seed)
    pick = sorted({int(np.argmin(lens)), int(np.argmax(lens)), *rng.choice(w.batch, 2, replace=False).tolist()})
    if os.environ.get("SP_FULL_SAMPLES"):
        pick = pick[: int(os.environ["SP_FULL_SAMPLES"])]
    W = H.oracle_weights_recursive(params, fusion)
    for b in pick:
        ref = H.oracle_outputs_recursive(w, kv, params, fusion, [b], W=W)[0]["logits"]
        err = H.check_logits(got[b:b + 1], ref[None], w.dtype, f"{w.name} b={b} N={lens[b]}")
        announce(f"[recursive full] {w.name}: b={b} N={lens[b]} max err {err:.3e}")
    assert np.all(np.isfinite(got))
    probe.close()
    del kv, params
    torch.cuda.empty_cache()


def test_split_k_projections(dev):
    """Widths at which the projections of 17..32 rows (24 per step here) split K
    over several workgroups (fusion, Q/K/V, o, gate/up, down), in the recursive
    form and in the one-pass form with last-row-only execution, against the
    oracle."""
    w = configs.Workload(name="split_k_bf16", dtype="bf16", batch=24, k=2, hidden=2048, n_q_heads=16,
                         n_kv_heads=4, head_dim=128, intermediate=3072, n_classes=3,
                         seq_len=("uniform", 0, 2100), seed=95)
    kv, params, fusion, kv_d, p_d, f_d = case(w, dev)
    probe = binding.Probe(w)
    got = probe.forward_recursive(kv_d, p_d, f_d).cpu().numpy()
    probe.close()
    err = H.check_logits(got, oracle_logits(w, kv, params, fusion), w.dtype, "recursive")
    announce(f"[split-k] recursive max err {err:.3e}")
    probe = binding.Probe(w, flags=binding.SP_FLAG_LAST_ROW_ONLY)
    got = probe.forward(kv_d, p_d).cpu().numpy()
    probe.close()
    ref = np.stack([o["logits"] for o in H.oracle_outputs(w, kv, params, range(w.batch))])
    err = H.check_logits(got, ref, w.dtype, "last row only")
    announce(f"[split-k] last-row-only max err {err:.3e}")
