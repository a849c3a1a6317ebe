"""GPU parity of the HIP probe forward against the fp64 oracle, through the C ABI.

Small workloads: every sequence, every logit, plus intermediate taps.  Full-size
workloads (the shapes the benchmark runs, same launch configuration): sampled
sequences the oracle recomputes one by one.  Invariances that must hold bit for
bit: batch order, block placement, contiguous vs paged storage, repeated runs.
"""
from __future__ import annotations

import dataclasses

import os

import numpy as np
import pytest
import torch

from paper_2608_28099_amd import binding, configs, inputs
from tests import helpers as H

pytestmark = pytest.mark.gpu

SMALL = [configs.TINY_F32, configs.TINY_PEAKY_F32, configs.TINY_RAGGED_F32, configs.SMALL_BF16,
         configs.SMALL_G5_BF16]


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    binding.load()
    return torch.device("cuda:0")


def small_case(w, dev, layout=None, block_size=None):
    lens = inputs.seq_lens(w)
    kv = inputs.kv_cache(w, lens, "cpu", layout=layout, block_size=block_size)
    params = inputs.params(w, "cpu")
    kv_d, p_d = H.to_device(kv, params, dev)
    return kv, params, kv_d, p_d


def announce(msg):
    print(msg, flush=True)


@pytest.mark.parametrize("w", SMALL, ids=lambda w: w.name)
def test_small_logits_match_oracle(w, dev):
    announce(f"[parity] {w.name}")
    kv, params, kv_d, p_d = small_case(w, dev)
    probe = binding.Probe(w)
    got = probe.forward(kv_d, p_d).cpu().numpy()
    ref = np.stack([o["logits"] for o in H.oracle_outputs(w, kv, params, range(w.batch))])
    err = H.check_logits(got, ref, w.dtype, w.name)
    announce(f"[parity] {w.name}: max err {err:.3e}")
    probe.close()


@pytest.mark.parametrize("w", SMALL, ids=lambda w: w.name)
def test_small_taps_match_oracle(w, dev):
    """Stage-wise: Q/K/V projections, attention output, residuals a and y."""
    announce(f"[taps] {w.name}")
    kv, params, kv_d, p_d = small_case(w, dev)
    probe = binding.Probe(w)
    probe.forward(kv_d, p_d)
    B, k, d = w.batch, w.k, w.hidden
    act = torch.float16 if w.dtype == "bf16" else torch.float32  # activations feeding the MFMAs
    outs = H.oracle_outputs(w, kv, params, range(B))
    qkv = probe.tap(binding.SP_TAP_QKV, B, dev).view(torch.float32).cpu().double().numpy()
    attn = probe.tap(binding.SP_TAP_ATTN, B, dev).view(act).cpu().double().numpy()
    a = probe.tap(binding.SP_TAP_A, B, dev).view(torch.float32).cpu().double().numpy()
    y = probe.tap(binding.SP_TAP_Y, B, dev).view(torch.float32).cpu().double().numpy()
    probe.close()
    W = H.oracle_weights(params)
    from oracle import probe as oracle
    u = oracle.rms_norm(params["soft_prompt"].double().numpy(), W["in_norm"], w.rms_eps)
    qkv_ref = np.concatenate([u @ W["w_q"].T, u @ W["w_k"].T, u @ W["w_v"].T], axis=1)
    # relative to the magnitude of each tensor: fp32 path ~1e-6; bf16-storage path
    # (fp16 operands, a few roundings of 2^-11) ~1e-3
    rel = 1e-4 if w.dtype == "f32" else 1e-2

    def close(x, r, what):
        scale = max(np.max(np.abs(r)), 1e-30)
        e = np.max(np.abs(x - r)) / scale
        assert e <= rel, f"{w.name} {what}: relative error {e:.3e}"

    close(qkv.reshape(k, -1), qkv_ref, "qkv")
    attn = attn.reshape(B, k, -1)
    for b in range(B):
        close(attn[b], outs[b]["o"], f"attention b={b}")
        close(a.reshape(B, k, d)[b], outs[b]["a"], f"a b={b}")
        close(y.reshape(B, k, d)[b], outs[b]["y"], f"y b={b}")


def test_mean_pool_and_bias(dev):
    w = configs.SMALL_BF16.replace(name="small_bf16_mean_bias", pool="mean", cls_bias=True, seed=21)
    kv, params, kv_d, p_d = small_case(w, dev)
    probe = binding.Probe(w)
    got = probe.forward(kv_d, p_d).cpu().numpy()
    ref = np.stack([o["logits"] for o in H.oracle_outputs(w, kv, params, range(w.batch))])
    H.check_logits(got, ref, w.dtype, w.name)
    probe.close()


@pytest.mark.parametrize("k", [1, 2, 17, 33, 64])
def test_soft_row_counts(k, dev):
    """k = 1 (SP-1), odd k crossing 16- and 32-row boundaries, and the maximum 64."""
    w = configs.SMALL_BF16.replace(name=f"small_k{k}", k=k, seed=30 + k)
    kv, params, kv_d, p_d = small_case(w, dev)
    probe = binding.Probe(w)
    got = probe.forward(kv_d, p_d).cpu().numpy()
    ref = np.stack([o["logits"] for o in H.oracle_outputs(w, kv, params, range(w.batch))])
    H.check_logits(got, ref, w.dtype, w.name)
    probe.close()


def test_rope_row_blocks_on_wide_batches(dev):
    """300 sequences of k = 6 soft rows: the RoPE scatter then takes several
    rows per workgroup (on a 256-CU device, blocks of 4 and 2 rows), so the
    per-row angle tables and the paired stores of every block position are
    checked: attention output and logits against the oracle for every
    sequence, in the one-pass form and with last-row-only (queries of the
    last row only)."""
    w = configs.Workload(name="wide_k6_bf16", dtype="bf16", batch=300, k=6, hidden=256, n_q_heads=4,
                         n_kv_heads=2, head_dim=64, intermediate=512, n_classes=2,
                         seq_len=("uniform", 0, 40), layout="paged", seed=61)
    announce(f"[rope rows] {w.name}")
    kv, params, kv_d, p_d = small_case(w, dev)
    outs = H.oracle_outputs(w, kv, params, range(w.batch))
    ref = np.stack([o["logits"] for o in outs])
    probe = binding.Probe(w)
    got = probe.forward(kv_d, p_d).cpu().numpy()
    attn = probe.tap(binding.SP_TAP_ATTN, w.batch, dev).view(torch.float16).cpu().double().numpy()
    probe.close()
    H.check_logits(got, ref, w.dtype, "one-pass")
    qw = w.n_q_heads * w.head_dim
    attn = attn.reshape(-1, qw)[: w.batch * w.k].reshape(w.batch, w.k, qw)
    for b in range(w.batch):
        o_ref = outs[b]["o"].reshape(w.k, qw)
        err = np.max(np.abs(attn[b] - o_ref)) / max(np.max(np.abs(o_ref)), 1e-30)
        assert err < 1e-2, (b, err)
    lro = binding.Probe(w, flags=binding.SP_FLAG_LAST_ROW_ONLY)
    got_l = lro.forward(kv_d, p_d).cpu().numpy()
    lro.close()
    H.check_logits(got_l, ref, w.dtype, "last-row-only")


@pytest.mark.parametrize("hd", [64, 128])
def test_head_dims_and_splits(hd, dev):
    """Several splits per sequence (split_len 256), head_dim 64 and 128, both dtypes."""
    for dtype in ("bf16", "f32"):
        w = configs.Workload(name=f"splits_{dtype}_{hd}", dtype=dtype, batch=3, k=3, hidden=256,
                             n_q_heads=4, n_kv_heads=2, head_dim=hd, intermediate=320, n_classes=2,
                             seq_len=("list", (700, 256, 1)), kv_std=1.0, weight_std=0.05, seed=40)
        kv, params, kv_d, p_d = small_case(w, dev)
        probe = binding.Probe(w, split_len=256)
        assert probe.plan(w.batch)["max_splits"] == 3
        got = probe.forward(kv_d, p_d).cpu().numpy()
        ref = np.stack([o["logits"] for o in H.oracle_outputs(w, kv, params, range(w.batch))])
        H.check_logits(got, ref, w.dtype, w.name)
        probe.close()


@pytest.mark.parametrize("case", [
    # (query heads, KV heads, k, lengths, splits): 64 rows per KV head (4 waves
    # per workgroup) with 3, 6 and 4 splits; 80 rows (5 waves) with 4 splits;
    # 160 rows (one workgroup of 10 waves) and 192 rows (12 waves)
    (16, 4, 16, (700, 256, 1, 0, 513, 768), 3),
    (16, 4, 16, (1500, 700, 1, 1290, 33), 6),
    (16, 4, 16, (1000, 257, 31, 769), 4),
    (10, 2, 16, (1024, 3, 600, 255), 4),
    (10, 2, 32, (700, 0, 33, 512), 3),
    (8, 2, 48, (300, 769, 17), 4),
], ids=["g4_s3", "g4_s6", "g4_s4", "g5_s4", "w10_s3", "w12_s4"])
def test_multi_split_wide_query_tiles(case, dev):
    """Several splits per sequence with 4- to 12-wave workgroups: ragged tails
    in any split, splits with no tokens, empty sequences."""
    n_q, n_kv, k, lens, n_splits = case
    w = configs.Workload(name=f"splits_g{n_q // n_kv}_k{k}_{n_splits}", dtype="bf16", batch=len(lens), k=k,
                         hidden=256, n_q_heads=n_q, n_kv_heads=n_kv, head_dim=128,
                         intermediate=320, n_classes=3, seq_len=("list", lens), kv_std=1.0,
                         weight_std=0.05, seed=41)
    announce(f"[multi-split] {w.name} lens={lens}")
    kv, params, kv_d, p_d = small_case(w, dev)
    probe = binding.Probe(w, split_len=256)
    plan = probe.plan(w.batch)
    assert plan["max_splits"] == n_splits
    assert plan["query_groups"] == 1 and plan["rows_per_kv_head"] == k * n_q // n_kv
    got = probe.forward(kv_d, p_d).cpu().numpy()
    ref = np.stack([o["logits"] for o in H.oracle_outputs(w, kv, params, range(w.batch))])
    H.check_logits(got, ref, w.dtype, w.name)
    probe.close()


def test_merge_rows_per_workgroup(dev):
    """A batch large enough that the merge gives each workgroup several soft
    rows (256 sequences x 8 KV heads, k = 48: blocks of 32 soft rows, the second
    block of each sequence partial), ragged and empty contexts."""
    w = configs.Workload(name="merge_blocks", dtype="bf16", batch=256, k=48, hidden=256, n_q_heads=16,
                         n_kv_heads=8, head_dim=128, intermediate=128, n_classes=3,
                         seq_len=("uniform", 0, 40), kv_std=1.0, weight_std=0.05, seed=42)
    announce(f"[merge blocks] {w.name}")
    kv, params, kv_d, p_d = small_case(w, dev)
    probe = binding.Probe(w)
    got = probe.forward(kv_d, p_d).cpu().numpy()
    ref = np.stack([o["logits"] for o in H.oracle_outputs(w, kv, params, range(w.batch))])
    H.check_logits(got, ref, w.dtype, w.name)
    probe.close()


def test_projection_tile_shapes(dev):
    """Shapes whose projections select the fallback tiles of the bf16 GEMM:
    64x64 (o-proj, down) and 32x64 (gate/up) at 256 rows x width 4096, the
    32-deep K step (width 4128 is not a multiple of 64) with head_dim 64, the
    split-K 256x128 tile of a deep down projection, the double-buffered
    256x256 gate/up tile on 304 rows (a second row tile of 48 rows), and the
    256x160 three-stage tile of the o and down products on 1280 rows x 7680
    (48 column tiles: one round where 256x128 takes two)."""
    cases = [
        configs.Workload(name="tiles_a", dtype="bf16", batch=16, k=16, hidden=4096, n_q_heads=8,
                         n_kv_heads=2, head_dim=128, intermediate=1024, n_classes=3,
                         seq_len=("uniform", 1, 300), seed=50),
        configs.Workload(name="tiles_b", dtype="bf16", batch=4, k=8, hidden=4128, n_q_heads=4,
                         n_kv_heads=2, head_dim=64, intermediate=512, n_classes=2,
                         seq_len=("list", (257, 64, 0, 33)), seed=51),
        # 144 rows and a down projection 8192 deep: 256 x 128 tiles with K split four ways
        configs.Workload(name="tiles_c", dtype="bf16", batch=9, k=16, hidden=512, n_q_heads=8,
                         n_kv_heads=2, head_dim=64, intermediate=8192, n_classes=2,
                         seq_len=("uniform", 0, 700), seed=52),
        # 304 rows, gate/up 1280 wide: 256 x 256 tiles in 64-deep double-buffered steps
        configs.Workload(name="tiles_d", dtype="bf16", batch=19, k=16, hidden=512, n_q_heads=8,
                         n_kv_heads=2, head_dim=64, intermediate=640, n_classes=2,
                         seq_len=("uniform", 0, 400), seed=53),
        # 1280 rows, o and down 7680 wide: 256 x 160 tiles
        configs.Workload(name="tiles_e", dtype="bf16", batch=80, k=16, hidden=7680, n_q_heads=8,
                         n_kv_heads=2, head_dim=128, intermediate=512, n_classes=2,
                         seq_len=("uniform", 0, 200), seed=54),
    ]
    for w in cases:
        announce(f"[tiles] {w.name}")
        kv, params, kv_d, p_d = small_case(w, dev)
        probe = binding.Probe(w)
        got = probe.forward(kv_d, p_d).cpu().numpy()
        ref = np.stack([o["logits"] for o in H.oracle_outputs(w, kv, params, range(w.batch))])
        err = H.check_logits(got, ref, w.dtype, w.name)
        announce(f"[tiles] {w.name}: max err {err:.3e}")
        probe.close()


def test_projection_split_launches(dev):
    """The launch plans that split one projection (on 256 compute units):
    gate/up on 272 rows x 2 x 16896 (264 tiles of 256x256, one round and 8 more)
    as 256x256 tiles over its first 16384 output columns and 256x128 tiles over
    the last 512 in a second launch; a down projection 8192 deep on 1040 rows x
    512 as 256x256 tiles with K split in two; and o and down on 2048 rows x 8448
    (264 tiles of 256x256) as 256x256 tiles over the first 8192 columns and
    256x128 over the last 256.  Logits and the residuals after the o-projection
    (SP_TAP_A) and the MLP (SP_TAP_Y) against the oracle, row by row."""
    cases = [
        configs.Workload(name="tiles_f", dtype="bf16", batch=17, k=16, hidden=256, n_q_heads=8,
                         n_kv_heads=2, head_dim=64, intermediate=16896, n_classes=2,
                         seq_len=("uniform", 0, 200), seed=55),
        configs.Workload(name="tiles_g", dtype="bf16", batch=65, k=16, hidden=512, n_q_heads=8,
                         n_kv_heads=2, head_dim=64, intermediate=8192, n_classes=3,
                         seq_len=("uniform", 0, 150), seed=56),
        configs.Workload(name="tiles_h", dtype="bf16", batch=128, k=16, hidden=8448, n_q_heads=8,
                         n_kv_heads=2, head_dim=64, intermediate=256, n_classes=2,
                         seq_len=("uniform", 0, 100), seed=57),
    ]
    for w in cases:
        announce(f"[split launches] {w.name}")
        kv, params, kv_d, p_d = small_case(w, dev)
        probe = binding.Probe(w)
        got = probe.forward(kv_d, p_d).cpu().numpy()
        taps = {n: probe.tap(t, w.batch, dev).view(torch.float32).cpu().double().numpy().reshape(w.batch, w.k, w.hidden)
                for n, t in (("a", binding.SP_TAP_A), ("y", binding.SP_TAP_Y))}
        probe.close()
        outs = H.oracle_outputs(w, kv, params, range(w.batch))
        H.check_logits(got, np.stack([o["logits"] for o in outs]), w.dtype, w.name)
        for n, x in taps.items():
            for b in range(w.batch):
                ref = outs[b][n]
                e = np.max(np.abs(x[b] - ref)) / np.max(np.abs(ref))
                assert e <= 1e-2, (w.name, n, b, e)


# ---------------------------------------------------------------- invariances (bitwise)

def test_invariances_are_bitwise(dev):
    w = configs.SMALL_BF16
    kv, params, kv_d, p_d = small_case(w, dev)
    probe = binding.Probe(w)
    base = probe.forward(kv_d, p_d).clone()
    again = probe.forward(kv_d, p_d).clone()
    assert torch.equal(base, again), "two identical runs differ"
    # block placement and block size
    for layout, bs, seed in (("paged", 16, 5), ("paged", 32, 6), ("contiguous", None, 0)):
        kv2 = inputs.repack(kv, layout, bs, perm_seed=seed)
        kv2_d, _ = H.to_device(kv2, params, dev)
        probe2 = binding.Probe(w, max_seq_len=w.max_seq_len())
        out = probe2.forward(kv2_d, p_d)
        assert torch.equal(out, base), f"{layout} bs={bs} differs"
        probe2.close()
    # batch order
    perm = [3, 0, 4, 2, 1]
    kvp = inputs.permute_batch(kv_d, perm)
    out = probe.forward(kvp, p_d)
    assert torch.equal(out, base[perm]), "batch permutation changes the logits"
    probe.close()


def test_attention_is_independent_of_the_grid(dev):
    """A sequence's attention output is the same bit for bit whether its launch
    is one round of workgroups (the co-resident workgroups then rotate their wave
    priorities) or several rounds (they do not): scheduling changes timing only."""
    w = configs.Workload(name="grid_rounds", dtype="bf16", batch=48, k=16, hidden=256, n_q_heads=32,
                         n_kv_heads=8, head_dim=128, intermediate=128, n_classes=2,
                         seq_len=("uniform", 600, 1024), kv_std=1.0, weight_std=0.05, seed=71)
    kv, params, kv_d, p_d = small_case(w, dev)
    probe = binding.Probe(w, split_len=256)
    plan = probe.plan(w.batch)
    assert plan["split_len"] == 256 and plan["max_splits"] == 4 and plan["query_groups"] == 1
    n = 4 * w.k * w.n_q_heads * w.head_dim  # attention output of the first four sequences
    # 8 KV heads x 4 splits x 48 sequences = 1536 four-wave workgroups: two rounds
    probe.forward(kv_d, p_d)
    many = probe.tap(binding.SP_TAP_ATTN, w.batch, dev).view(torch.float16)[:n].clone()
    # the first four sequences alone: 128 workgroups, one round
    bt = None if kv_d.block_table is None else kv_d.block_table[:4]
    few_kv = dataclasses.replace(kv_d, block_table=bt, seq_lens=kv_d.seq_lens[:4])
    probe.forward(few_kv, p_d)
    few = probe.tap(binding.SP_TAP_ATTN, 4, dev).view(torch.float16)[:n].clone()
    assert torch.equal(many, few), "the attention output depends on the grid"
    probe.close()


def test_kv_cache_is_not_written(dev):
    """Sec. 3.3: the soft rows' K/V go to scratch; the head's cache is untouched."""
    w = configs.TINY_RAGGED_F32
    kv, params, kv_d, p_d = small_case(w, dev)
    before = kv_d.pool.clone()
    bt_before = kv_d.block_table.clone()
    probe = binding.Probe(w)
    probe.forward(kv_d, p_d)
    torch.cuda.synchronize()
    assert torch.equal(kv_d.pool.view(torch.int32), before.view(torch.int32))
    assert torch.equal(kv_d.block_table, bt_before)
    probe.close()


def test_empty_batch_and_host_errors(dev):
    w = configs.SMALL_BF16
    kv, params, kv_d, p_d = small_case(w, dev)
    probe = binding.Probe(w)
    sentinel = torch.full((w.batch, w.n_classes), 123.0, device=dev)
    stream = torch.cuda.current_stream().cuda_stream
    wt = binding.make_weights(p_d)
    # B = 0: no-op
    st = binding.sp_probe_forward(probe.h, binding.make_kv(kv_d, 0), kv_d.seq_lens.data_ptr(),
                                  kv_d.block_table.data_ptr(), p_d["soft_prompt"].data_ptr(), wt,
                                  sentinel.data_ptr(), stream)
    assert st == 0
    # batch above capacity, a null weight, a misaligned pointer, a bad block size
    bad = []
    kvc = binding.make_kv(kv_d, w.batch + 1)
    bad.append((kvc, wt, binding.SP_OK - 6))
    wt_null = binding.make_weights(dict(p_d, w_o=None))
    bad.append((binding.make_kv(kv_d), wt_null, -1))
    kvm = binding.make_kv(kv_d)
    kvm.k_base += 2
    bad.append((kvm, wt, -1))
    kvb = binding.make_kv(kv_d)
    kvb.block_size = 24
    bad.append((kvb, wt, -1))
    for kvx, wtx, want in bad:
        st = binding.sp_probe_forward(probe.h, kvx, kv_d.seq_lens.data_ptr(),
                                      kv_d.block_table.data_ptr(), p_d["soft_prompt"].data_ptr(),
                                      wtx, sentinel.data_ptr(), stream)
        assert st == want, (st, want)
    torch.cuda.synchronize()
    assert torch.all(sentinel == 123.0), "logits written despite an error"
    probe.close()


def test_profile_mode_reports_every_stage(dev):
    w = configs.SMALL_BF16
    kv, params, kv_d, p_d = small_case(w, dev)
    probe = binding.Probe(w, flags=binding.SP_FLAG_PROFILE)
    for _ in range(3):
        probe.forward(kv_d, p_d)
    stages, n = probe.profile_read()
    assert n == 3
    assert all(v > 0 for v in stages.values()), stages
    probe.close()


# ---------------------------------------------------------------- full-size workloads

FULL = [configs.QWEN4B_BF16, configs.QWEN9B_BF16, configs.QWEN27B_BF16, configs.LONG_9B_BF16]


@pytest.mark.slow
@pytest.mark.parametrize("w", FULL, ids=lambda w: w.name)
def test_full_size_every_sequence(w, dev):
    """The workload at its full size on the GPU, in the benchmark's launch
    configuration; the oracle recomputes every sequence one by one (480 in all:
    about a minute of host time)."""
    announce(f"[full] {w.name}: generating on the GPU")
    lens = inputs.seq_lens(w)
    kv = inputs.kv_cache(w, lens, dev)
    params = inputs.params(w, dev)
    probe = binding.Probe(w)
    announce(f"[full] {w.name}: plan {probe.plan(w.batch)}")
    # the benchmark's launch configuration reads the fp16 weight image; the
    # forward without it returns the same logits bit for bit
    img = binding.pack_weights(w, params)
    got_t = probe.forward(kv, dict(params, packed=img)).clone()
    plain = probe.forward(kv, params).clone()
    torch.cuda.synchronize()
    assert torch.equal(got_t, plain)
    assert probe.check_device_error() == 0
    got = got_t.cpu().numpy()
    del img, plain
    announce(f"[full] {w.name}: forward done")
    assert np.all(np.isfinite(got))
    n = w.batch
    if os.environ.get("SP_FULL_SAMPLES"):
        n = min(n, int(os.environ["SP_FULL_SAMPLES"]))
    W = H.oracle_weights(params)
    errs = []
    for b in range(n):
        ref = H.oracle_outputs(w, kv, params, [b], W=W)[0]["logits"]
        errs.append(H.check_logits(got[b:b + 1], ref[None], w.dtype, f"{w.name} b={b} N={lens[b]}"))
        if b % 16 == 15 or b == n - 1:
            announce(f"[full] {w.name}: {b + 1}/{n} sequences, max err so far {max(errs):.3e}")
    errs = np.array(errs)
    announce(f"[full] {w.name}: max {errs.max():.3e} (N={lens[int(errs.argmax())]}), "
             f"p50 {np.median(errs):.3e} over {n} sequences")
    probe.close()
    del kv, params
    torch.cuda.empty_cache()


def test_debug_mode_reports_invalid_device_data(dev):
    """SP_FLAG_DEBUG: a seq_len past max_seq_len, a negative one, or a block id past
    the pool makes the forward (one-pass, multi-task or recursive) skip its work and
    sp_probe_check_device_error report SP_ERR_DEVICE_DATA; valid data then runs clean
    and matches the oracle."""
    w = configs.SMALL_BF16
    kv, params, kv_d, p_d = small_case(w, dev)
    fusion = {k: v.to(dev) for k, v in inputs.fusion_params(w, "cpu").items()}
    tasks = {k: (None if v is None else v.to(dev)) for k, v in inputs.task_params(w, 2, "cpu").items()}
    probe = binding.Probe(w, flags=binding.SP_FLAG_DEBUG, max_tasks=2)
    good_lens = kv_d.seq_lens.clone()
    good_table = kv_d.block_table.clone()
    bad_cases = []
    lens = good_lens.clone(); lens[2] = w.max_seq_len() + 1; bad_cases.append(("long seq_len", lens, good_table))
    lens = good_lens.clone(); lens[0] = -3; bad_cases.append(("negative seq_len", lens, good_table))
    table = good_table.clone(); table[4, 0] = kv_d.num_blocks + 7; bad_cases.append(("block id", good_lens, table))
    runs = {
        "one-pass": lambda kvx, out: probe.forward(kvx, p_d, out),
        "recursive": lambda kvx, out: probe.forward_recursive(kvx, p_d, fusion, out),
        "tasks": None,
    }
    for what, lens, table in bad_cases:
        for name, run in runs.items():
            kvx = inputs.KVCache(kv_d.pool, table, lens, kv_d.block_size, kv_d.max_blocks_per_seq, kv_d.n_kv,
                                 kv_d.head_dim)
            out = torch.full((w.batch, w.n_classes), 5.0, device=dev)
            if name == "tasks":
                out2 = torch.full((w.batch, 2, w.n_classes), 5.0, device=dev)
                probe.forward_multi(kvx, p_d, tasks["soft_prompts"], tasks["w_cls"], tasks["b_cls"], out2)
                assert probe.check_device_error() == -7, (what, name)
                assert torch.all(out2 == 5.0), (what, name)
            else:
                run(kvx, out)
                assert probe.check_device_error() == -7, (what, name)
                assert torch.all(out == 5.0), (what, name)
    got = probe.forward(kv_d, p_d).cpu().numpy()
    assert probe.check_device_error() == 0
    ref = np.stack([o["logits"] for o in H.oracle_outputs(w, kv, params, range(w.batch))])
    H.check_logits(got, ref, w.dtype, "after the errors")
    probe.close()


def test_largest_hidden_width(dev):
    """hidden = 16384, the widest the row kernels take (RMSNorm, RoPE scatter,
    classifier), against the oracle."""
    w = configs.Workload(name="wide_bf16", dtype="bf16", batch=2, k=2, hidden=16384, n_q_heads=4,
                         n_kv_heads=2, head_dim=64, intermediate=64, n_classes=2,
                         seq_len=("list", (40, 3)), seed=97)
    kv, params, kv_d, p_d = small_case(w, dev)
    probe = binding.Probe(w)
    got = probe.forward(kv_d, p_d).cpu().numpy()
    ref = np.stack([o["logits"] for o in H.oracle_outputs(w, kv, params, range(w.batch))])
    H.check_logits(got, ref, w.dtype, "one-pass")
    probe.close()


def test_many_tasks(dev):
    """Sixteen tasks of four soft rows in one call (64 soft rows, 256 query rows
    per KV head over several query groups), every task against the oracle."""
    from oracle import probe as oracle
    w = configs.SMALL_BF16.replace(name="small_16_tasks", seed=98)
    T = 16
    kv, params, kv_d, p_d = small_case(w, dev)
    tasks = inputs.task_params(w, T, "cpu")
    probe = binding.Probe(w, max_tasks=T)
    got = probe.forward_multi(kv_d, p_d, tasks["soft_prompts"].to(dev), tasks["w_cls"].to(dev)).cpu().numpy()
    probe.close()
    kvs = [tuple(t.double().numpy() for t in kv.logical_kv(b)) for b in range(w.batch)]
    ref = oracle.probe_batch_tasks(kvs, tasks["soft_prompts"].double().numpy(), tasks["w_cls"].double().numpy(),
                                   None, H.oracle_weights(params), H.head_shape(w))
    for t in range(T):
        H.check_logits(got[:, t], ref[:, t], w.dtype, f"task {t}")


def test_work_list_over_many_sequences(dev):
    """1500 ragged sequences (0-1200 tokens) in 256-token splits: the attention's
    work list then spans two scan blocks of 1024 sequences and ranks 1500 last
    splits; every sequence's logits match the oracle (a split dropped or taken
    twice would change that sequence's)."""
    w = configs.Workload(name="many_seqs_bf16", dtype="bf16", batch=1500, k=2, hidden=256, n_q_heads=4,
                         n_kv_heads=2, head_dim=64, intermediate=512, n_classes=2,
                         seq_len=("uniform", 0, 1200), seed=97)
    announce(f"[work list] {w.name}")
    kv, params, kv_d, p_d = small_case(w, dev)
    probe = binding.Probe(w, split_len=256)
    plan = probe.plan(w.batch)
    assert plan["split_len"] == 256 and plan["max_splits"] == 5
    got = probe.forward(kv_d, p_d).cpu().numpy()
    assert probe.check_device_error() == 0
    probe.close()
    ref = np.stack([o["logits"] for o in H.oracle_outputs(w, kv, params, range(w.batch))])
    err = H.check_logits(got, ref, w.dtype, w.name)
    announce(f"[work list] {w.name}: max err {err:.3e} over {w.batch} sequences")
