"""GPU tests of the fp16 weight image, the status word, the workspace guards and
the long split whose block-id windows are re-loaded, through the C ABI.

- The image (sp_probe_pack_weights) holds the same values the projections
  otherwise convert per fragment, so every forward returns the same logits
  bit for bit with and without it, and both match the oracle.
- A seq_len past max_seq_len is clamped and reported in any mode; an fp16
  activation out of range is reported as SP_ERR_RANGE.
- Guard words between workspace areas and canary words around the caller's
  logits stay intact over successful forwards.
"""
from __future__ import annotations

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


def case(w, dev):
    lens = inputs.seq_lens(w)
    kv = inputs.kv_cache(w, lens, "cpu")
    params = inputs.params(w, "cpu")
    kv_d, p_d = H.to_device(kv, params, dev)
    return kv, params, kv_d, p_d


@pytest.mark.parametrize("w", [configs.SMALL_BF16, configs.SMALL_G5_BF16], ids=lambda w: w.name)
def test_image_gives_identical_logits(w, dev):
    print(f"[image] {w.name}", flush=True)
    kv, params, kv_d, p_d = case(w, dev)
    img = binding.pack_weights(w, p_d)
    probe = binding.Probe(w)
    plain = probe.forward(kv_d, p_d).clone()
    packed = probe.forward(kv_d, dict(p_d, packed=img)).clone()
    # the image replaces the seven matrices: the forward must not read them
    nulls = {n: None for n in ("w_q", "w_k", "w_v", "w_o", "w_gate", "w_up", "w_down")}
    packed_only = probe.forward(kv_d, dict(p_d, packed=img, **nulls)).clone()
    torch.cuda.synchronize()
    assert torch.equal(plain, packed) and torch.equal(plain, packed_only)
    ref = np.stack([o["logits"] for o in H.oracle_outputs(w, kv, params, range(w.batch))])
    H.check_logits(packed.cpu().numpy(), ref, w.dtype, "with the image")
    assert probe.check_device_error() == 0
    probe.close()


def test_image_in_multi_task_and_recursive_forwards(dev):
    w = configs.SMALL_BF16_SP5
    kv, params, kv_d, p_d = case(w, dev)
    fusion = {k: v.to(dev) for k, v in inputs.fusion_params(w, "cpu").items()}
    tasks = {k: (None if v is None else v.to(dev)) for k, v in inputs.task_params(w, 3, "cpu").items()}
    img = binding.pack_weights(w, p_d)
    probe = binding.Probe(w, max_tasks=3)
    a = probe.forward_recursive(kv_d, p_d, fusion).clone()
    b = probe.forward_recursive(kv_d, dict(p_d, packed=img), fusion).clone()
    c = probe.forward_multi(kv_d, p_d, tasks["soft_prompts"], tasks["w_cls"], tasks["b_cls"]).clone()
    d = probe.forward_multi(kv_d, dict(p_d, packed=img), tasks["soft_prompts"], tasks["w_cls"],
                            tasks["b_cls"]).clone()
    torch.cuda.synchronize()
    assert torch.equal(a, b) and torch.equal(c, d)
    ref = np.stack([o["logits"] for o in H.oracle_outputs_recursive(w, kv, params, fusion, range(w.batch))])
    H.check_logits(b.cpu().numpy(), ref, w.dtype, "recursive with the image")
    probe.close()


def test_image_header_is_checked_in_debug_mode(dev):
    """An image of another shape fails the debug-mode header check: the forward
    skips its work and reports SP_ERR_DEVICE_DATA."""
    w = configs.SMALL_BF16
    kv, params, kv_d, p_d = case(w, dev)
    other = w.replace(name="other", intermediate=1024)
    p_other = H.to_device(kv, inputs.params(other, "cpu"), dev)[1]
    img_other = binding.pack_weights(other, p_other)
    probe = binding.Probe(w, flags=binding.SP_FLAG_DEBUG)
    out = torch.full((w.batch, w.n_classes), 5.0, device=dev)
    probe.forward(kv_d, dict(p_d, packed=img_other), out)
    assert probe.check_device_error() == binding.SP_ERR_DEVICE_DATA
    assert torch.all(out == 5.0)
    img = binding.pack_weights(w, p_d)
    probe.forward(kv_d, dict(p_d, packed=img), out)
    assert probe.check_device_error() == 0
    probe.close()


def test_pack_rejects_bad_arguments(dev):
    w = configs.SMALL_BF16
    _, _, _, p_d = case(w, dev)
    cfg = binding.make_config(w)
    n = binding.sp_probe_packed_bytes(cfg)
    img = torch.empty(n, dtype=torch.uint8, device=dev)
    s = torch.cuda.current_stream().cuda_stream
    wt = binding.make_weights(p_d)
    assert binding.sp_probe_pack_weights(cfg, wt, img.data_ptr(), n - 1, s) == -1
    assert binding.sp_probe_pack_weights(cfg, wt, img.data_ptr() + 8, n - 8, s) == -1
    wt.w_up = None
    assert binding.sp_probe_pack_weights(cfg, wt, img.data_ptr(), n, s) == -1


def test_seq_len_past_max_is_clamped_and_reported(dev):
    """Outside debug mode a seq_len past max_seq_len is clamped: the sequence is
    classified on its first max_seq_len tokens (checked against the oracle on
    that prefix) and sp_probe_check_device_error reports SP_ERR_DEVICE_DATA
    once; a clean forward then reports SP_OK."""
    w = configs.SMALL_BF16
    kv, params, kv_d, p_d = case(w, dev)
    cap = 100
    probe = binding.Probe(w, max_seq_len=cap)
    got = probe.forward(kv_d, p_d).cpu().numpy()
    assert probe.check_device_error() == binding.SP_ERR_DEVICE_DATA
    assert probe.check_device_error() == 0
    W = H.oracle_weights(params)
    soft = params["soft_prompt"].double().numpy()
    ref = []
    for b in range(w.batch):
        k, v = kv.logical_kv(b)
        k, v = k.double().numpy()[:, :cap], v.double().numpy()[:, :cap]
        ref.append(oracle.probe_sequence(k, v, soft, W, H.head_shape(w))["logits"])
    H.check_logits(got, np.stack(ref), w.dtype, "clamped")
    lens = kv_d.seq_lens.clamp(max=cap)
    kvc = inputs.KVCache(kv_d.pool, kv_d.block_table, lens, kv_d.block_size, kv_d.max_blocks_per_seq,
                         kv_d.n_kv, kv_d.head_dim)
    again = probe.forward(kvc, p_d).cpu().numpy()
    assert probe.check_device_error() == 0
    assert np.array_equal(again, got)
    probe.close()


def test_swiglu_past_fp16_range_is_reported(dev):
    """Gate and up weights scaled so that SwiGLU products exceed 65504: the fp16
    activation is out of range and the forward reports SP_ERR_RANGE (the
    documented limit of SP_BF16); the unscaled head reports SP_OK."""
    w = configs.SMALL_BF16
    kv, params, kv_d, p_d = case(w, dev)
    probe = binding.Probe(w)
    probe.forward(kv_d, p_d)
    assert probe.check_device_error() == 0
    big = dict(p_d, w_gate=(p_d["w_gate"].float() * 400).to(torch.bfloat16),
               w_up=(p_d["w_up"].float() * 400).to(torch.bfloat16))
    # the product really leaves fp16's range (checked on the host from the oracle's SwiGLU input)
    Wb = H.oracle_weights({k: (None if v is None else v.cpu()) for k, v in big.items()})
    k0, v0 = kv.logical_kv(4)
    o = oracle.probe_sequence(k0.double().numpy(), v0.double().numpy(), params["soft_prompt"].double().numpy(),
                              Wb, H.head_shape(w))
    assert np.max(np.abs(o["s"])) > 65504
    probe.forward(kv_d, big)
    assert probe.check_device_error() == binding.SP_ERR_RANGE
    img = binding.pack_weights(w, big)
    probe.forward(kv_d, dict(big, packed=img))
    assert probe.check_device_error() == binding.SP_ERR_RANGE
    probe.forward(kv_d, p_d)
    assert probe.check_device_error() == 0
    probe.close()


def test_guards_and_logit_canaries_survive_forwards(dev):
    """Canary words on both sides of the logits and the workspace's own guard
    words stay intact over one-pass, multi-task, recursive and last-row-only
    forwards at the handle's largest sizes."""
    w = configs.SMALL_G5_BF16
    kv, params, kv_d, p_d = case(w, dev)
    fusion = {k: v.to(dev) for k, v in inputs.fusion_params(w, "cpu").items()}
    T = 3
    tasks = {k: (None if v is None else v.to(dev)) for k, v in inputs.task_params(w, T, "cpu").items()}
    canary = -7.0e37
    pad = 64
    for flags in (0, binding.SP_FLAG_LAST_ROW_ONLY):
        ww = w.replace(pool="last") if flags else w
        probe = binding.Probe(ww, max_tasks=T, flags=flags)
        for name in ("one-pass", "multi", "recursive"):
            n = w.batch * (T if name == "multi" else 1) * w.n_classes
            buf = torch.full((n + 2 * pad,), canary, dtype=torch.float32, device=dev)
            out = buf[pad:pad + n]
            if name == "one-pass":
                probe.forward(kv_d, p_d, out.view(w.batch, w.n_classes))
            elif name == "multi":
                probe.forward_multi(kv_d, p_d, tasks["soft_prompts"], tasks["w_cls"], tasks["b_cls"],
                                    out.view(w.batch, T, w.n_classes))
            elif not flags:
                probe.forward_recursive(kv_d, p_d, fusion, out.view(w.batch, w.n_classes))
            else:
                continue
            torch.cuda.synchronize()
            assert torch.all(buf[:pad] == canary) and torch.all(buf[pad + n:] == canary), name
            assert torch.isfinite(out).all(), name
            assert probe.check_device_error() == 0, (flags, name)
        probe.close()


def test_long_split_reloads_block_id_windows(dev):
    """One paged sequence of 40,000 tokens in 16-token blocks with 32,768-token
    splits: the first split spans 2048 blocks, so the attention re-loads its
    block-id window three times (windows 0-3) and the second split ends in a
    ragged tail.  The attention output (SP_TAP_ATTN) matches the oracle's
    element by element, and so do the logits."""
    w = configs.Workload(name="long_window_bf16", dtype="bf16", batch=2, k=4, hidden=256, n_q_heads=8,
                         n_kv_heads=2, head_dim=128, intermediate=512, n_classes=2,
                         seq_len=("list", (40000, 33001)), layout="paged", seed=71)
    kv, params, kv_d, p_d = case(w, dev)
    probe = binding.Probe(w, split_len=32768)
    plan = probe.plan(w.batch)
    assert plan["split_len"] == 32768 and plan["max_splits"] == 2
    got = probe.forward(kv_d, p_d).cpu().numpy()
    attn = probe.tap(binding.SP_TAP_ATTN, w.batch, dev).view(torch.float16).cpu().double().numpy()
    probe.close()
    outs = H.oracle_outputs(w, kv, params, range(w.batch))
    ref = np.stack([o["logits"] for o in outs])
    H.check_logits(got, ref, w.dtype, "logits")
    qw = w.n_q_heads * w.head_dim
    attn = attn.reshape(-1, qw)[: w.batch * w.k].reshape(w.batch, w.k, qw)
    for b in range(w.batch):
        o_ref = outs[b]["o"].reshape(w.k, qw)
        scale = np.max(np.abs(o_ref))
        err = np.max(np.abs(attn[b] - o_ref)) / scale
        assert err < 1e-2, (b, err)
