"""GPU parity of the head and input variants against the fp64 oracle, through the
C ABI: the frozen-LM-head yes/no read-out (Sec. 6.7, Table 7: the classifier
reads rows of a vocabulary matrix) for the one-pass, multi-task and recursive
forwards, and the Eagle3 input of the recursive form (Sec. 3.1: the first
hidden state projected from three base-model hidden states)."""
from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import probe as oracle
from paper_2608_28099_amd import binding, configs, inputs
from tests import helpers as H

pytestmark = pytest.mark.gpu

VOCAB = 1000


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    binding.load()
    return torch.device("cuda:0")


def announce(msg):
    print(msg, flush=True)


def base(w, dev):
    lens = inputs.seq_lens(w)
    kv = inputs.kv_cache(w, lens, "cpu")
    params = inputs.params(w, "cpu")
    kv_d, p_d = H.to_device(kv, params, dev)
    return kv, params, kv_d, p_d


def kv_list(kv, B):
    return [tuple(t.double().numpy() for t in kv.logical_kv(b)) for b in range(B)]


@pytest.mark.parametrize("w", [configs.TINY_RAGGED_F32, configs.SMALL_BF16, configs.SMALL_G5_BF16],
                         ids=lambda w: w.name)
def test_lm_head_readout_one_pass(w, dev):
    announce(f"[lm head] {w.name}")
    kv, params, kv_d, p_d = base(w, dev)
    lm = inputs.lm_head_params(w, VOCAB, 1, "cpu")
    probe = binding.Probe(w)
    pd = dict(p_d, w_cls=lm["lm_head"].to(dev), cls_rows=lm["cls_rows"][0].contiguous().to(dev))
    got = probe.forward(kv_d, pd).cpu().numpy()
    probe.close()
    W = H.oracle_weights(params)
    W.update(w_cls=lm["lm_head"].double().numpy(), cls_rows=lm["cls_rows"][0].numpy())
    ref = oracle.probe_batch(kv_list(kv, w.batch), params["soft_prompt"].double().numpy(), W, H.head_shape(w))
    err = H.check_logits(got, ref, w.dtype, w.name)
    announce(f"[lm head] {w.name}: max err {err:.3e}")


def test_lm_head_readout_tasks_and_recursive(dev):
    w = configs.SMALL_BF16_SP5
    kv, params, kv_d, p_d = base(w, dev)
    lm = inputs.lm_head_params(w, VOCAB, 2, "cpu")
    head_d, rows_d = lm["lm_head"].to(dev), lm["cls_rows"].to(dev)
    tasks = inputs.task_params(w, 2, "cpu")
    fusion = inputs.fusion_params(w, "cpu")
    probe = binding.Probe(w, max_tasks=2)
    got_t = probe.forward_multi(kv_d, p_d, tasks["soft_prompts"].to(dev), head_d, None,
                                cls_rows=rows_d).cpu().numpy()
    f_d = {k: v.to(dev) for k, v in fusion.items()}
    got_r = probe.forward_recursive(kv_d, dict(p_d, w_cls=head_d, cls_rows=rows_d[0].contiguous()), f_d).cpu().numpy()
    probe.close()
    W = H.oracle_weights(params)
    kvs = kv_list(kv, w.batch)
    ref_t = oracle.probe_batch_tasks(kvs, tasks["soft_prompts"].double().numpy(), lm["lm_head"].double().numpy(),
                                     None, W, H.head_shape(w), cls_rows=lm["cls_rows"].numpy())
    for t in range(2):
        H.check_logits(got_t[:, t], ref_t[:, t], w.dtype, f"tasks, task {t}")
    Wr = H.oracle_weights_recursive(params, fusion)
    Wr.update(w_cls=lm["lm_head"].double().numpy(), cls_rows=lm["cls_rows"][0].numpy())
    ref_r = np.stack([o["logits"] for o in H.oracle_outputs_recursive(w, kv, params, fusion, range(w.batch), W=Wr)])
    err = H.check_logits(got_r, ref_r, w.dtype, "recursive")
    announce(f"[lm head] recursive: max err {err:.3e}")


def test_lm_head_rows_checked_in_debug_mode(dev):
    """A label row outside the vocabulary is reported (SP_ERR_DEVICE_DATA) and the
    classifier reads nothing; the next valid forward is clean."""
    w = configs.SMALL_BF16
    kv, params, kv_d, p_d = base(w, dev)
    lm = inputs.lm_head_params(w, VOCAB, 1, "cpu")
    head_d = lm["lm_head"].to(dev)
    probe = binding.Probe(w, flags=binding.SP_FLAG_DEBUG)
    bad = torch.tensor([3, VOCAB + 5000], dtype=torch.int32, device=dev)
    out = torch.full((w.batch, w.n_classes), 9.0, device=dev)
    probe.forward(kv_d, dict(p_d, w_cls=head_d, cls_rows=bad, cls_vocab=VOCAB), out)
    assert probe.check_device_error() == -7
    assert torch.all(out == 9.0)
    good = lm["cls_rows"][0].contiguous().to(dev)
    probe.forward(kv_d, dict(p_d, w_cls=head_d, cls_rows=good), out)
    assert probe.check_device_error() == 0
    assert torch.all(torch.isfinite(out))
    probe.close()


@pytest.mark.parametrize("w", [configs.TINY_F32_SP2, configs.SMALL_BF16_SP5, configs.SMALL_G5_BF16_SP2],
                         ids=lambda w: w.name)
def test_eagle3_input(w, dev):
    """The first hidden state projected from three hidden states, some entries of
    which exceed fp16's range (the bf16 path stages them with row scales)."""
    announce(f"[eagle3] {w.name}")
    kv, params, kv_d, p_d = base(w, dev)
    fusion = inputs.fusion_params(w, "cpu")
    e3 = inputs.eagle3_params(w, "cpu")
    f_d = {k: v.to(dev) for k, v in fusion.items()}
    f_d.update(hidden_last=e3["hidden3"].to(dev), w_hidden_fuse=e3["w_hidden_fuse"].to(dev))
    probe = binding.Probe(w)
    got = probe.forward_recursive(kv_d, p_d, f_d).cpu().numpy()
    probe.close()
    W = H.oracle_weights_recursive(params, fusion)
    W["w_hidden_fuse"] = e3["w_hidden_fuse"].double().numpy()
    fus = dict(fusion, hidden_last=e3["hidden3"])
    ref = np.stack([o["logits"] for o in H.oracle_outputs_recursive(w, kv, params, fus, range(w.batch), W=W)])
    err = H.check_logits(got, ref, w.dtype, w.name)
    announce(f"[eagle3] {w.name}: max err {err:.3e}")
