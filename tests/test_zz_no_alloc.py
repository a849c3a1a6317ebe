"""The forward that allocates nothing (sp_probe_forward_noalloc, static device
scratch) against sp_probe_forward on a handle, through the C ABI: two calls in
a row, the second with a smaller input (and a third of another shape, whose
leftover contents the next call must not see), each bit-identical to the
handle's logits and within the oracle's bar; configs too large for the scratch
and the debug / profiling flags are refused before anything is enqueued."""
from __future__ import annotations

import numpy as np
import pytest
import torch

from paper_2608_28099_amd import binding, configs, inputs
from tests import helpers as H

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    binding.load()
    return torch.device("cuda:0")


def noalloc(w, kv_d, p_d, batch, out, max_batch=None):
    cfg = binding.make_config(w, max_batch=max_batch)
    kvs = binding.make_kv(kv_d, batch)
    wt = binding.make_weights(p_d)
    stream = torch.cuda.current_stream().cuda_stream
    return binding.sp_probe_forward_noalloc(cfg, kvs, kv_d.seq_lens.data_ptr(),
                                            None if kv_d.block_table is None else kv_d.block_table.data_ptr(),
                                            p_d["soft_prompt"].data_ptr(), wt, out.data_ptr(), stream)


def test_noalloc_matches_the_handle_forward(dev):
    calls = [(configs.SMALL_G5_BF16, None), (configs.SMALL_G5_BF16, 2), (configs.SMALL_BF16, 3),
             (configs.SMALL_BF16, 1)]
    for w, batch in calls:
        print(f"[noalloc] {w.name} batch {batch}", flush=True)
        lens = inputs.seq_lens(w)
        kv = inputs.kv_cache(w, lens, "cpu")
        params = inputs.params(w, "cpu")
        kv_d, p_d = H.to_device(kv, params, dev)
        B = w.batch if batch is None else batch
        cfg = binding.make_config(w)
        assert binding.sp_probe_plan_config(cfg, 256)["workspace_bytes"] <= 64 << 20
        out = torch.full((B, w.n_classes), float("nan"), device=dev)
        assert noalloc(w, kv_d, p_d, B, out) == 0
        probe = binding.Probe(w)
        ref_gpu = probe.forward(kv_d, p_d, batch=B).clone()
        probe.close()
        torch.cuda.synchronize()
        assert torch.equal(out, ref_gpu), w.name
        ref = np.stack([o["logits"] for o in H.oracle_outputs(w, kv, params, range(B))])
        H.check_logits(out.cpu().numpy(), ref, w.dtype, f"noalloc {w.name} B={B}")


def test_noalloc_refusals(dev):
    w = configs.SMALL_BF16
    lens = inputs.seq_lens(w)
    kv_d, p_d = H.to_device(inputs.kv_cache(w, lens, "cpu"), inputs.params(w, "cpu"), dev)
    out = torch.full((w.batch, w.n_classes), 7.0, device=dev)
    big = configs.QWEN9B_BF16
    cfg = binding.make_config(big)
    assert binding.sp_probe_plan_config(cfg, 256)["workspace_bytes"] > 64 << 20
    lib = binding.load()
    kvs = binding.make_kv(kv_d)
    wt = binding.make_weights(p_d)
    s = torch.cuda.current_stream().cuda_stream
    args = (kv_d.seq_lens.data_ptr(), kv_d.block_table.data_ptr(), p_d["soft_prompt"].data_ptr())
    assert binding.sp_probe_forward_noalloc(cfg, kvs, *args, wt, out.data_ptr(), s) == -6
    for flag in (binding.SP_FLAG_DEBUG, binding.SP_FLAG_PROFILE):
        cfg = binding.make_config(w, flags=flag)
        assert binding.sp_probe_forward_noalloc(cfg, kvs, *args, wt, out.data_ptr(), s) == -2
    assert lib.sp_probe_forward_noalloc(None, None, None, None, None, None, None, None) == -1
    torch.cuda.synchronize()
    assert torch.all(out == 7.0)
