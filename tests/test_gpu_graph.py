"""The forwards under HIP graph capture: sp_probe_forward, _multi and _recursive
allocate nothing, synchronise nothing and record no memset, so a captured call
replays.  Every replay, with eager calls of the same handle between replays,
must equal the eager result bit for bit."""
from __future__ import annotations

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


def capture(fn):
    """Warm up on a side stream (as torch requires before capture), then capture fn()."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        fn()
    torch.cuda.synchronize()
    return graph


@pytest.mark.parametrize("mode", ["one", "multi", "recursive"])
def test_forward_replays_in_a_graph(mode, dev):
    w = configs.SMALL_BF16
    print(f"[graph] {w.name} {mode}", flush=True)
    lens = inputs.seq_lens(w)
    kv = inputs.kv_cache(w, lens, "cpu")
    params = inputs.params(w, "cpu")
    kv_d, p_d = H.to_device(kv, params, dev)
    T = 3 if mode == "multi" else 1
    probe = binding.Probe(w, max_tasks=T)
    if mode == "multi":
        tasks = {k: (None if v is None else v.to(dev)) for k, v in inputs.task_params(w, T, "cpu").items()}
        run = lambda out=None: probe.forward_multi(kv_d, p_d, tasks["soft_prompts"], tasks["w_cls"],
                                                   tasks["b_cls"], logits=out)
    elif mode == "recursive":
        fusion = {k: v.to(dev) for k, v in inputs.fusion_params(w, "cpu").items()}
        run = lambda out=None: probe.forward_recursive(kv_d, p_d, fusion, logits=out)
    else:
        run = lambda out=None: probe.forward(kv_d, p_d, logits=out)
    eager = run().clone()
    out = torch.empty_like(eager)
    graph = capture(lambda: run(out))
    for i in range(3):
        out.fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager), f"replay {i} differs from the eager forward"
        again = run()                      # eager work on the same handle between replays
        torch.cuda.synchronize()
        assert torch.equal(again, eager)
    probe.close()
