"""Writes input_sha256.json: SHA-256 of the seeded synthetic inputs each
workload generates on the CPU (context lengths, block table, KV pool, head
weights, soft prompts, classifier, fusion inputs), so that a change in the
generators or in the random streams they draw from shows up as a failing
test rather than as silently different benchmark inputs.  Large workloads hash
everything but the KV pool (the same code draws the small workloads' pools,
which are hashed whole), and of their head matrices only W_q and W_k, no
fusion inputs (the same code draws every matrix).  Calls only paper_2608_28099_amd.inputs (no method
arithmetic).  Run from the repository root:  python tests/golden/make_input_sha256.py
"""
from __future__ import annotations

import hashlib
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "input_sha256.json")
POOL_LIMIT = 64 << 20   # pools up to this many bytes are hashed whole
MATRIX_LIMIT = 16 << 20  # larger head matrices are skipped, except W_q and W_k


def digest(t) -> str:
    import numpy as np
    import torch
    if isinstance(t, np.ndarray):
        b = np.ascontiguousarray(t).tobytes()
    else:
        t = t.detach().contiguous().cpu()
        b = t.view(torch.uint8).numpy().tobytes() if t.dtype != torch.bool else t.numpy().tobytes()
    return hashlib.sha256(b).hexdigest()


def workload_hashes(w) -> dict:
    from paper_2608_28099_amd import inputs
    out = {}
    lens = inputs.seq_lens(w)
    out["seq_lens"] = digest(lens)
    big = w.hidden * w.intermediate * 2 > MATRIX_LIMIT
    skip = ("w_v", "w_o", "w_gate", "w_up", "w_down") if big else ()
    names = [n for n in ("soft_prompt", "in_norm", "w_q", "w_k", "w_v", "w_o", "post_norm", "w_gate", "w_up",
                         "w_down", "final_norm", "w_cls", "b_cls") if n not in skip]
    for name, t in inputs.params(w, "cpu", only=names).items():
        if t is not None:
            out[name] = digest(t)
    if not big:
        for name, t in inputs.fusion_params(w, "cpu").items():
            out["fusion." + name] = digest(t)
    est = int(lens.astype("int64").sum()) * w.n_kv_heads * w.head_dim * 2 * (2 if w.dtype == "bf16" else 4)
    if est <= POOL_LIMIT:
        kv = inputs.kv_cache(w, lens, "cpu")
        out["kv.pool"] = digest(kv.pool)
        if kv.block_table is not None:
            out["kv.block_table"] = digest(kv.block_table)
    return out


def all_workloads():
    from paper_2608_28099_amd import configs
    return {**configs.WORKLOADS, **configs.STRESS}


def main():
    data = {name: workload_hashes(w) for name, w in sorted(all_workloads().items())}
    with open(OUT, "w") as f:
        json.dump(data, f, indent=1, sort_keys=True)
        f.write("\n")
    print(f"wrote {OUT}: {len(data)} workloads")


if __name__ == "__main__":
    main()
