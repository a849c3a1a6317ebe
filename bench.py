"""Benchmark of the Speculative Probing classification forward on one MI355X.

One step = one sp_probe_forward over the whole batch of the workload (soft-row
prep, split attention over the paged KV cache, merge, o-projection, norm,
SwiGLU MLP, final norm and classifier), inputs already resident in HBM; the
head's projections read its fp16 weight image, made once before timing (the
head is frozen).  --mode recursive: one step = one sp_probe_forward_recursive
(recursive SP-k with the MTP input fusion: k single-row passes of the head,
each reading the whole cache once) on the recursive workload.

Three timed passes, each after its own warm-up:
  1. the contract's: exactly --steps steps bracketed by device synchronisation
     on a handle without profiling -> value (classifications/s) and ms_per_step;
  2. max(50, --steps) steps, each bracketed by HIP events on the launch stream
     -> median, p10 and p90 per-step times;
  3. --steps steps on a handle with per-stage HIP events -> the stage times and
     the roofline of the attention stage (split kernel + merge, the two
     attention kernels) and of the split kernel alone.
KV caches under 1 GB are rotated over enough copies to exceed 1 GB, so that no
step finds the previous step's KV in the caches.

Prints one JSON line: the contract fields, roofline (algorithmic KV bytes per
attention stage / its mean duration, against 8 TB/s and against the device's
measured streaming-read rate), cpu_baseline (the fp64 oracle on the host cores
over a bounded sample of the same workload's sequences).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "classifications/sec at 1 MI355X; attention KV-read GB/s as % of HBM peak"
HBM_PEAK_GBPS = 8000.0
MFMA_PEAK_TFLOPS = 2500.0   # dense fp16 / bf16 matrix-core peak
DEFAULT_WORKLOAD = {"one-pass": "long_9b_bf16", "recursive": "long_9b_bf16_sp5"}
DTYPE_LABEL = {"bf16": "bf16 storage; fp16xfp16->fp32 MFMA projections (fp16 image of the bf16 weights); "
                       "attention on the stored bf16 K/V: bf16 MFMA with hi+lo bf16 queries and probabilities "
                       "up to 6 query tiles per KV head, fp16 MFMA (K/V converted in LDS) from 7; soft keys as "
                       "hi+lo bf16 MFMA products; fp32 softmax, norms, residual stream and logits",
               "f32": "f32"}
ROTATE_BELOW = 1 << 30      # KV caches smaller than this are rotated over copies
ATTN_SRCS = [os.path.join(ROOT, "paper_2608_28099_amd", "csrc", f) for f in ("attention.hip", "merge.hip")]
PROFILES = os.path.join(ROOT, "profiles")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--mode", choices=("one-pass", "recursive"), default="one-pass")
    ap.add_argument("--workload", default=None)
    ap.add_argument("--tasks", type=int, default=1,
                    help="one-pass mode: monitoring tasks sharing the cache in one call")
    ap.add_argument("--last-row-only", action="store_true",
                    help="one-pass mode: run only the rows the LAST read-out uses past the attention")
    ap.add_argument("--split-len", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="oracle sample: sequences are timed until this much CPU time has passed")
    ap.add_argument("--library-gemm", action="store_true",
                    help="also time the vendor library's GEMM (torch.matmul, fp16) on the projection shapes")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="run only a plain 1 GiB device copy (HBM counter calibration)")
    return ap.parse_args()


def attention_source_hash() -> str:
    h = hashlib.sha256()
    for f in ATTN_SRCS:
        h.update(open(f, "rb").read())
    return h.hexdigest()[:16]


def traffic_per_launch(workload: str):
    """HBM bytes per attention stage (split kernel + merge) from committed
    counter runs on this workload, if they were taken on the current attention
    and merge sources; else None."""
    try:
        rec = json.load(open(os.path.join(PROFILES, f"attention_{workload}_traffic.json")))
    except (OSError, ValueError):
        return None
    if rec.get("attention_src_sha256_16") != attention_source_hash():
        return None
    return rec.get("hbm_bytes_per_stage")


def projection_rates(w, T, args, recursive, stages, n_fwd, mfma_peak):
    """Achieved MFMA throughput of the projection stages (their algorithmic FLOP
    over the stage's mean HIP-event time per forward) against the dense peak
    and against the rate this device's matrix cores sustain (mfma_peak)."""
    d, I, qkv = w.hidden, w.intermediate, (w.n_q_heads + 2 * w.n_kv_heads) * w.head_dim
    qw = w.n_q_heads * w.head_dim
    if recursive:   # k steps of B rows each (the fusion's B x d x d product is in soft prep)
        rows = w.batch * w.k
    else:
        rows = w.batch * T * (1 if args.last_row_only else w.k)
    flop = {"o_proj": 2.0 * rows * d * qw, "gate_up": 2.0 * rows * 2 * I * d, "down": 2.0 * rows * d * I}
    out = {}
    for name, f in flop.items():
        ms = stages[name] / n_fwd
        tf = f / (ms * 1e-3) / 1e12
        out[name] = {"gflop": round(f / 1e9, 2), "ms": round(ms, 4), "tflops": round(tf, 1),
                     "frac_of_peak": round(tf / MFMA_PEAK_TFLOPS, 4),
                     "frac_of_measured_mfma_peak": round(tf / mfma_peak, 4)}
    out["measured_mfma_peak_tflops"] = round(mfma_peak, 1)
    return out


def library_gemm_ms(torch, dev, w, rows):
    """The vendor library's GEMM (torch.matmul on fp16 operands, fp16 output,
    no fused epilogue) on the projection shapes of `rows` rows, for context
    only: the forward never calls it.  Median of 10 launches, each after a
    512 MiB write that evicts the caches, as the forward's weights are
    evicted between uses."""
    d, I, qw = w.hidden, w.intermediate, w.n_q_heads * w.head_dim
    shapes = {"o_proj": (rows, d, qw), "gate_up": (rows, 2 * I, d), "down": (rows, d, I)}
    junk = torch.empty(128 << 20, dtype=torch.float32, device=dev)
    out = {}
    for name, (m, n, k) in shapes.items():
        a = torch.randn(m, k, device=dev, dtype=torch.float16)
        b = torch.randn(n, k, device=dev, dtype=torch.float16) * 0.05
        bt = b.t()
        c = torch.matmul(a, bt)
        times = []
        for _ in range(10):
            junk.add_(1.0)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            torch.matmul(a, bt, out=c)
            e1.record()
            e1.synchronize()
            times.append(e0.elapsed_time(e1))
        times.sort()
        ms = (times[4] + times[5]) / 2
        out[name] = {"ms": round(ms, 4), "tflops": round(2.0 * m * n * k / (ms * 1e-3) / 1e12, 1)}
        del a, b, bt, c
    del junk
    return out


def copy_rate(torch, dev):
    """Device-to-device copy of 1 GiB (bytes read + written per second): the
    streaming rate HBM sustains for a plain copy on this machine, for context."""
    n = 1 << 30
    src = torch.empty(n, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(5):
        dst.copy_(src)
    b.record()
    torch.cuda.synchronize()
    rate = 5 * 2 * n / (a.elapsed_time(b) * 1e-3) / 1e9
    del src, dst
    return round(rate, 1)


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, kv, params, seconds: float, fusion=None, tasks=None):
    """The oracle, as written, timed on the host over whole sequences of the
    workload (the recursive oracle when fusion inputs are given; every task's
    probe per sequence when tasks are given)."""
    import numpy as np
    import threadpoolctl

    from oracle import probe as oracle
    W = {k: (None if v is None else v.double().cpu().numpy()) for k, v in params.items() if k != "soft_prompt"}
    if fusion is not None:
        W.update({"fc_norm_h": fusion["fc_norm_hidden"].double().cpu().numpy(),
                  "fc_norm_e": fusion["fc_norm_embed"].double().cpu().numpy(),
                  "w_fc": fusion["w_fc"].double().cpu().numpy()})
        h_last = fusion["hidden_last"].double().cpu().numpy()
    soft = params["soft_prompt"].double().cpu().numpy()
    shape = oracle.HeadShape(w.n_q_heads, w.n_kv_heads, w.head_dim, w.rms_eps, w.rope_base, w.pool)
    threads = max((i.get("num_threads", 1) for i in threadpoolctl.threadpool_info()), default=1)
    done, spent, toks = 0, 0.0, 0
    for b in range(w.batch):
        k, v = kv.logical_kv(b)
        k, v = k.double().cpu().numpy(), v.double().cpu().numpy()
        t = time.perf_counter()
        if fusion is not None:
            oracle.probe_sequence_recursive(k, v, soft, h_last[b], W, shape)
        elif tasks is not None:
            f = lambda x: None if x is None else x.double().cpu().numpy()
            oracle.probe_batch_tasks([(k, v)], f(tasks["soft_prompts"]), f(tasks["w_cls"]),
                                     f(tasks["b_cls"]), W, shape)
        else:
            oracle.probe_sequence(k, v, soft, W, shape)
        spent += time.perf_counter() - t
        done += 1
        toks += k.shape[1]
        del k, v
        if spent >= seconds:
            break
    n_tasks = 1 if tasks is None else tasks["soft_prompts"].shape[0]
    return {"value": done * n_tasks / spent, "unit": "classifications/s", "cores": threads, "kind": "oracle",
            "cpu": cpu_model(),
            "sample": f"{done} of {w.batch} sequences ({toks} context tokens) x {n_tasks} task(s), "
                      f"fp64 numpy, {spent:.1f} s"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the forward is independent "
              "per sequence and would shard by sequence, but only the one-GPU path exists.",
              file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    from paper_2608_28099_amd import binding, configs, inputs

    dev = torch.device("cuda:0")
    if args.calibrate_copy:
        n = 1 << 30
        src = torch.ones(n, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibration": "device copy", "bytes_read": n, "bytes_written": n, "launches": 3}))
        return

    recursive = args.mode == "recursive"
    name = args.workload or DEFAULT_WORKLOAD[args.mode]
    w = configs.WORKLOADS.get(name) or configs.STRESS.get(name) or configs.RECURSIVE[name]
    print(f"[bench] {w.name}: generating inputs on the GPU", file=sys.stderr, flush=True)
    lens = inputs.seq_lens(w)
    kv = inputs.kv_cache(w, lens, dev)
    params = inputs.params(w, dev)
    fusion = inputs.fusion_params(w, dev) if recursive else None
    T = 1 if recursive else args.tasks
    tasks = inputs.task_params(w, T, dev) if T > 1 else None
    logits = torch.empty((w.batch, T, w.n_classes), dtype=torch.float32, device=dev)
    flags = binding.SP_FLAG_LAST_ROW_ONLY if args.last_row_only else 0
    # the frozen head's fp16 image, made once (bf16 storage)
    run_params = dict(params)
    if w.dtype == "bf16":
        run_params["packed"] = binding.pack_weights(w, params, max_tasks=T)
    # KV copies so that the KV the steps read, rotated, exceeds ROTATE_BELOW bytes
    esz = 2 if w.dtype == "bf16" else 4
    kv_bytes = int(lens.astype("int64").sum()) * w.n_kv_heads * w.head_dim * 2 * esz
    n_rot = 1 if kv_bytes >= ROTATE_BELOW else min(64, -(-ROTATE_BELOW // max(kv_bytes, 1)) + 1)
    kvs = [kv] + [inputs.KVCache(kv.pool.clone(), kv.block_table, kv.seq_lens, kv.block_size,
                                 kv.max_blocks_per_seq, kv.n_kv, kv.head_dim) for _ in range(n_rot - 1)]
    plain = binding.Probe(w, split_len=args.split_len, flags=flags, max_tasks=T)
    prof = binding.Probe(w, split_len=args.split_len, flags=flags | binding.SP_FLAG_PROFILE, max_tasks=T)
    torch.cuda.synchronize()

    def step(probe, i):
        kvi = kvs[i % n_rot]
        if recursive:
            probe.forward_recursive(kvi, run_params, fusion, logits)
        elif tasks is not None:
            probe.forward_multi(kvi, run_params, tasks["soft_prompts"], tasks["w_cls"], tasks["b_cls"], logits)
        else:
            probe.forward(kvi, run_params, logits)

    # 1. the contract's timed region
    for i in range(args.warmup):
        step(plain, i)
    torch.cuda.synchronize()
    print(f"[bench] timing {args.steps} steps", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(plain, i)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_per_step = 1000.0 * elapsed / args.steps
    assert bool(torch.isfinite(logits).all()), "non-finite logits"
    assert plain.check_device_error() == 0, "device-side status after the timed steps"

    # 2. per-step HIP events on the launch stream
    n_dist = max(50, args.steps)
    stream = torch.cuda.current_stream(dev)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n_dist)]
    for i in range(n_dist):
        evs[i][0].record(stream)
        step(plain, i)
        evs[i][1].record(stream)
    torch.cuda.synchronize()
    per_step = np.array([a.elapsed_time(b) for a, b in evs])
    dist = {"steps": n_dist, "median_ms": round(float(np.median(per_step)), 4),
            "p10_ms": round(float(np.percentile(per_step, 10)), 4),
            "p90_ms": round(float(np.percentile(per_step, 90)), 4),
            "value_at_median": round(w.batch * T / (float(np.median(per_step)) * 1e-3), 1)}

    # 3. per-stage events
    for i in range(args.warmup):
        step(prof, i)
    torch.cuda.synchronize()
    prof.profile_read()  # discard warm-up events
    for i in range(args.steps):
        step(prof, i)
    torch.cuda.synchronize()
    stages, n_fwd = prof.profile_read()   # the event pool keeps the last forwards that fit (all of them here)
    assert 0 < n_fwd <= args.steps

    launches = w.k if recursive else 1   # attention launches per step
    attn_ms = stages["attention"] / (n_fwd * launches)
    stage_ms = (stages["attention"] + stages["merge"]) / (n_fwd * launches)
    achieved = kv_bytes / (stage_ms * 1e-3) / 1e9
    achieved_k1 = kv_bytes / (attn_ms * 1e-3) / 1e9
    # streaming-read ceiling of this device, over a 4 GiB buffer
    buf = torch.empty(1 << 32, dtype=torch.uint8, device=dev)
    buf.fill_(1)
    read_peak = binding.measure_read_gbps(buf, reps=10)
    del buf
    # counters are taken per launch shape: the workload, its task count and row pruning
    variant = w.name + (f"_tasks{T}" if T > 1 else "") + ("_last_row_only" if args.last_row_only else "")
    traffic = traffic_per_launch(variant)
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": traffic,
                "kernel": ("attn_split_bf16 + merge_splits" if w.dtype == "bf16" else "attn_split_f32 + merge_splits"),
                "algorithmic_bytes_per_launch": kv_bytes, "mean_launch_ms": round(stage_ms, 4),
                "measured_read_peak_gbps": round(read_peak, 1),
                "frac_of_measured_read_peak": round(achieved / read_peak, 4),
                "split_kernel_only": {"mean_launch_ms": round(attn_ms, 4), "achieved": round(achieved_k1, 1),
                                      "frac": round(achieved_k1 / HBM_PEAK_GBPS, 4)}}
    plan = plain.plan_recursive(w.batch) if recursive else plain.plan(w.batch)
    out = {
        "metric": (METRIC if not recursive else "recursive SP-k classifications/sec at 1 MI355X"),
        "value": round(w.batch * T / (ms_per_step * 1e-3), 1), "unit": "classifications/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": DTYPE_LABEL[w.dtype],
        "data": f"synthetic (seeded; random-init head weights; {w.layout} KV ~N(0,1))",
        "config": {"workload": w.name, "batch": w.batch, "seq_len": list(w.seq_len), "k": w.k,
                   "hidden": w.hidden, "n_q_heads": w.n_q_heads, "n_kv_heads": w.n_kv_heads,
                   "head_dim": w.head_dim, "intermediate": w.intermediate, "n_classes": w.n_classes,
                   "kv_layout": w.layout, "block_size": kv.block_size, "kv_bytes": kv_bytes,
                   "kv_copies_rotated": n_rot, "weights": ("fp16 image" if "packed" in run_params else "as stored"),
                   "split_len": plan["split_len"], "parallelism": "single GPU",
                   "mode": args.mode, "attention_launches_per_step": launches, "tasks": T,
                   "last_row_only": bool(args.last_row_only)},
        "step_time_distribution": dist,
        "roofline": roofline,
        "attention_gbps": round(achieved, 1),
        "stages_ms": {k: round(v / n_fwd, 4) for k, v in stages.items()},
        "projections": projection_rates(w, T, args, recursive, stages, n_fwd, binding.measure_mfma_tflops(dev)),
        "hbm_copy_gbps": copy_rate(torch, dev),
    }
    if args.library_gemm:
        # the recursive form runs k launches of B rows each; the one-pass form one launch
        rows, launches_per_fwd = (w.batch, w.k) if recursive else (w.batch * T * (1 if args.last_row_only else w.k), 1)
        lib = library_gemm_ms(torch, dev, w, rows)
        for name, r in lib.items():
            r["ms"] = round(r["ms"] * launches_per_fwd, 4)
            r["launches_per_forward"] = launches_per_fwd
            r["ours_over_library_time"] = round(out["projections"][name]["ms"] / r["ms"], 3)
        out["projections"]["library_gemm_fp16"] = lib
    plain.close()
    prof.close()
    if not args.no_cpu_baseline:
        print("[bench] timing the oracle on the host", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(w, kv, params, args.cpu_seconds, fusion, tasks)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
