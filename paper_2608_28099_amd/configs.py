"""Workload definitions for the Speculative Probing classification forward.

Each workload fixes the shape of the frozen one-decoder-layer speculative head
(hidden width, query / KV heads, head width, SwiGLU width), the number k of
soft-prompt positions appended after every sequence (Sec. 3.2), the number of
classes of the linear head, the batch, the context-length distribution and the
storage of the head's resident KV cache (Sec. 3.3, Eq. 1-3).  The paper gives
the hidden widths of the Qwen3.5 heads (Sec. 5.1) and k in {1, 2, 5}
(Sec. 6.6); the remaining shape fields and the value distributions are the
synthetic stand-ins for the paper's models and datasets, whose weights and
records are not available.

Nothing here computes any part of the method.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field


@dataclass(frozen=True)
class Workload:
    name: str
    dtype: str                 # "f32" or "bf16": storage type of weights, soft prompt and KV cache
    batch: int
    k: int                     # soft-prompt positions appended per sequence
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    intermediate: int
    n_classes: int
    seq_len: tuple             # ("fixed", N) | ("uniform", lo, hi) | ("loguniform", lo, hi) | ("list", (N0, N1, ...))
    layout: str = "paged"      # "paged" (16-token blocks, seeded shuffled block table) or "contiguous"
    block_size: int = 16
    spare_blocks: int = 8      # NaN-poisoned blocks never referenced by any sequence
    kv_std: float = 1.0
    weight_std: float = 0.02
    soft_std: float = 0.02
    gain_std: float = 0.02     # norm gains are 1 + N(0, gain_std^2)
    rope_base: float = 10000.0
    rms_eps: float = 1e-6
    pool: str = "last"         # "last" or "mean"
    seed: int = 0
    cls_bias: bool = False

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def rows_per_kv_head(self) -> int:
        return self.k * self.group

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)

    def max_seq_len(self) -> int:
        kind = self.seq_len[0]
        if kind == "fixed":
            return int(self.seq_len[1])
        if kind in ("uniform", "loguniform"):
            return int(self.seq_len[2])
        if kind == "list":
            return int(max(self.seq_len[1])) if len(self.seq_len[1]) else 0
        raise ValueError(kind)


# The five workloads.  Shapes: hidden 2560 / 4096 follow the Qwen3.5-4B / 9B heads
# (Sec. 5.1); the 27B-shaped workload uses hidden 5120 with 40 query heads.
TINY_F32 = Workload(
    name="tiny_f32", dtype="f32", batch=4, k=4, hidden=256, n_q_heads=4, n_kv_heads=2,
    head_dim=64, intermediate=1024, n_classes=2, seq_len=("fixed", 256), layout="paged",
    kv_std=0.02, seed=0)

QWEN4B_BF16 = Workload(
    name="4b_bf16", dtype="bf16", batch=64, k=16, hidden=2560, n_q_heads=32, n_kv_heads=8,
    head_dim=128, intermediate=9728, n_classes=2, seq_len=("uniform", 512, 4096),
    layout="contiguous", kv_std=1.0, seed=1)

QWEN9B_BF16 = Workload(
    name="9b_bf16", dtype="bf16", batch=128, k=16, hidden=4096, n_q_heads=32, n_kv_heads=8,
    head_dim=128, intermediate=12288, n_classes=3, seq_len=("loguniform", 1024, 8192),
    layout="paged", kv_std=1.0, seed=2)

QWEN27B_BF16 = Workload(
    name="27b_bf16", dtype="bf16", batch=256, k=32, hidden=5120, n_q_heads=40, n_kv_heads=8,
    head_dim=128, intermediate=17408, n_classes=2, seq_len=("loguniform", 2048, 32768),
    layout="paged", kv_std=1.0, seed=3)

LONG_9B_BF16 = Workload(
    name="long_9b_bf16", dtype="bf16", batch=32, k=16, hidden=4096, n_q_heads=32, n_kv_heads=8,
    head_dim=128, intermediate=12288, n_classes=4, seq_len=("fixed", 131072), layout="paged",
    kv_std=1.0, seed=4)

WORKLOADS = {w.name: w for w in (TINY_F32, QWEN4B_BF16, QWEN9B_BF16, QWEN27B_BF16, LONG_9B_BF16)}

# Stress variants used by the parity tests.
# Peaky scores: with KV ~ N(0, 0.02^2) the softmax of the tiny workload is almost
# uniform, so a wrong scale or a missing max-subtraction would go unnoticed.
TINY_PEAKY_F32 = TINY_F32.replace(name="tiny_peaky_f32", kv_std=3.0, weight_std=0.2, seed=10)
# Ragged lengths around block boundaries, including an empty context.
TINY_RAGGED_F32 = TINY_F32.replace(
    name="tiny_ragged_f32", batch=6, seq_len=("list", (0, 1, 15, 16, 17, 255)), kv_std=1.0,
    weight_std=0.1, seed=11)
# bf16 at small sizes: same logic, bf16 numerics, head_dim 128 as in the large workloads.
SMALL_BF16 = Workload(
    name="small_bf16", dtype="bf16", batch=5, k=4, hidden=512, n_q_heads=8, n_kv_heads=2,
    head_dim=128, intermediate=768, n_classes=3, seq_len=("list", (0, 1, 33, 100, 517)),
    layout="paged", kv_std=1.0, seed=12)
# Group size 5 (the 27B-shaped grouping) at small sizes, mean pooling, classifier bias.
SMALL_G5_BF16 = Workload(
    name="small_g5_bf16", dtype="bf16", batch=3, k=8, hidden=640, n_q_heads=10, n_kv_heads=2,
    head_dim=128, intermediate=1024, n_classes=2, seq_len=("list", (47, 300, 1000)),
    layout="paged", kv_std=1.0, seed=13, pool="mean", cls_bias=True)

STRESS = {w.name: w for w in (TINY_PEAKY_F32, TINY_RAGGED_F32, SMALL_BF16, SMALL_G5_BF16)}

# Recursive SP-k (the MTP input fusion of Sec. 3.1 chained over k steps,
# Sec. 3.2) on the same head shapes, with the paper's k in {1, 2, 5}.  The
# long-context one is the benchmark's recursive workload.
TINY_F32_SP2 = TINY_F32.replace(name="tiny_f32_sp2", k=2, weight_std=0.1, seed=60)
TINY_RAGGED_F32_SP5 = TINY_RAGGED_F32.replace(name="tiny_ragged_f32_sp5", k=5, seed=61)
SMALL_BF16_SP5 = SMALL_BF16.replace(name="small_bf16_sp5", k=5, seed=62)
SMALL_BF16_SP1 = SMALL_BF16.replace(name="small_bf16_sp1", k=1, seed=63)
SMALL_G5_BF16_SP2 = SMALL_G5_BF16.replace(name="small_g5_bf16_sp2", k=2, seed=64)   # mean, bias
QWEN9B_BF16_SP5 = QWEN9B_BF16.replace(name="9b_bf16_sp5", k=5)
QWEN27B_BF16_SP2 = QWEN27B_BF16.replace(name="27b_bf16_sp2", k=2)
LONG_9B_BF16_SP5 = LONG_9B_BF16.replace(name="long_9b_bf16_sp5", k=5)

RECURSIVE = {w.name: w for w in (TINY_F32_SP2, TINY_RAGGED_F32_SP5, SMALL_BF16_SP5, SMALL_BF16_SP1,
                                 SMALL_G5_BF16_SP2, QWEN9B_BF16_SP5, QWEN27B_BF16_SP2,
                                 LONG_9B_BF16_SP5)}
