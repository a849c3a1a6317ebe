"""Seeded synthetic inputs for the probe forward: frozen head weights, soft
prompts, classifier, context lengths and the head's resident KV cache.

This module serves both the HIP path and the oracle and therefore holds none of
the method's arithmetic: it draws random numbers, lays them out in memory and
gathers them back (pure indexing).  Every tensor is a pure function of
(workload seed, tensor tag, device): the same call on the same device always
returns the same bytes.

KV cache storage (the boundary's paged layout).  The pool is one tensor
``pool[num_blocks, n_kv, 2, block_size * head_dim]``.  For block ``p`` and KV
head ``g``:
  * ``pool[p, g, 0]`` is the K tile in 16-byte chunks of the head dimension:
    element (t, i) at ``((i // x) * block_size + t) * x + i % x`` with
    x = 16 / element size (8 for bf16, 4 for fp32);
  * ``pool[p, g, 1]`` is the V tile, dim-major: element (t, i) at ``i*block_size + t``.
Token slots past a sequence's length and every spare block are filled with NaN,
so any read of them that reaches an output shows up as NaN.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Optional

import numpy as np
import torch

from .configs import Workload

# Tensor tags for seed derivation.
_TAGS = {
    "seq_len": 1, "perm": 2, "kv": 3, "soft": 10, "in_norm": 11, "w_q": 12, "w_k": 13, "w_v": 14,
    "w_o": 15, "post_norm": 16, "w_gate": 17, "w_up": 18, "w_down": 19, "final_norm": 20,
    "w_cls": 21, "b_cls": 22, "fc_norm_hidden": 23, "fc_norm_embed": 24, "w_fc": 25,
    "hidden_last": 26, "lm_head": 27, "cls_rows": 28, "w_hidden_fuse": 29, "hidden3": 30,
}

TORCH_DTYPE = {"f32": torch.float32, "bf16": torch.bfloat16}


def _seed(w: Workload, tag: str, extra: int = 0) -> int:
    ss = np.random.SeedSequence([w.seed, _TAGS[tag], extra])
    return int(ss.generate_state(1, dtype=np.uint64)[0] & ((1 << 62) - 1))


def _gen(w: Workload, tag: str, device, extra: int = 0) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(_seed(w, tag, extra))
    return g


def seq_lens(w: Workload) -> np.ndarray:
    """Context length N_b of every sequence (int32 [B]).

    uniform: integers in [lo, hi] inclusive; loguniform: round(exp(U(ln lo, ln hi)))
    clamped to [lo, hi]; fixed: N for every sequence; list: the given lengths."""
    kind = w.seq_len[0]
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([w.seed, _TAGS["seq_len"]])))
    if kind == "fixed":
        out = np.full(w.batch, int(w.seq_len[1]), dtype=np.int64)
    elif kind == "uniform":
        lo, hi = int(w.seq_len[1]), int(w.seq_len[2])
        out = rng.integers(lo, hi + 1, size=w.batch)
    elif kind == "loguniform":
        lo, hi = int(w.seq_len[1]), int(w.seq_len[2])
        out = np.rint(np.exp(rng.uniform(math.log(lo), math.log(hi), size=w.batch)))
        out = np.clip(out, lo, hi)
    elif kind == "list":
        out = np.asarray(w.seq_len[1], dtype=np.int64)
        if out.shape != (w.batch,):
            raise ValueError("seq_len list must have one entry per sequence")
    else:
        raise ValueError(kind)
    return out.astype(np.int32)


def _normal(shape, mean, std, dtype, device, gen) -> torch.Tensor:
    t = torch.empty(shape, dtype=dtype, device=device)
    t.normal_(mean, std, generator=gen)
    return t


def params(w: Workload, device="cpu", only=None) -> dict:
    """Frozen head weights ([out, in] row-major), norm gains, soft prompts and the
    linear classifier, in the workload's storage dtype (classifier bias: fp32).
    only: names to draw (each tensor has its own stream, so a subset has the
    same bytes as in the full set); default all."""
    dt = TORCH_DTYPE[w.dtype]
    d, hd, I = w.hidden, w.head_dim, w.intermediate
    qd, kvd = w.n_q_heads * hd, w.n_kv_heads * hd
    ws, gs = w.weight_std, w.gain_std
    spec = {
        "soft_prompt": ((w.k, d), 0.0, w.soft_std, dt, "soft"),
        "in_norm": ((d,), 1.0, gs, dt, "in_norm"),
        "w_q": ((qd, d), 0.0, ws, dt, "w_q"),
        "w_k": ((kvd, d), 0.0, ws, dt, "w_k"),
        "w_v": ((kvd, d), 0.0, ws, dt, "w_v"),
        "w_o": ((d, qd), 0.0, ws, dt, "w_o"),
        "post_norm": ((d,), 1.0, gs, dt, "post_norm"),
        "w_gate": ((I, d), 0.0, ws, dt, "w_gate"),
        "w_up": ((I, d), 0.0, ws, dt, "w_up"),
        "w_down": ((d, I), 0.0, ws, dt, "w_down"),
        "final_norm": ((d,), 1.0, gs, dt, "final_norm"),
        "w_cls": ((w.n_classes, d), 0.0, ws, dt, "w_cls"),
        "b_cls": ((w.n_classes,), 0.0, 1.0, torch.float32, "b_cls"),
    }
    p = {}
    for name, (shape, mean, std, tdt, tag) in spec.items():
        if only is not None and name not in only:
            continue
        if name == "b_cls" and not w.cls_bias:
            p[name] = None
            continue
        p[name] = _normal(shape, mean, std, tdt, device, _gen(w, tag, device))
    return p


def task_params(w: Workload, n_tasks: int, device="cpu") -> dict:
    """Per-task inputs of a multi-task call: soft_prompts [T][k][d], w_cls [T][C][d]
    and b_cls [T][C] (None without a bias).  Task 0 has the single-task values of
    params(); task t > 0 draws its own from the same distributions."""
    dt = TORCH_DTYPE[w.dtype]
    d = w.hidden
    soft = [_normal((w.k, d), 0.0, w.soft_std, dt, device, _gen(w, "soft", device, t)) for t in range(n_tasks)]
    wc = [_normal((w.n_classes, d), 0.0, w.weight_std, dt, device, _gen(w, "w_cls", device, t))
          for t in range(n_tasks)]
    bc = ([_normal((w.n_classes,), 0.0, 1.0, torch.float32, device, _gen(w, "b_cls", device, t))
           for t in range(n_tasks)] if w.cls_bias else None)
    return {"soft_prompts": torch.stack(soft).contiguous(), "w_cls": torch.stack(wc).contiguous(),
            "b_cls": torch.stack(bc).contiguous() if bc is not None else None}


def fusion_params(w: Workload, device="cpu") -> dict:
    """Inputs of the recursive form only (MTP input fusion, Sec. 3.1): the two
    pre-fusion norm gains (1 + N(0, gain_std^2)), the fusion matrix w_fc [d][2d]
    (N(0, weight_std^2)) and the base model's last hidden state of every
    sequence, hidden_last [B][d] ~ N(0, 1), all in the storage dtype."""
    dt = TORCH_DTYPE[w.dtype]
    d = w.hidden
    return {
        "fc_norm_hidden": _normal((d,), 1.0, w.gain_std, dt, device, _gen(w, "fc_norm_hidden", device)),
        "fc_norm_embed": _normal((d,), 1.0, w.gain_std, dt, device, _gen(w, "fc_norm_embed", device)),
        "w_fc": _normal((d, 2 * d), 0.0, w.weight_std, dt, device, _gen(w, "w_fc", device)),
        "hidden_last": _normal((w.batch, d), 0.0, 1.0, dt, device, _gen(w, "hidden_last", device)),
    }


def lm_head_params(w: Workload, vocab: int, n_tasks: int = 1, device="cpu") -> dict:
    """Vocabulary read-out inputs: a frozen LM head [vocab][d] ~ N(0, weight_std^2) in
    the storage dtype and, per task, C distinct label-token rows (int32 [T][C])."""
    dt = TORCH_DTYPE[w.dtype]
    head = _normal((vocab, w.hidden), 0.0, w.weight_std, dt, device, _gen(w, "lm_head", device))
    rng = np.random.default_rng(_seed(w, "cls_rows"))
    rows = np.stack([rng.choice(vocab, w.n_classes, replace=False) for _ in range(n_tasks)]).astype(np.int32)
    return {"lm_head": head, "cls_rows": torch.from_numpy(rows).to(device)}


def eagle3_params(w: Workload, device="cpu") -> dict:
    """Eagle3 input: the projection w_hidden_fuse [d][3d] ~ N(0, weight_std^2) and three
    base-model hidden states per sequence, hidden3 [B][3d] ~ N(0, 1), with a few
    large entries per state (magnitudes up to 1e5, as base models' massive
    activations can be; beyond fp16's range on purpose)."""
    dt = TORCH_DTYPE[w.dtype]
    d = w.hidden
    wf = _normal((d, 3 * d), 0.0, w.weight_std, dt, device, _gen(w, "w_hidden_fuse", device))
    g = _gen(w, "hidden3", device)
    h = torch.randn((w.batch, 3 * d), generator=g, device=device, dtype=torch.float32)
    idx = torch.randint(0, 3 * d, (w.batch, 4), generator=g, device=device)
    big = torch.tensor([3.0e3, -2.0e4, 1.0e5, 600.0], device=device).expand(w.batch, 4)
    h.scatter_(1, idx, big)
    return {"w_hidden_fuse": wf, "hidden3": h.to(dt)}


@dataclass
class KVCache:
    """The head's resident KV cache in the boundary's paged layout."""
    pool: torch.Tensor                  # [num_blocks, n_kv, 2, block_size*head_dim]
    block_table: Optional[torch.Tensor]  # int32 [B, max_blocks_per_seq] or None (contiguous)
    seq_lens: torch.Tensor              # int32 [B], same device as pool
    block_size: int
    max_blocks_per_seq: int
    n_kv: int
    head_dim: int

    @property
    def num_blocks(self) -> int:
        return self.pool.shape[0]

    @property
    def stride_block(self) -> int:
        return self.pool.stride(0)

    @property
    def stride_head(self) -> int:
        return self.pool.stride(1)

    @property
    def v_offset(self) -> int:
        return self.block_size * self.head_dim

    def physical_blocks(self, b: int) -> torch.Tensor:
        if self.block_table is None:
            return torch.arange(b * self.max_blocks_per_seq, (b + 1) * self.max_blocks_per_seq,
                                device=self.pool.device)
        return self.block_table[b].long()

    @property
    def x(self) -> int:
        return 16 // self.pool.element_size()

    def logical_kv(self, b: int):
        """(K, V) of sequence b as dense [n_kv, N_b, head_dim] tensors on the pool's device."""
        n = int(self.seq_lens[b])
        nblk = -(-n // self.block_size)
        blocks = self.physical_blocks(b)[:nblk]
        tiles = self.pool.index_select(0, blocks)            # [nblk, n_kv, 2, bs*hd]
        bs, hd = self.block_size, self.head_dim
        x = self.x
        k = tiles[:, :, 0].reshape(nblk, self.n_kv, hd // x, bs, x).permute(0, 1, 3, 2, 4)
        k = k.reshape(nblk, self.n_kv, bs, hd)
        v = tiles[:, :, 1].reshape(nblk, self.n_kv, hd, bs).transpose(2, 3)
        k = k.permute(1, 0, 2, 3).reshape(self.n_kv, nblk * bs, hd)[:, :n]
        v = v.permute(1, 0, 2, 3).reshape(self.n_kv, nblk * bs, hd)[:, :n]
        return k.contiguous(), v.contiguous()


def _poison_tail(pool: torch.Tensor, blk: int, used: int, bs: int, hd: int) -> None:
    n_kv = pool.shape[1]
    x = 16 // pool.element_size()
    kt = pool[blk, :, 0].view(n_kv, hd // x, bs, x)
    vt = pool[blk, :, 1].view(n_kv, hd, bs)
    kt[:, :, used:, :] = float("nan")
    vt[:, :, used:] = float("nan")


def kv_cache(w: Workload, lens: np.ndarray, device="cpu", layout: Optional[str] = None,
             block_size: Optional[int] = None, perm_seed: int = 0) -> KVCache:
    """Build the KV pool for context lengths ``lens``.

    paged: blocks of ``block_size`` tokens, a seeded random permutation of the
    physical blocks (``perm_seed`` selects another permutation), ``spare_blocks``
    extra NaN blocks, unused block-table entries pointing at a spare block.
    Values are drawn in physical order; ``repack`` stores the same logical KV in
    another layout.  contiguous: one block per sequence whose size is
    the smallest power of two >= the longest context, no block table."""
    layout = layout or w.layout
    dt = TORCH_DTYPE[w.dtype]
    n_kv, hd = w.n_kv_heads, w.head_dim
    B = len(lens)
    max_len = max(int(lens.max()) if B else 0, w.max_seq_len(), 1)
    if layout == "contiguous":
        bs = block_size or max(16, 1 << (max_len - 1).bit_length())
        mbps = -(-max_len // bs)
        nblocks_seq = [mbps] * B
        num_blocks = B * mbps
    elif layout == "paged":
        bs = block_size or w.block_size
        mbps = -(-max_len // bs)
        nblocks_seq = [-(-int(n) // bs) for n in lens]
        num_blocks = sum(nblocks_seq) + w.spare_blocks
    else:
        raise ValueError(layout)
    if bs < 16 or (bs & (bs - 1)):
        raise ValueError("block_size must be a power of two >= 16")

    pool = torch.empty((num_blocks, n_kv, 2, bs * hd), dtype=dt, device=device)
    gen = _gen(w, "kv", device)
    chunk = max(1, (1 << 30) // max(1, pool[0].numel() * pool.element_size()))
    for c0 in range(0, num_blocks, chunk):
        pool[c0:c0 + chunk].normal_(0.0, w.kv_std, generator=gen)
    if layout == "paged":
        order = torch.randperm(num_blocks, generator=_gen(w, "perm", "cpu", perm_seed))
        used = sum(nblocks_seq)
        phys, spare = order[:used], order[used:]
        bt = torch.empty((B, mbps), dtype=torch.int32)
        bt[:] = int(spare[0]) if len(spare) else 0
        pos = 0
        for b, nb in enumerate(nblocks_seq):
            bt[b, :nb] = phys[pos:pos + nb].to(torch.int32)
            pos += nb
        if len(spare):
            pool.index_fill_(0, spare.to(device), float("nan"))
        for b, nb in enumerate(nblocks_seq):
            rem = int(lens[b]) - (nb - 1) * bs
            if nb and rem < bs:
                _poison_tail(pool, int(bt[b, nb - 1]), rem, bs, hd)
        block_table = bt.to(device)
    else:
        for b in range(B):
            n = int(lens[b])
            nb = -(-n // bs) if n else 0
            for j in range(nb, mbps):
                pool[b * mbps + j] = float("nan")
            rem = n - (nb - 1) * bs
            if nb and rem < bs:
                _poison_tail(pool, b * mbps + nb - 1, rem, bs, hd)
        block_table = None
    return KVCache(pool=pool, block_table=block_table,
                   seq_lens=torch.as_tensor(np.asarray(lens, dtype=np.int32)).to(device),
                   block_size=bs, max_blocks_per_seq=mbps, n_kv=n_kv, head_dim=hd)


def repack(kv: KVCache, layout: str, block_size: Optional[int] = None, perm_seed: int = 0) -> KVCache:
    """Store the same logical KV in another layout / block size / block placement."""
    B = kv.seq_lens.shape[0]
    lens = kv.seq_lens.cpu().numpy()
    n_kv, hd = kv.n_kv, kv.head_dim
    dev, dt = kv.pool.device, kv.pool.dtype
    max_len = max(int(lens.max()) if B else 0, kv.max_blocks_per_seq * kv.block_size, 1)
    if layout == "contiguous":
        bs = block_size or max(16, 1 << (max_len - 1).bit_length())
    else:
        bs = block_size or 16
    mbps = -(-max_len // bs)
    nblocks_seq = [mbps] * B if layout == "contiguous" else [-(-int(n) // bs) for n in lens]
    spare = 0 if layout == "contiguous" else 3
    num_blocks = sum(nblocks_seq) + spare
    pool = torch.full((num_blocks, n_kv, 2, bs * hd), float("nan"), dtype=dt, device=dev)
    if layout == "paged":
        g = torch.Generator(device="cpu")
        g.manual_seed(1000 + perm_seed)
        order = torch.randperm(num_blocks, generator=g)
    else:
        order = torch.arange(num_blocks)
    bt = torch.empty((B, mbps), dtype=torch.int32)
    bt[:] = int(order[-1])
    pos = 0
    for b in range(B):
        nb = nblocks_seq[b]
        bt[b, :nb] = order[pos:pos + nb].to(torch.int32)
        pos += nb
        n = int(lens[b])
        if n == 0:
            continue
        k, v = kv.logical_kv(b)                             # [n_kv, n, hd]
        npad = -(-n // bs) * bs
        kp = torch.full((n_kv, npad, hd), float("nan"), dtype=dt, device=dev)
        vp = torch.full((n_kv, npad, hd), float("nan"), dtype=dt, device=dev)
        kp[:, :n] = k
        vp[:, :n] = v
        for j in range(npad // bs):
            p = int(bt[b, j])
            x = 16 // pool.element_size()
            kt = kp[:, j * bs:(j + 1) * bs].reshape(n_kv, bs, hd // x, x).permute(0, 2, 1, 3)
            pool[p, :, 0] = kt.reshape(n_kv, bs * hd)
            pool[p, :, 1] = vp[:, j * bs:(j + 1) * bs].transpose(1, 2).reshape(n_kv, bs * hd)
    return KVCache(pool=pool, block_table=None if layout == "contiguous" else bt.to(dev),
                   seq_lens=kv.seq_lens.clone(), block_size=bs, max_blocks_per_seq=mbps,
                   n_kv=n_kv, head_dim=hd)


def permute_batch(kv: KVCache, perm) -> KVCache:
    """The same pool with sequences reordered (block-table rows permuted)."""
    perm_t = torch.as_tensor(perm, dtype=torch.long)
    if kv.block_table is None:
        raise ValueError("permute a paged cache")
    return KVCache(pool=kv.pool, block_table=kv.block_table[perm_t.to(kv.block_table.device)].contiguous(),
                   seq_lens=kv.seq_lens[perm_t.to(kv.seq_lens.device)].contiguous(),
                   block_size=kv.block_size, max_blocks_per_seq=kv.max_blocks_per_seq,
                   n_kv=kv.n_kv, head_dim=kv.head_dim)
