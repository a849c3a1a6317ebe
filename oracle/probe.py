"""Oracle for the Speculative Probing classification forward.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path imports, calls or links
this module: only the tests, the smoke check and the benchmark's CPU-baseline
leg use it.  It shares no code, table or helper with the HIP library.

A plain, slow, fp64 numpy statement of what the probe computes for one sequence
(Sec. 3.2 "Speculative Probing", Sec. 3.3 Eq. 1-3), on the exact stored input
values (bf16 and fp32 inputs convert to fp64 without rounding):

  1. positions p_j = N + j for the k soft rows j = 0..k-1 appended after the N
     context tokens (Eq. 1-3 index the new rows n+1..n+k; here 0-based);
  2. u_j = RMSNorm(x_j; gamma_in), x_j the j-th soft-prompt vector, which takes
     the place of the token embedding at that position (Sec. 3.2, k = 1 case);
  3. q_j = W_q u_j, kappa_j = W_k u_j, v_j = W_v u_j, split into heads;
  4. RoPE (rotate-half pairs (i, i + hd/2), angle p_j * base^(-2i/hd)) on every
     query head and key head; values are not rotated;
  5. for query head h, KV head g = floor(h / G) with G = n_q / n_kv: the keys are
     the cached K_{1:n} of head g followed by the rotated soft keys of rows 0..j
     (causal among the soft rows, own row included), the values likewise
     (Eq. 2, Eq. 3); scores q.k / sqrt(hd), softmax with max subtraction, and
     the output is the probability-weighted sum of the values (Eq. 1);
  6. a_j = x_j + W_o concat_h(o_{j,h});
  7. y_j = a_j + W_down(silu(W_gate w_j) * (W_up w_j)), w_j = RMSNorm(a_j; gamma_post);
  8. f_j = RMSNorm(y_j; gamma_final); pooled = f_{k-1} ("last", the read-out of
     the k-th step, Sec. 3.2) or the mean of f_0..f_{k-1} ("mean", the "pooled
     final hidden state" of the Fig. 2 caption);
  9. logits = W_cls pooled (+ b_cls): the linear head of Sec. 3.2 with C rows
     instead of one, returned before any sigmoid.

Readings of points the paper leaves open (one pass instead of the recursive
chaining, soft prompt fed straight into the layer, the layer's internals,
causal mask among the soft rows, post-RoPE cached keys, contiguous GQA
grouping) are listed with the design notes of the repository.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class HeadShape:
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    rms_eps: float = 1e-6
    rope_base: float = 10000.0
    pool: str = "last"          # "last" | "mean"


def f64(x) -> np.ndarray:
    """Exact conversion of stored values to fp64."""
    return np.asarray(x, dtype=np.float64)


def rms_norm(x: np.ndarray, gain: np.ndarray, eps: float) -> np.ndarray:
    """Each row divided by the square root of (mean of its squares + eps), times gain."""
    x = f64(x)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * f64(gain)


def rope(x: np.ndarray, positions: np.ndarray, base: float) -> np.ndarray:
    """Rotary embedding, rotate-half pairing.

    x: [T, H, hd]; positions: [T].  Pair (i, i + hd/2) of row t is rotated by the
    angle positions[t] * base^(-2i/hd), angles formed in fp64."""
    x = f64(x)
    hd = x.shape[-1]
    half = hd // 2
    theta = float(base) ** (-(2.0 * np.arange(half, dtype=np.float64)) / hd)
    ang = f64(positions)[:, None] * theta[None, :]            # [T, half]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(z: np.ndarray) -> np.ndarray:
    """z * sigmoid(z)."""
    z = f64(z)
    return z / (1.0 + np.exp(-z))


def softmax_rows(s: np.ndarray) -> np.ndarray:
    """Row softmax with max subtraction; -inf entries get probability 0."""
    m = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def cached_attention(q_rot, k_cache, v_cache, k_soft, v_soft):
    """Attention of the k soft queries over [cached; new] keys (Eq. 1-3).

    q_rot:  [k, n_q, hd]  rotated soft queries
    k_cache, v_cache: [n_kv, N, hd]  the head's cached K (post-RoPE) and V
    k_soft: [k, n_kv, hd]  rotated soft keys;  v_soft: [k, n_kv, hd]
    Returns o [k, n_q, hd] and the probabilities, one [k, N + k] array per query
    head (columns N.. are the soft keys; entries above the diagonal are 0)."""
    q_rot, k_cache, v_cache = f64(q_rot), f64(k_cache), f64(v_cache)
    k_soft, v_soft = f64(k_soft), f64(v_soft)
    k, n_q, hd = q_rot.shape
    n_kv, n = k_cache.shape[0], k_cache.shape[1]
    group = n_q // n_kv
    scale = 1.0 / np.sqrt(hd)
    future = np.triu(np.ones((k, k), dtype=bool), 1)          # soft key j' > query j
    o = np.empty((k, n_q, hd))
    probs = []
    for h in range(n_q):
        g = h // group
        s_cache = q_rot[:, h, :] @ k_cache[g].T * scale         # [k, N]
        s_soft = q_rot[:, h, :] @ k_soft[:, g, :].T * scale     # [k, k]
        s_soft = np.where(future, -np.inf, s_soft)
        p = softmax_rows(np.concatenate([s_cache, s_soft], axis=1))
        o[:, h, :] = p[:, :n] @ v_cache[g] + p[:, n:] @ v_soft[:, g, :]
        probs.append(p)
    return o, probs


def probe_sequence(k_cache, v_cache, soft_prompt, weights: dict, shape: HeadShape) -> dict:
    """Logits and intermediate values for one sequence.

    k_cache, v_cache: [n_kv, N, hd]; soft_prompt: [k, d]; weights: dict with
    in_norm, w_q, w_k, w_v, w_o, post_norm, w_gate, w_up, w_down, final_norm,
    w_cls ([out, in] matrices) and optional b_cls."""
    W = {key: (None if val is None else f64(val)) for key, val in weights.items()}
    x = f64(soft_prompt)
    k, d = x.shape
    n = int(np.shape(k_cache)[1])
    hq, hkv, hd = shape.n_q_heads, shape.n_kv_heads, shape.head_dim
    pos = n + np.arange(k)

    u = rms_norm(x, W["in_norm"], shape.rms_eps)
    q = (u @ W["w_q"].T).reshape(k, hq, hd)
    kap = (u @ W["w_k"].T).reshape(k, hkv, hd)
    v = (u @ W["w_v"].T).reshape(k, hkv, hd)
    q_rot = rope(q, pos, shape.rope_base)
    k_rot = rope(kap, pos, shape.rope_base)

    o, probs = cached_attention(q_rot, k_cache, v_cache, k_rot, v)
    o_flat = o.reshape(k, hq * hd)
    a = x + o_flat @ W["w_o"].T
    w_in = rms_norm(a, W["post_norm"], shape.rms_eps)
    s = silu(w_in @ W["w_gate"].T) * (w_in @ W["w_up"].T)
    y = a + s @ W["w_down"].T
    f = rms_norm(y, W["final_norm"], shape.rms_eps)
    if shape.pool == "last":
        pooled = f[k - 1]
    elif shape.pool == "mean":
        pooled = np.mean(f, axis=0)
    else:
        raise ValueError(shape.pool)
    logits = W["w_cls"] @ pooled
    if W.get("b_cls") is not None:
        logits = logits + W["b_cls"]
    return {"u": u, "q_rot": q_rot, "k_rot": k_rot, "v": v, "probs": probs, "o": o_flat,
            "a": a, "s": s, "y": y, "f": f, "pooled": pooled, "logits": logits}


def probe_batch(kv_list, soft_prompt, weights: dict, shape: HeadShape, taps: bool = False):
    """Logits [B, C] for a batch; kv_list[b] = (k_cache_b, v_cache_b), each [n_kv, N_b, hd].

    Every sequence is classified on its own (Sec. 3.3): the batch is a loop."""
    outs = [probe_sequence(kc, vc, soft_prompt, weights, shape) for kc, vc in kv_list]
    logits = np.stack([o["logits"] for o in outs]) if outs else np.zeros((0, f64(weights["w_cls"]).shape[0]))
    return (logits, outs) if taps else logits
