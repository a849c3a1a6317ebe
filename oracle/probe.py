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
     the k-th step, Sec. 3.2) or the mean of f_0..f_{k-1} ("mean", the pooled
     read-out the Fig. 2 caption names);
  9. logits = W_cls pooled (+ b_cls): the linear head of Sec. 3.2 with C rows
     instead of one, returned before any sigmoid.

Readings of points the paper leaves open (one pass instead of the recursive
chaining, soft prompt fed straight into the layer, the layer's internals,
causal mask among the soft rows, post-RoPE cached keys, contiguous GQA
grouping) are listed with the design notes of the repository.

The recursive form the paper evaluates (SP-k: the MTP input fusion of
Sec. 3.1, chained over k steps as in Sec. 3.2) is ``probe_sequence_recursive``
at the end of this module.
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


def read_out(W: dict, pooled: np.ndarray) -> np.ndarray:
    """Logits of the pooled final hidden state: the linear head W_cls (Sec. 3.2), or,
    when W holds ``cls_rows``, the rows of a vocabulary matrix W_cls (the frozen
    LM head of the classification-head ablation, Sec. 6.7: with the rows of the
    yes and no tokens, logits[0] - logits[1] is the yes/no score)."""
    w_cls = W["w_cls"]
    if W.get("cls_rows") is not None:
        w_cls = w_cls[np.asarray(W["cls_rows"], dtype=np.int64)]
    logits = w_cls @ pooled
    if W.get("b_cls") is not None:
        logits = logits + W["b_cls"]
    return logits


def _weights64(weights: dict) -> dict:
    """Weights as fp64 arrays; integer row indices stay integers."""
    return {key: (None if val is None else (np.asarray(val, dtype=np.int64) if key == "cls_rows" else f64(val)))
            for key, val in weights.items()}


def probe_sequence(k_cache, v_cache, soft_prompt, weights: dict, shape: HeadShape) -> dict:
    """Logits and intermediate values for one sequence.

    k_cache, v_cache: [n_kv, N, hd]; soft_prompt: [k, d]; weights: dict with
    in_norm, w_q, w_k, w_v, w_o, post_norm, w_gate, w_up, w_down, final_norm,
    w_cls ([out, in] matrices) and optional b_cls."""
    W = _weights64(weights)
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
    logits = read_out(W, pooled)
    return {"u": u, "q_rot": q_rot, "k_rot": k_rot, "v": v, "probs": probs, "o": o_flat,
            "a": a, "s": s, "y": y, "f": f, "pooled": pooled, "logits": logits}


def probe_batch(kv_list, soft_prompt, weights: dict, shape: HeadShape, taps: bool = False):
    """Logits [B, C] for a batch; kv_list[b] = (k_cache_b, v_cache_b), each [n_kv, N_b, hd].

    Every sequence is classified on its own (Sec. 3.3): the batch is a loop."""
    outs = [probe_sequence(kc, vc, soft_prompt, weights, shape) for kc, vc in kv_list]
    logits = np.stack([o["logits"] for o in outs]) if outs else np.zeros((0, f64(weights["w_cls"]).shape[0]))
    return (logits, outs) if taps else logits


# ---------------------------------------------------------------- recursive SP-k
#
# Sec. 3.1 (MTP architecture) and Sec. 3.2 (recursive soft prompts): the head's
# input at a position is the projection W_fc [RMSNorm(h; gamma_h);
# RMSNorm(e; gamma_e)] of a hidden state h and an embedding e; SP-k replaces the
# embedding of step i with the learned vector e_i, takes the base model's last
# hidden state as h for the first step and the head's own output hidden state
# of step i-1 for every later step, and classifies the output of step k.
#
# Readings (the paper leaves them open):
#   * w_fc is stored [d][2d]; its columns 0..d-1 multiply the normed hidden
#     state and columns d..2d-1 the normed soft-prompt vector (the order in
#     which Sec. 3.1 lists the two inputs);
#   * the output hidden state a step hands on (and the one the classifier
#     reads) is the final-normed f_t;
#   * step t (0-based) sits at position N + t and attends to the N cached keys
#     plus the soft keys of steps 0..t (its own included);
#   * the read-out options are those of the one-pass form: f of the last step,
#     or the mean of f over the k steps.

def recursive_step(x_t, t, n, k_cache, v_cache, soft_k, soft_v, W, shape):
    """One application of the decoder layer to the fused input x_t [d] at
    position n + t.  soft_k / soft_v (lists of [n_kv, hd]) hold the rotated soft
    keys and the values of steps 0..t-1 and receive this step's.  Returns the
    step's taps (x, q_rot, probabilities, o, a, s, y, f)."""
    hq, hkv, hd = shape.n_q_heads, shape.n_kv_heads, shape.head_dim
    group = hq // hkv
    u = rms_norm(x_t, W["in_norm"], shape.rms_eps)
    q = (W["w_q"] @ u).reshape(1, hq, hd)
    kap = (W["w_k"] @ u).reshape(1, hkv, hd)
    v = (W["w_v"] @ u).reshape(hkv, hd)
    pos = np.array([n + t])
    q_rot = rope(q, pos, shape.rope_base)[0]
    soft_k.append(rope(kap, pos, shape.rope_base)[0])
    soft_v.append(v)
    keys_soft = np.stack(soft_k)                    # [t+1, n_kv, hd]
    vals_soft = np.stack(soft_v)
    kc, vc = f64(k_cache), f64(v_cache)
    o = np.empty((hq, hd))
    probs = []
    for h in range(hq):
        g = h // group
        keys = np.concatenate([kc[g], keys_soft[:, g, :]])     # [n + t + 1, hd]
        vals = np.concatenate([vc[g], vals_soft[:, g, :]])
        p = softmax_rows((keys @ q_rot[h] / np.sqrt(hd))[None, :])[0]
        o[h] = p @ vals
        probs.append(p)
    a = x_t + W["w_o"] @ o.reshape(hq * hd)
    w_in = rms_norm(a, W["post_norm"], shape.rms_eps)
    s = silu(W["w_gate"] @ w_in) * (W["w_up"] @ w_in)
    y = a + W["w_down"] @ s
    f = rms_norm(y, W["final_norm"], shape.rms_eps)
    return {"x": x_t, "q_rot": q_rot, "probs": probs, "o": o.reshape(hq * hd), "a": a, "s": s,
            "y": y, "f": f}


def probe_sequence_recursive(k_cache, v_cache, soft_prompt, h_last, weights: dict,
                             shape: HeadShape) -> dict:
    """Recursive SP-k logits and per-step values for one sequence.

    k_cache, v_cache: [n_kv, N, hd]; soft_prompt: [k, d] (e_1..e_k); h_last: [d],
    the base model's last hidden state ([3d] with w_hidden_fuse); weights: the
    one-pass keys plus fc_norm_h [d], fc_norm_e [d], w_fc [d][2d] and optionally
    w_hidden_fuse [d][3d] (Eagle3 input).  Returned arrays stack the
    steps: x, a, y, f are [k, d], o is [k, n_q*hd]."""
    W = _weights64(weights)
    e = f64(soft_prompt)
    k, d = e.shape
    n = int(np.shape(k_cache)[1])
    h = f64(h_last)
    if W.get("w_hidden_fuse") is not None:
        # Eagle3 input (Sec. 3.1, Eagle3 paragraph): h_last holds three hidden
        # states of the base model (low, mid, high layer) concatenated, and the
        # first hidden state is their projection (no norm before it)
        h = W["w_hidden_fuse"] @ h
    soft_k, soft_v, steps = [], [], []
    for t in range(k):
        z = np.concatenate([rms_norm(h, W["fc_norm_h"], shape.rms_eps),
                            rms_norm(e[t], W["fc_norm_e"], shape.rms_eps)])
        x_t = W["w_fc"] @ z
        st = recursive_step(x_t, t, n, k_cache, v_cache, soft_k, soft_v, W, shape)
        steps.append(st)
        h = st["f"]
    f = np.stack([st["f"] for st in steps])
    if shape.pool == "last":
        pooled = f[k - 1]
    elif shape.pool == "mean":
        pooled = np.mean(f, axis=0)
    else:
        raise ValueError(shape.pool)
    logits = read_out(W, pooled)
    out = {name: np.stack([st[name] for st in steps]) for name in ("x", "o", "a", "y", "f")}
    out.update({"probs": [st["probs"] for st in steps], "pooled": pooled, "logits": logits})
    return out


def probe_batch_recursive(kv_list, soft_prompt, h_last, weights: dict, shape: HeadShape,
                          taps: bool = False):
    """Recursive SP-k logits [B, C]; h_last [B, d] holds each sequence's last base hidden state."""
    outs = [probe_sequence_recursive(kc, vc, soft_prompt, h_last[b], weights, shape)
            for b, (kc, vc) in enumerate(kv_list)]
    logits = np.stack([o["logits"] for o in outs]) if outs else np.zeros((0, f64(weights["w_cls"]).shape[0]))
    return (logits, outs) if taps else logits


# ---------------------------------------------------------------- several tasks on one cache
#
# Sec. 3.3 (cost paragraph): classifiers with different soft prompts and heads
# can share the same KV cache, so several monitoring tasks run at once.  Each
# task is an independent probe: its soft rows see the cache and their own
# task's soft rows only, and it has its own classifier.  The definition is
# therefore the single-task probe once per task.

def probe_batch_tasks(kv_list, soft_prompts, w_cls, b_cls, weights: dict, shape: HeadShape,
                      cls_rows=None):
    """Logits [B, T, C]: task t uses soft_prompts[t] ([k, d]), w_cls[t] ([C, d]) and
    b_cls[t] (or no bias when b_cls is None) with the shared frozen head.  With
    cls_rows ([T, C]) w_cls is one vocabulary matrix and task t reads its rows
    cls_rows[t]."""
    per_task = []
    for t in range(len(soft_prompts)):
        W = dict(weights, w_cls=w_cls[t] if cls_rows is None else w_cls,
                 b_cls=None if b_cls is None else b_cls[t],
                 cls_rows=None if cls_rows is None else cls_rows[t])
        per_task.append(probe_batch(kv_list, soft_prompts[t], W, shape))
    return np.stack(per_task, axis=1)
