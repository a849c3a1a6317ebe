"""Independent statements used to pin the oracle (test code only).

Written in a different style from the oracle, sharing none of its code, so that
a slip in one is not repeated in the other:

* ``full_layer``: the head's decoder layer run over a whole token sequence at
  once, with a causal mask matrix, GQA by repeating KV heads, and RoPE as a
  complex rotation.  Sec. 3.3 states that the soft rows' outputs computed from
  the cached K/V (Eq. 1-3) are the same as running the layer over the
  sequence with the soft rows appended; this gives that second computation.
* ``textbook_decode``: single-query attention with explicit Python loops.
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import expit


def _rms(x, gain, eps):
    d = x.shape[-1]
    rms = np.linalg.norm(x, axis=-1, keepdims=True) / math.sqrt(d)
    return x * gain / np.sqrt(rms ** 2 + eps)


def _rope_complex(x, pos, base):
    """x [T, H, hd]: treat (x[i], x[i + hd/2]) as the complex number x[i] + 1j x[i+hd/2]
    and multiply by exp(1j * pos * base^(-2i/hd))."""
    hd = x.shape[-1]
    half = hd // 2
    z = x[..., :half] + 1j * x[..., half:]
    freqs = np.exp(-np.log(base) * (2.0 * np.arange(half)) / hd)
    rot = np.exp(1j * np.outer(pos, freqs))[:, None, :]
    zr = z * rot
    return np.concatenate([zr.real, zr.imag], axis=-1)


def full_layer(x_seq, weights, n_q, n_kv, hd, eps, base, pos_offset=0):
    """Decoder layer over every row of x_seq [T, d] with a causal mask.

    Returns dict: f (final-normed rows [T, d]), k_rot [n_kv, T, hd] (post-RoPE
    keys), v [n_kv, T, hd], attn [T, n_q*hd], a, y."""
    W = {k: (None if v is None else np.asarray(v, np.float64)) for k, v in weights.items()}
    x = np.asarray(x_seq, np.float64)
    T, d = x.shape
    pos = np.arange(T) + pos_offset
    h = _rms(x, W["in_norm"], eps)
    q = np.einsum("td,ed->te", h, W["w_q"]).reshape(T, n_q, hd)
    kk = np.einsum("td,ed->te", h, W["w_k"]).reshape(T, n_kv, hd)
    vv = np.einsum("td,ed->te", h, W["w_v"]).reshape(T, n_kv, hd)
    q = _rope_complex(q, pos, base)
    kk = _rope_complex(kk, pos, base)
    G = n_q // n_kv
    k_rep = np.repeat(kk, G, axis=1)                        # [T, n_q, hd], head h uses kv head h // G
    v_rep = np.repeat(vv, G, axis=1)
    scores = np.einsum("thc,shc->hts", q, k_rep) / math.sqrt(hd)
    allowed = np.tril(np.ones((T, T), dtype=bool))
    scores = np.where(allowed[None], scores, -np.inf)
    scores = scores - scores.max(axis=-1, keepdims=True)
    p = np.exp(scores)
    p = p / p.sum(axis=-1, keepdims=True)
    attn = np.einsum("hts,shc->thc", p, v_rep).reshape(T, n_q * hd)
    a = x + attn @ W["w_o"].T
    g_in = _rms(a, W["post_norm"], eps)
    gate = g_in @ W["w_gate"].T
    mlp = (gate * expit(gate) * (g_in @ W["w_up"].T)) @ W["w_down"].T
    y = a + mlp
    f = _rms(y, W["final_norm"], eps)
    return {"f": f, "k_rot": kk.transpose(1, 0, 2), "v": vv.transpose(1, 0, 2), "attn": attn,
            "a": a, "y": y}


def textbook_decode(q, keys, values):
    """Single-query attention: softmax(q.k_t / sqrt(hd)) weighted sum of v_t, by loops."""
    hd = len(q)
    scores = []
    for kt in keys:
        s = 0.0
        for i in range(hd):
            s += float(q[i]) * float(kt[i])
        scores.append(s / math.sqrt(hd))
    mx = max(scores)
    ws = [math.exp(s - mx) for s in scores]
    tot = sum(ws)
    out = [0.0] * hd
    for wt, vt in zip(ws, values):
        for i in range(hd):
            out[i] += wt / tot * float(vt[i])
    return np.array(out)


def draft_without_cache(x_ctx, e, h_last, weights, n_q, n_kv, hd, eps, base):
    """Recursive SP-k computed the way a head without a KV cache would draft:
    every step re-runs ``full_layer`` over the whole sequence [context rows;
    fused rows of steps 0..t] and keeps the last row.  The fused row of step t
    is w_fc applied to the two normed inputs stacked as (hidden, soft vector),
    the hidden being the base model's last state for t = 0 and the previous
    step's final-normed output after that.

    Returns dict: x [k, d] fused rows, f [k, d] final-normed outputs of the
    steps, and the full_layer result of the last step (rows N.. are the steps)."""
    W = {k: (None if v is None else np.asarray(v, np.float64)) for k, v in weights.items()}
    x_ctx = np.asarray(x_ctx, np.float64).reshape(-1, np.shape(e)[1])
    e = np.asarray(e, np.float64)
    hid = np.asarray(h_last, np.float64)
    rows, outs, last = [], [], None
    for t in range(e.shape[0]):
        stacked = np.concatenate([_rms(hid[None], W["fc_norm_h"], eps)[0],
                                  _rms(e[t][None], W["fc_norm_e"], eps)[0]])
        row = np.einsum("ij,j->i", W["w_fc"], stacked)
        rows.append(row)
        last = full_layer(np.concatenate([x_ctx, np.stack(rows)]), W, n_q, n_kv, hd, eps, base)
        hid = last["f"][-1]
        outs.append(hid)
    return {"x": np.stack(rows), "f": np.stack(outs), "last": last}
