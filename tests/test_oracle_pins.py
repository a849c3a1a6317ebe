"""Pins of the oracle against facts the paper and the mathematics fix (CPU only).

Each test names the passage or the mathematical fact it checks.  Between them
they are meant to catch a dropped term, a wrong sign, index or position, a
transposed operand or a wrong scale anywhere in the oracle.
"""
from __future__ import annotations

import math

import numpy as np
import pytest

from oracle import probe as O
from tests import independent as ind


def rand_weights(rng, d, n_q, n_kv, hd, inter, C, std=0.2, gain_std=0.1, bias=False):
    return {
        "in_norm": 1 + gain_std * rng.standard_normal(d),
        "w_q": std * rng.standard_normal((n_q * hd, d)),
        "w_k": std * rng.standard_normal((n_kv * hd, d)),
        "w_v": std * rng.standard_normal((n_kv * hd, d)),
        "w_o": std * rng.standard_normal((d, n_q * hd)),
        "post_norm": 1 + gain_std * rng.standard_normal(d),
        "w_gate": std * rng.standard_normal((inter, d)),
        "w_up": std * rng.standard_normal((inter, d)),
        "w_down": std * rng.standard_normal((d, inter)),
        "final_norm": 1 + gain_std * rng.standard_normal(d),
        "w_cls": std * rng.standard_normal((C, d)),
        "b_cls": rng.standard_normal(C) if bias else None,
    }


SHAPES = [
    # (d, n_q, n_kv, hd, inter, k, N)
    (16, 4, 2, 4, 24, 3, 7),     # GQA, group 2
    (24, 6, 2, 8, 20, 4, 0),     # empty context: soft rows attend only to each other
    (16, 2, 2, 8, 12, 1, 5),     # MHA, k = 1
    (20, 5, 1, 4, 16, 2, 9),     # MQA, group 5
]


# ---------------------------------------------------------------- building blocks

def test_rms_norm_closed_form():
    """RMSNorm of a constant vector c*1 is c / sqrt(c^2 + eps) times the gain."""
    for c, eps in [(3.0, 0.0), (-2.0, 1e-6), (0.5, 0.25)]:
        x = np.full((1, 8), c)
        gain = np.arange(1, 9, dtype=np.float64)
        out = O.rms_norm(x, gain, eps)
        np.testing.assert_allclose(out[0], c / math.sqrt(c * c + eps) * gain, rtol=1e-15)


def test_rms_norm_scale_invariance_and_unit_rms():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, 32))
    out = O.rms_norm(x, np.ones(32), 0.0)
    np.testing.assert_allclose(np.sqrt(np.mean(out ** 2, axis=1)), 1.0, rtol=1e-14)
    np.testing.assert_allclose(O.rms_norm(7.5 * x, np.ones(32), 0.0), out, rtol=1e-13)


def test_rope_matches_complex_rotation():
    """Rotate-half RoPE equals multiplication of x[i] + 1j x[i+hd/2] by exp(1j p theta_i)."""
    rng = np.random.default_rng(1)
    x = rng.standard_normal((6, 3, 16))
    pos = np.array([0, 1, 5, 100, 4097, 131087])
    # the two compute theta_i by different fp64 routes; at position p an angle differs
    # by at most about p * 1e-15 rad, i.e. 1.3e-10 at p = 131087
    np.testing.assert_allclose(O.rope(x, pos, 10000.0), ind._rope_complex(x, pos, 10000.0),
                               rtol=0, atol=1e-9)


def test_rope_closed_forms():
    # position 0 is the identity
    x = np.arange(8, dtype=np.float64).reshape(1, 1, 8)
    np.testing.assert_array_equal(O.rope(x, np.array([0]), 10000.0), x)
    # hd = 2: a single pair rotated by exactly `pos` radians (theta_0 = 1)
    v = np.array([[[1.0, 0.0]]])
    r = O.rope(v, np.array([3]), 10000.0)[0, 0]
    np.testing.assert_allclose(r, [math.cos(3), math.sin(3)], atol=1e-15)
    # norm preservation
    rng = np.random.default_rng(2)
    y = rng.standard_normal((4, 2, 32))
    ry = O.rope(y, np.array([1, 10, 1000, 100000]), 10000.0)
    np.testing.assert_allclose(np.linalg.norm(ry, axis=-1), np.linalg.norm(y, axis=-1), rtol=1e-13)
    # second pair of hd = 4 turns at base^(-1/2) per position
    v4 = np.array([[[0.0, 1.0, 0.0, 0.0]]])
    r4 = O.rope(v4, np.array([2]), 100.0)[0, 0]
    ang = 2 * 100.0 ** -0.5
    np.testing.assert_allclose(r4, [0, math.cos(ang), 0, math.sin(ang)], atol=1e-15)


def test_silu_closed_form():
    """silu(z) = z * sigmoid(z): silu(0) = 0, silu(ln 3) = 0.75 ln 3, silu(-ln 3) = -0.25 ln 3."""
    l3 = math.log(3.0)
    np.testing.assert_allclose(O.silu(np.array([0.0, l3, -l3])), [0.0, 0.75 * l3, -0.25 * l3],
                               rtol=1e-15, atol=1e-300)


# ---------------------------------------------------------------- attention (Eq. 1-3)

def test_softmax_rows_sum_to_one_and_mask():
    rng = np.random.default_rng(3)
    d, n_q, n_kv, hd, inter, k, N = 16, 4, 2, 4, 24, 4, 11
    W = rand_weights(rng, d, n_q, n_kv, hd, inter, 2)
    kc, vc = rng.standard_normal((2, n_kv, N, hd))
    out = O.probe_sequence(kc, vc, 0.3 * rng.standard_normal((k, d)), W,
                           O.HeadShape(n_q, n_kv, hd, 1e-6, 10000.0))
    for p in out["probs"]:
        np.testing.assert_allclose(p.sum(axis=1), 1.0, atol=1e-13)
        # soft key j' is invisible to soft query j < j'
        soft = p[:, N:]
        assert np.all(soft[np.triu_indices(k, 1)] == 0.0)
        assert np.all(np.diag(soft) > 0.0)


def test_constant_values_give_that_constant():
    """If every visible value row equals c, the attention output is c (weights sum to 1)."""
    rng = np.random.default_rng(4)
    k, n_q, n_kv, hd, N = 3, 4, 2, 8, 10
    c = rng.standard_normal(hd)
    o, _ = O.cached_attention(rng.standard_normal((k, n_q, hd)), rng.standard_normal((n_kv, N, hd)),
                              np.broadcast_to(c, (n_kv, N, hd)), rng.standard_normal((k, n_kv, hd)),
                              np.broadcast_to(c, (k, n_kv, hd)))
    np.testing.assert_allclose(o, np.broadcast_to(c, o.shape), atol=1e-13)


def test_identical_keys_give_mean_of_visible_values():
    """Equal scores: soft query j averages the N cached values and soft values 0..j."""
    rng = np.random.default_rng(5)
    k, n_q, n_kv, hd, N = 3, 2, 1, 4, 5
    key = rng.standard_normal(hd)
    vc = rng.standard_normal((n_kv, N, hd))
    vs = rng.standard_normal((k, n_kv, hd))
    o, _ = O.cached_attention(rng.standard_normal((k, n_q, hd)), np.broadcast_to(key, (n_kv, N, hd)),
                              vc, np.broadcast_to(key, (k, n_kv, hd)), vs)
    for j in range(k):
        expect = (vc[0].sum(axis=0) + vs[: j + 1, 0].sum(axis=0)) / (N + j + 1)
        for h in range(n_q):
            np.testing.assert_allclose(o[j, h], expect, atol=1e-13)


def test_huge_scores_select_the_top_key():
    """Scores of order 1e4: the softmax is one-hot on the highest-scoring visible key
    (exp of the others underflows to 0), so the output is that key's value.  A
    softmax without max subtraction overflows here."""
    rng = np.random.default_rng(13)
    k, n_q, n_kv, hd, N = 2, 2, 1, 4, 6
    kc = rng.standard_normal((n_kv, N, hd))
    vc = rng.standard_normal((n_kv, N, hd))
    ks = rng.standard_normal((k, n_kv, hd))
    vs = rng.standard_normal((k, n_kv, hd))
    q = 5e3 * rng.standard_normal((k, n_q, hd))
    o, _ = O.cached_attention(q, kc, vc, ks, vs)
    for j in range(k):
        keys = np.concatenate([kc[0], ks[: j + 1, 0]])
        vals = np.concatenate([vc[0], vs[: j + 1, 0]])
        for h in range(n_q):
            np.testing.assert_allclose(o[j, h], vals[np.argmax(keys @ q[j, h])], atol=1e-12)


@pytest.mark.parametrize("shape", SHAPES)
def test_cached_path_equals_full_recompute(shape):
    """Eq. 1-3: attention of the appended rows over [cached K/V; new K/V] equals the
    decoder layer run over the whole sequence with the soft rows appended
    (positions N..N+k-1, causal mask)."""
    d, n_q, n_kv, hd, inter, k, N = shape
    rng = np.random.default_rng(hash(shape) % (1 << 32))
    W = rand_weights(rng, d, n_q, n_kv, hd, inter, 3, bias=True)
    x_ctx = rng.standard_normal((N, d))
    x_soft = 0.5 * rng.standard_normal((k, d))
    eps, base = 1e-6, 10000.0
    full = ind.full_layer(np.concatenate([x_ctx, x_soft]), W, n_q, n_kv, hd, eps, base)
    kc = full["k_rot"][:, :N]
    vc = full["v"][:, :N]
    for pool in ("last", "mean"):
        out = O.probe_sequence(kc, vc, x_soft, W, O.HeadShape(n_q, n_kv, hd, eps, base, pool))
        np.testing.assert_allclose(out["o"], full["attn"][N:], rtol=0, atol=1e-12)
        np.testing.assert_allclose(out["a"], full["a"][N:], rtol=0, atol=1e-12)
        np.testing.assert_allclose(out["y"], full["y"][N:], rtol=0, atol=1e-12)
        np.testing.assert_allclose(out["f"], full["f"][N:], rtol=0, atol=1e-12)
        f_soft = full["f"][N:]
        pooled = f_soft[-1] if pool == "last" else f_soft.mean(axis=0)
        np.testing.assert_allclose(out["logits"], np.asarray(W["w_cls"]) @ pooled + W["b_cls"],
                                   rtol=0, atol=1e-12)


def test_full_recompute_is_shift_invariant():
    """RoPE makes scores depend on position differences only: shifting every
    position of the whole sequence leaves the layer's outputs unchanged."""
    rng = np.random.default_rng(6)
    d, n_q, n_kv, hd, inter = 16, 4, 2, 8, 20
    W = rand_weights(rng, d, n_q, n_kv, hd, inter, 2)
    x = rng.standard_normal((9, d))
    f0 = ind.full_layer(x, W, n_q, n_kv, hd, 1e-6, 10000.0)["f"]
    f1 = ind.full_layer(x, W, n_q, n_kv, hd, 1e-6, 10000.0, pos_offset=37)["f"]
    np.testing.assert_allclose(f0, f1, atol=1e-11)


def test_k1_reduces_to_single_query_decode():
    """With k = 1 (SP-1, Sec. 3.2) each query head does ordinary single-query decode
    attention over the N cached keys plus its own key."""
    rng = np.random.default_rng(7)
    d, n_q, n_kv, hd, inter, N = 12, 4, 2, 6, 10, 6
    W = rand_weights(rng, d, n_q, n_kv, hd, inter, 2)
    kc, vc = rng.standard_normal((2, n_kv, N, hd))
    out = O.probe_sequence(kc, vc, rng.standard_normal((1, d)), W, O.HeadShape(n_q, n_kv, hd))
    G = n_q // n_kv
    for h in range(n_q):
        g = h // G
        keys = list(kc[g]) + [out["k_rot"][0, g]]
        vals = list(vc[g]) + [out["v"][0, g]]
        ref = ind.textbook_decode(out["q_rot"][0, h], keys, vals)
        np.testing.assert_allclose(out["o"][0, h * hd:(h + 1) * hd], ref, atol=1e-13)


def test_mqa_and_mha_do_not_depend_on_grouping_convention():
    """With one KV head (MQA) every query head uses it; with G = 1 (MHA) head h uses KV
    head h.  Both cases are fixed without any grouping convention."""
    rng = np.random.default_rng(8)
    k, hd, N = 2, 4, 5
    for n_q, n_kv in ((6, 1), (3, 3)):
        q = rng.standard_normal((k, n_q, hd))
        kc, vc = rng.standard_normal((2, n_kv, N, hd))
        ks, vs = rng.standard_normal((2, k, n_kv, hd))
        o, _ = O.cached_attention(q, kc, vc, ks, vs)
        for h in range(n_q):
            g = 0 if n_kv == 1 else h
            for j in range(k):
                keys = list(kc[g]) + [ks[t, g] for t in range(j + 1)]
                vals = list(vc[g]) + [vs[t, g] for t in range(j + 1)]
                np.testing.assert_allclose(o[j, h], ind.textbook_decode(q[j, h], keys, vals), atol=1e-13)


# ---------------------------------------------------------------- closed-form whole forward

def test_hand_worked_forward():
    """A case worked by hand.  d = hd = 4, one head, k = 2 soft rows, N = 2, eps = 0.
    W_q = 0 makes every score 0, so each soft query averages the values it sees;
    W_gate = 0 makes the MLP output 0 (silu(0) = 0).
      x0 = (2,2,2,2) -> u0 = (1,1,1,1);  x1 = (0,0,0,4) -> u1 = (0,0,0,2);  W_v = I
      cached V = (3,0,0,0), (0,3,0,0)
      o0 = mean of cache + v0 = (4/3, 4/3, 1/3, 1/3)
      o1 = mean of cache + v0 + v1 = (1, 1, 1/4, 3/4)
      W_o = I: a0 = (10/3, 10/3, 7/3, 7/3), a1 = (1, 1, 1/4, 19/4); y = a
      f_j = a_j / rms(a_j): rms(a1)^2 = 24.625/4, rms(a0)^2 = 298/36
      W_cls = [[1,0,0,0],[0,0,0,1]]"""
    d = hd = 4
    Z, I4 = np.zeros((4, 4)), np.eye(4)
    W = {"in_norm": np.ones(d), "w_q": Z, "w_k": Z, "w_v": I4, "w_o": I4, "post_norm": np.ones(d),
         "w_gate": np.zeros((3, d)), "w_up": np.ones((3, d)), "w_down": np.ones((d, 3)),
         "final_norm": np.ones(d), "w_cls": np.array([[1.0, 0, 0, 0], [0, 0, 0, 1.0]]), "b_cls": None}
    kc = np.random.default_rng(9).standard_normal((1, 2, hd))   # irrelevant: q = 0
    vc = np.array([[[3.0, 0, 0, 0], [0, 3.0, 0, 0]]])
    x = np.array([[2.0, 2, 2, 2], [0, 0, 0, 4.0]])
    r1 = math.sqrt(24.625 / 4)
    r0 = math.sqrt(298.0 / 36)
    out = O.probe_sequence(kc, vc, x, W, O.HeadShape(1, 1, hd, 0.0, 10000.0, "last"))
    np.testing.assert_allclose(out["o"], [[4 / 3, 4 / 3, 1 / 3, 1 / 3], [1, 1, 0.25, 0.75]], atol=1e-15)
    np.testing.assert_allclose(out["logits"], [1 / r1, 4.75 / r1], rtol=1e-14)
    out = O.probe_sequence(kc, vc, x, W, O.HeadShape(1, 1, hd, 0.0, 10000.0, "mean"))
    np.testing.assert_allclose(out["logits"], [(10 / 3 / r0 + 1 / r1) / 2, (7 / 3 / r0 + 4.75 / r1) / 2],
                               rtol=1e-14)


def test_single_soft_row_without_context_attends_to_itself():
    """N = 0, k = 1: softmax over one key is 1, so the attention output is v_0 = W_v u_0
    whatever W_q and W_k are."""
    rng = np.random.default_rng(10)
    d, n_q, n_kv, hd = 8, 2, 1, 4
    W = rand_weights(rng, d, n_q, n_kv, hd, 6, 2)
    x = rng.standard_normal((1, d))
    out = O.probe_sequence(np.zeros((n_kv, 0, hd)), np.zeros((n_kv, 0, hd)), x, W,
                           O.HeadShape(n_q, n_kv, hd))
    v0 = O.rms_norm(x, W["in_norm"], 1e-6) @ W["w_v"].T
    np.testing.assert_allclose(out["o"], np.tile(v0, (1, n_q)), atol=1e-14)


# ---------------------------------------------------------------- head and batch

def test_linear_head():
    """Sec. 3.2: the head is linear.  C = 1 gives z = w.a; permuting W_cls rows
    permutes the logits; a bias adds."""
    rng = np.random.default_rng(11)
    d, n_q, n_kv, hd, inter, k, N = 16, 4, 2, 4, 24, 2, 6
    W = rand_weights(rng, d, n_q, n_kv, hd, inter, 4)
    kc, vc = rng.standard_normal((2, n_kv, N, hd))
    x = rng.standard_normal((k, d))
    shape = O.HeadShape(n_q, n_kv, hd)
    base = O.probe_sequence(kc, vc, x, W, shape)
    W1 = dict(W, w_cls=W["w_cls"][2:3])
    np.testing.assert_allclose(O.probe_sequence(kc, vc, x, W1, shape)["logits"],
                               [W["w_cls"][2] @ base["pooled"]], rtol=1e-14)
    perm = [3, 0, 2, 1]
    Wp = dict(W, w_cls=W["w_cls"][perm])
    np.testing.assert_allclose(O.probe_sequence(kc, vc, x, Wp, shape)["logits"], base["logits"][perm],
                               rtol=1e-14)
    b = np.array([1.0, -2.0, 0.5, 0.0])
    np.testing.assert_allclose(O.probe_sequence(kc, vc, x, dict(W, b_cls=b), shape)["logits"],
                               base["logits"] + b, rtol=1e-14)


def test_batch_order_invariance():
    """Sec. 3.3: each sequence is classified on its own; reordering the batch
    reorders the logits."""
    rng = np.random.default_rng(12)
    d, n_q, n_kv, hd, inter, k = 16, 4, 2, 4, 24, 3
    W = rand_weights(rng, d, n_q, n_kv, hd, inter, 2)
    x = rng.standard_normal((k, d))
    kv = [tuple(rng.standard_normal((2, n_kv, n, hd))) for n in (0, 3, 17, 9)]
    shape = O.HeadShape(n_q, n_kv, hd)
    ref = O.probe_batch(kv, x, W, shape)
    perm = [2, 0, 3, 1]
    np.testing.assert_array_equal(O.probe_batch([kv[i] for i in perm], x, W, shape), ref[perm])


def test_tasks_are_independent_probes():
    """Sec. 3.3: classifiers sharing one cache are independent: task t's logits are
    the single-task probe's with its own soft prompt and head, whatever the other
    tasks hold; a permutation of the tasks permutes the output."""
    rng = np.random.default_rng(51)
    d, n_q, n_kv, hd, inter, k, C, T = 16, 4, 2, 4, 20, 3, 2, 3
    W = rand_weights(rng, d, n_q, n_kv, hd, inter, C)
    kvs = [tuple(rng.standard_normal((2, n_kv, n, hd))) for n in (4, 0, 7)]
    soft = rng.standard_normal((T, k, d))
    wc = rng.standard_normal((T, C, d))
    bc = rng.standard_normal((T, C))
    hs = O.HeadShape(n_q, n_kv, hd)
    out = O.probe_batch_tasks(kvs, soft, wc, bc, W, hs)
    assert out.shape == (3, T, C)
    for t in range(T):
        single = O.probe_batch(kvs, soft[t], dict(W, w_cls=wc[t], b_cls=bc[t]), hs)
        np.testing.assert_array_equal(out[:, t], single)
    soft2 = soft.copy()
    soft2[1] = -soft2[1]
    out2 = O.probe_batch_tasks(kvs, soft2, wc, bc, W, hs)
    np.testing.assert_array_equal(out2[:, 0], out[:, 0])
    np.testing.assert_array_equal(out2[:, 2], out[:, 2])
    perm = [2, 0, 1]
    np.testing.assert_array_equal(O.probe_batch_tasks(kvs, soft[perm], wc[perm], bc[perm], W, hs), out[:, perm])


def test_lm_head_readout_reads_only_the_label_rows():
    """Sec. 6.7 / Table 7: the frozen-LM-head read-out scores the pooled state with
    the rows of the label tokens only.  It equals the linear head made of those
    rows; the other vocabulary rows have no effect; swapping the two labels
    negates the yes/no score."""
    rng = np.random.default_rng(61)
    d, n_q, n_kv, hd, inter, k, V = 16, 4, 2, 4, 20, 3, 50
    W = rand_weights(rng, d, n_q, n_kv, hd, inter, 2)
    vocab = rng.standard_normal((V, d))
    kc, vc = rng.standard_normal((2, n_kv, 6, hd))
    soft = rng.standard_normal((k, d))
    hs = O.HeadShape(n_q, n_kv, hd)
    yes, no = 17, 42
    lm = O.probe_sequence(kc, vc, soft, dict(W, w_cls=vocab, cls_rows=[yes, no]), hs)
    lin = O.probe_sequence(kc, vc, soft, dict(W, w_cls=vocab[[yes, no]]), hs)
    np.testing.assert_array_equal(lm["logits"], lin["logits"])
    other = vocab.copy()
    other[[i for i in range(V) if i not in (yes, no)]] *= -3.0
    np.testing.assert_array_equal(
        O.probe_sequence(kc, vc, soft, dict(W, w_cls=other, cls_rows=[yes, no]), hs)["logits"], lm["logits"])
    sw = O.probe_sequence(kc, vc, soft, dict(W, w_cls=vocab, cls_rows=[no, yes]), hs)["logits"]
    assert sw[0] - sw[1] == -(lm["logits"][0] - lm["logits"][1])
    # tasks reading different rows of one shared vocabulary matrix
    rows = np.array([[yes, no], [3, 4]])
    out = O.probe_batch_tasks([(kc, vc)], np.stack([soft, soft]), vocab, None, W, hs, cls_rows=rows)
    np.testing.assert_array_equal(out[0, 0], lm["logits"])
    np.testing.assert_array_equal(out[0, 1], O.probe_sequence(kc, vc, soft, dict(W, w_cls=vocab[[3, 4]]), hs)["logits"])
