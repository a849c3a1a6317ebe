"""Pins of the recursive SP-k oracle (Sec. 3.1 MTP input fusion, Sec. 3.2
recursive soft prompts) against independent statements (CPU only).

* the per-step recomputation without a cache (``independent.draft_without_cache``)
  fixes the positions, the soft keys each step sees, the residual from the
  fused row and the hand-over of the final-normed state;
* the fusion special cases fix which half of w_fc multiplies which input:
  w_fc = [0 | I] ignores the hidden state and reduces every step to a row of
  one causal pass over RMSNorm(e; gamma_e); w_fc = [I | 0] ignores the soft
  prompt;
* RMSNorm makes the result invariant to positive scaling of either input
  (eps = 0).
"""
from __future__ import annotations

import numpy as np
import pytest

from oracle import probe as O
from tests import independent as ind
from tests.test_oracle_pins import rand_weights

SHAPES = [
    # (d, n_q, n_kv, hd, inter, k, N)
    (16, 4, 2, 4, 24, 3, 7),     # GQA, group 2
    (24, 6, 2, 8, 20, 4, 0),     # empty context
    (16, 2, 2, 8, 12, 1, 5),     # MHA, SP-1
    (20, 5, 1, 4, 16, 5, 9),     # MQA, SP-5
]


def fusion_weights(rng, d, gain_std=0.1, std=0.3):
    return {"fc_norm_h": 1 + gain_std * rng.standard_normal(d),
            "fc_norm_e": 1 + gain_std * rng.standard_normal(d),
            "w_fc": std * rng.standard_normal((d, 2 * d))}


def setup(shape, seed, eps=1e-6):
    d, n_q, n_kv, hd, inter, k, N = shape
    rng = np.random.default_rng(seed)
    W = rand_weights(rng, d, n_q, n_kv, hd, inter, 3, bias=True)
    W.update(fusion_weights(rng, d))
    x_ctx = rng.standard_normal((N, d))
    e = 0.5 * rng.standard_normal((k, d))
    h_last = 2.0 * rng.standard_normal(d)
    full_ctx = ind.full_layer(x_ctx, W, n_q, n_kv, hd, eps, 10000.0) if N else None
    kc = full_ctx["k_rot"] if N else np.zeros((n_kv, 0, hd))
    vc = full_ctx["v"] if N else np.zeros((n_kv, 0, hd))
    return W, x_ctx, e, h_last, kc, vc


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("pool", ["last", "mean"])
def test_recursive_equals_drafting_without_cache(shape, pool):
    """Sec. 3.2: each step's output equals re-running the layer over the whole
    sequence with the fused rows of the steps so far appended (positions N..N+t,
    causal), fed back step by step."""
    d, n_q, n_kv, hd, inter, k, N = shape
    W, x_ctx, e, h_last, kc, vc = setup(shape, hash(shape) % (1 << 32))
    out = O.probe_sequence_recursive(kc, vc, e, h_last, W, O.HeadShape(n_q, n_kv, hd, 1e-6, 10000.0, pool))
    ref = ind.draft_without_cache(x_ctx, e, h_last, W, n_q, n_kv, hd, 1e-6, 10000.0)
    np.testing.assert_allclose(out["x"], ref["x"], rtol=0, atol=1e-12)
    np.testing.assert_allclose(out["f"], ref["f"], rtol=0, atol=1e-12)
    last = ref["last"]
    np.testing.assert_allclose(out["a"][-1], last["a"][-1], rtol=0, atol=1e-12)
    np.testing.assert_allclose(out["y"][-1], last["y"][-1], rtol=0, atol=1e-12)
    pooled = ref["f"][-1] if pool == "last" else ref["f"].mean(axis=0)
    np.testing.assert_allclose(out["logits"], W["w_cls"] @ pooled + W["b_cls"], rtol=0, atol=1e-12)


@pytest.mark.parametrize("shape", SHAPES)
def test_embedding_half_only_is_one_causal_pass(shape):
    """w_fc = [0 | I]: every fused row is RMSNorm(e_t; gamma_e) whatever the
    hidden state, so the k steps are the k rows of one causal pass of the layer
    over [context; RMSNorm(E; gamma_e)] (Eq. 1-3), and h_last has no effect."""
    d, n_q, n_kv, hd, inter, k, N = shape
    W, x_ctx, e, h_last, kc, vc = setup(shape, 11 + k)
    W["w_fc"] = np.concatenate([np.zeros((d, d)), np.eye(d)], axis=1)
    hs = O.HeadShape(n_q, n_kv, hd, 1e-6, 10000.0, "mean")
    out = O.probe_sequence_recursive(kc, vc, e, h_last, W, hs)
    rows = ind._rms(e, W["fc_norm_e"], 1e-6)
    full = ind.full_layer(np.concatenate([x_ctx, rows]), W, n_q, n_kv, hd, 1e-6, 10000.0)
    np.testing.assert_allclose(out["f"], full["f"][N:], rtol=0, atol=1e-12)
    np.testing.assert_allclose(out["y"], full["y"][N:], rtol=0, atol=1e-12)
    other = O.probe_sequence_recursive(kc, vc, e, -3.0 * h_last + 1.0, W, hs)
    np.testing.assert_allclose(other["logits"], out["logits"], rtol=0, atol=1e-12)


@pytest.mark.parametrize("shape", SHAPES)
def test_hidden_half_only_ignores_the_soft_prompt(shape):
    """w_fc = [I | 0]: the soft prompt has no effect, and the first step's fused
    row is RMSNorm(h_last; gamma_h): SP-1 is then one decode step of the layer on
    that row."""
    d, n_q, n_kv, hd, inter, k, N = shape
    W, x_ctx, e, h_last, kc, vc = setup(shape, 23 + k)
    W["w_fc"] = np.concatenate([np.eye(d), np.zeros((d, d))], axis=1)
    hs = O.HeadShape(n_q, n_kv, hd, 1e-6, 10000.0, "last")
    out = O.probe_sequence_recursive(kc, vc, e, h_last, W, hs)
    other = O.probe_sequence_recursive(kc, vc, np.flip(e, 0) * 7.0 - 1.0, h_last, W, hs)
    np.testing.assert_allclose(other["f"], out["f"], rtol=0, atol=1e-12)
    row = ind._rms(h_last[None], W["fc_norm_h"], 1e-6)
    full = ind.full_layer(np.concatenate([x_ctx, row]), W, n_q, n_kv, hd, 1e-6, 10000.0)
    np.testing.assert_allclose(out["f"][0], full["f"][N], rtol=0, atol=1e-12)


def test_scaling_either_input_changes_nothing():
    """Both inputs enter only through RMSNorm, so with eps = 0 scaling h_last or
    any soft vector by a positive factor leaves every step unchanged."""
    shape = (16, 4, 2, 4, 24, 3, 6)
    d, n_q, n_kv, hd, inter, k, N = shape
    W, x_ctx, e, h_last, kc, vc = setup(shape, 31)
    hs = O.HeadShape(n_q, n_kv, hd, 0.0, 10000.0, "mean")
    base = O.probe_sequence_recursive(kc, vc, e, h_last, W, hs)
    scaled = O.probe_sequence_recursive(kc, vc, e * np.array([[3.0], [0.25], [17.0]]), 40.0 * h_last, W, hs)
    np.testing.assert_allclose(scaled["f"], base["f"], rtol=0, atol=1e-12)
    np.testing.assert_allclose(scaled["logits"], base["logits"], rtol=0, atol=1e-12)


def test_steps_are_causal():
    """A later soft vector cannot change earlier steps (each step sees only the
    soft keys of steps up to itself)."""
    shape = (16, 4, 2, 4, 24, 4, 5)
    d, n_q, n_kv, hd, inter, k, N = shape
    W, x_ctx, e, h_last, kc, vc = setup(shape, 37)
    hs = O.HeadShape(n_q, n_kv, hd)
    base = O.probe_sequence_recursive(kc, vc, e, h_last, W, hs)
    e2 = e.copy()
    e2[2:] = -e2[2:] + 0.3
    changed = O.probe_sequence_recursive(kc, vc, e2, h_last, W, hs)
    np.testing.assert_allclose(changed["f"][:2], base["f"][:2], rtol=0, atol=0)
    assert np.max(np.abs(changed["f"][2:] - base["f"][2:])) > 1e-3


def test_batch_is_a_loop_over_sequences():
    """Sec. 3.3: sequences are classified independently; each uses its own h_last."""
    rng = np.random.default_rng(41)
    d, n_q, n_kv, hd, inter, k = 16, 4, 2, 4, 24, 2
    W = rand_weights(rng, d, n_q, n_kv, hd, inter, 2)
    W.update(fusion_weights(rng, d))
    kvs = [tuple(rng.standard_normal((2, n_kv, n, hd))) for n in (3, 0, 6)]
    e = rng.standard_normal((k, d))
    h = rng.standard_normal((3, d))
    hs = O.HeadShape(n_q, n_kv, hd)
    logits = O.probe_batch_recursive(kvs, e, h, W, hs)
    rev = O.probe_batch_recursive(kvs[::-1], e, h[::-1], W, hs)
    np.testing.assert_array_equal(rev, logits[::-1])
    for b in range(3):
        one = O.probe_sequence_recursive(kvs[b][0], kvs[b][1], e, h[b], W, hs)["logits"]
        np.testing.assert_array_equal(one, logits[b])


def test_eagle3_input_selects_and_scales():
    """Sec. 3.1 (Eagle3): the first hidden state is a projection of three base-model
    hidden states.  Selecting one of them ([0 | 0 | I], [I | 0 | 0]) is the MTP
    recursion on that state; with eps = 0 a positive common scale of the three
    states changes nothing (they enter through RMSNorm after a linear map)."""
    shape = (16, 4, 2, 4, 24, 3, 6)
    d, n_q, n_kv, hd, inter, k, N = shape
    W, x_ctx, e, h_last, kc, vc = setup(shape, 43)
    rng = np.random.default_rng(44)
    h3 = rng.standard_normal((3, d))
    hs = O.HeadShape(n_q, n_kv, hd, 1e-6, 10000.0, "mean")
    Z, I = np.zeros((d, d)), np.eye(d)
    for sel, blocks in ((2, [Z, Z, I]), (0, [I, Z, Z])):
        got = O.probe_sequence_recursive(kc, vc, e, h3.reshape(-1), dict(W, w_hidden_fuse=np.concatenate(blocks, 1)), hs)
        ref = ind.draft_without_cache(x_ctx, e, h3[sel], W, n_q, n_kv, hd, 1e-6, 10000.0)
        np.testing.assert_allclose(got["f"], ref["f"], rtol=0, atol=1e-12)
    hs0 = O.HeadShape(n_q, n_kv, hd, 0.0, 10000.0, "mean")
    Wf = dict(W, w_hidden_fuse=0.3 * rng.standard_normal((d, 3 * d)))
    a = O.probe_sequence_recursive(kc, vc, e, h3.reshape(-1), Wf, hs0)
    b = O.probe_sequence_recursive(kc, vc, e, 250.0 * h3.reshape(-1), Wf, hs0)
    np.testing.assert_allclose(b["logits"], a["logits"], rtol=0, atol=1e-11)
