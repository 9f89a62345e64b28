"""Pins of the query front-end oracle (module ``Q``): a hand-worked fixture, brute force with
explicit loops, closed forms and invariants of the convolution, the query linear and LayerNorm.

Each pin raises AssertionError on a mismatch and takes the oracle module as an argument, so the
mutation tests can run it against copies with planted mistakes.
"""
from __future__ import annotations

import json
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _fixture():
    with open(os.path.join(GOLDEN, "query_front_end_d2.json")) as f:
        return json.load(f)


def pin_golden_front_end(Q):
    g = _fixture()
    x, hist, w = np.array(g["x"]), np.array(g["hist"]), np.array(g["conv_w"])
    assert np.array_equal(Q.causal_conv(x, w, hist), np.array(g["expect_conv"]))
    Wr, Wc = np.array(g["W_q_row"]), np.array(g["W_q_col"])
    gr, br = np.array(g["gamma_row"]), np.array(g["beta_row"])
    gc, bc = np.array(g["gamma_col"]), np.array(g["beta_col"])
    # shared query: one query serves both key sets
    qr, qc = Q.query_front_end(x, w, Wr, gr[None, None], br[None, None], heads=1, dk=4,
                               shared=True, hist=hist, eps=0.0)
    assert np.allclose(qr[:, 0], g["expect_q_row"], rtol=1e-14, atol=1e-14)
    assert np.array_equal(qr, qc)
    # separate row and column queries: W_q = [row block | column block]
    qr, qc = Q.query_front_end(x, w, np.concatenate([Wr, Wc], axis=1),
                               np.stack([gr, gc])[:, None], np.stack([br, bc])[:, None], heads=1,
                               dk=4, shared=False, hist=hist, eps=0.0)
    assert np.allclose(qr[:, 0], g["expect_q_row"], rtol=1e-14, atol=1e-14)
    assert np.allclose(qc[0, 0], g["expect_q_col_l0"], rtol=1e-14, atol=1e-14)
    K = Q.key_norm(np.array(g["K"]), np.ones((1, 4)), np.zeros((1, 4)), eps=0.0)
    assert np.allclose(K, g["expect_K"], rtol=1e-14, atol=1e-14)


def _conv_loops(x, w, hist):
    """The convolution as explicit loops over (sequence, token, channel, tap)."""
    B, L, d = x.shape
    kc = w.shape[0]
    y = np.zeros((B, L, d))
    for b in range(B):
        for l in range(L):
            for c in range(d):
                s = 0.0
                for j in range(kc):
                    src = l - j
                    v = x[b, src, c] if src >= 0 else (hist[b, kc - 1 + src, c] if hist is not None else 0.0)
                    s += w[j, c] * v
                y[b, l, c] = s
    return y


def pin_conv_brute_force(Q, seeds=range(6)):
    for seed in seeds:
        rng = np.random.default_rng(seed)
        B, L, d, kc = 2, 1 + seed % 5, 3, 1 + seed % 4
        x = rng.standard_normal((B, L, d))
        w = rng.standard_normal((kc, d))
        hist = rng.standard_normal((B, kc - 1, d)) if seed % 2 else None
        assert np.allclose(Q.causal_conv(x, w, hist), _conv_loops(x, w, hist), rtol=1e-13, atol=1e-13)


def pin_conv_closed_forms(Q):
    rng = np.random.default_rng(7)
    x = rng.standard_normal((2, 6, 5))
    hist = rng.standard_normal((2, 3, 5))
    # a delta at tap 0 is the identity; a delta at tap s shifts by s (history fills the start)
    for s in range(4):
        w = np.zeros((4, 5))
        w[s] = 1.0
        y = Q.causal_conv(x, w, hist)
        full = np.concatenate([hist, x], axis=1)
        assert np.array_equal(y, full[:, 3 - s: 3 - s + 6])
    # a constant sequence (history included) gives the column sums of the taps
    c = np.full((1, 4, 5), 2.5)
    w = rng.standard_normal((3, 5))
    assert np.allclose(Q.causal_conv(c, w, np.full((1, 2, 5), 2.5)), 2.5 * w.sum(axis=0), rtol=1e-14)


def pin_conv_chunks(Q):
    """Causality: the convolution of a whole sequence equals that of its chunks, each given the
    K_c - 1 tokens before it as history (decode steps and prefill chunks agree)."""
    rng = np.random.default_rng(3)
    B, L, d, kc = 2, 9, 4, 4
    x = rng.standard_normal((B, L, d))
    w = rng.standard_normal((kc, d))
    whole = Q.causal_conv(x, w, None)
    padded = np.concatenate([np.zeros((B, kc - 1, d)), x], axis=1)
    for cut in ((0, 1), (1, 5), (5, 9), (3, 4)):
        a, b = cut
        part = Q.causal_conv(x[:, a:b], w, padded[:, a: a + kc - 1])
        assert np.allclose(part, whole[:, a:b], rtol=1e-14, atol=1e-14)


def pin_layer_norm_invariants(Q):
    rng = np.random.default_rng(11)
    v = rng.standard_normal((5, 3, 16)) * 3.0 + 1.5
    one, zero = np.ones(16), np.zeros(16)
    y = Q.layer_norm(v, one, zero, 0.0)
    assert np.allclose(y.mean(axis=-1), 0.0, atol=1e-13)
    assert np.allclose((y ** 2).mean(axis=-1), 1.0, rtol=1e-13)          # population variance
    # invariant under a positive scale and a shift of each vector
    assert np.allclose(Q.layer_norm(4.0 * v - 7.0, one, zero, 0.0), y, rtol=1e-12, atol=1e-12)
    # gamma scales and beta shifts elementwise
    g, b = rng.standard_normal(16), rng.standard_normal(16)
    assert np.allclose(Q.layer_norm(v, g, b, 0.0), y * g + b, rtol=1e-13, atol=1e-13)
    # epsilon adds to the variance
    eps = 0.25
    var = ((v - v.mean(-1, keepdims=True)) ** 2).mean(-1, keepdims=True)
    assert np.allclose(Q.layer_norm(v, one, zero, eps), y * np.sqrt(var / (var + eps)), rtol=1e-13)


def pin_query_linear_one_hot(Q):
    rng = np.random.default_rng(5)
    W = rng.standard_normal((6, 10))
    assert np.array_equal(Q.query_linear(np.eye(6), W), W)
    y = rng.standard_normal((4, 6))
    # linear in its input
    assert np.allclose(Q.query_linear(2.0 * y, W), 2.0 * Q.query_linear(y, W), rtol=1e-14)


def pin_front_end_layout(Q):
    """Heads and axes take consecutive D_k blocks of the query linear's output, in the order
    (axis, head); a head whose W_q block is another head's gives that head's query."""
    rng = np.random.default_rng(9)
    B, L, d, H, dk = 2, 3, 5, 3, 4
    x = rng.standard_normal((B, L, d))
    w = rng.standard_normal((2, d))
    W = rng.standard_normal((d, 2 * H * dk))
    g = rng.standard_normal((2, H, dk))
    b = rng.standard_normal((2, H, dk))
    qr, qc = Q.query_front_end(x, w, W, g, b, heads=H, dk=dk, shared=False, eps=1e-5)
    y = Q.causal_conv(x, w).reshape(B * L, d)
    for a, q in ((0, qr), (1, qc)):
        for h in range(H):
            blk = W[:, (a * H + h) * dk:(a * H + h + 1) * dk]
            want = Q.layer_norm(y @ blk, g[a, h], b[a, h], 1e-5)
            assert np.allclose(q[:, h], want, rtol=1e-12, atol=1e-12)


def pin_key_norm_rows(Q):
    rng = np.random.default_rng(2)
    K = rng.standard_normal((2, 7, 8)) * 2.0 + 0.3
    g, b = np.ones((2, 8)), np.zeros((2, 8))
    Kn = Q.key_norm(K, g, b, eps=0.0)
    assert np.allclose(Kn.mean(-1), 0.0, atol=1e-13) and np.allclose((Kn ** 2).mean(-1), 1.0, rtol=1e-13)
    g2 = rng.standard_normal((2, 8))
    Kg = Q.key_norm(K, g2, b, eps=0.0)
    assert np.allclose(Kg, Kn * g2[:, None, :], rtol=1e-13, atol=1e-13)    # per-head gamma


QUERY_PINS = [pin_golden_front_end, pin_conv_brute_force, pin_conv_closed_forms, pin_conv_chunks,
              pin_layer_norm_invariants, pin_query_linear_one_hot, pin_front_end_layout,
              pin_key_norm_rows]
