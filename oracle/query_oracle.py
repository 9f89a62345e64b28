"""UltraMem query front-end and key normalisation: a plain CPU oracle in fp64.  TEST
INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline leg may use this
module.  It shares no code with the GPU library.

The memory layer turns hidden states into the two axis queries with three of the adjustments
Sec. 3.2 ("Improve PKM with a bag of tricks") lists, in this order:

1. causal depthwise convolution   Trick 4: added before the query linear layer
2. query linear                   the linear layer q(x) of eq. (2) that maps D_i to D_k (per head;
                                  Trick 5 shares one query between the two key sets)
3. query LayerNorm                Trick 2: LN on the query (and on the keys)

Readings where the paper is silent (each is also a test):

* The input is the hidden states x [B, L, d] of B sequences of L consecutive tokens; token
  t = b * L + l.  The convolution runs along each sequence.  Taps before a sequence's first
  token in this batch read the given history (the K_c - 1 hidden states that precede it; zeros
  at the start of a sequence), so a decode step (L = 1) and a prefill chunk compute the same
  outputs as the whole sequence would.
* The convolution has K_c taps per channel, y[b, l, c] = sum_j w[j, c] x[b, l - j, c] (tap 0 is
  the current token), and no bias.  K_c is not stated; the workloads use 4.
* Without sharing, the query linear produces 2 H D_k outputs per token: the row queries of the
  H heads, then the column queries.  With sharing (Trick 5) it produces H D_k, and the same query
  serves both key sets.
* LayerNorm normalises each head's query (and each key) over its D_k elements with the
  population variance, then scales and shifts elementwise with its own gamma, beta in R^{D_k}
  (one pair per head and axis; the appendix initialises the query weight to 1 / sqrt(E(Y)) and
  the key weight to 1 / sqrt(D_k)).  epsilon is not stated; the workloads use 1e-5.  With the
  Tucker rank r the normalised query is then split into its r slices (eq. (4)).
* Keys are parameters, so their LayerNorm is computed once and the scoring takes the normalised
  keys.
"""
from __future__ import annotations

import numpy as np

__all__ = ["causal_conv", "query_linear", "layer_norm", "query_front_end", "key_norm"]


def causal_conv(x, w, hist=None) -> np.ndarray:
    """Trick 4: depthwise causal convolution along each sequence.

    x [B, L, d]; w [K_c, d] (tap j multiplies the token j steps back); hist [B, K_c - 1, d] (the
    hidden states before each sequence's first token here, oldest first) or None (zeros)."""
    x = np.asarray(x, np.float64)
    w = np.asarray(w, np.float64)
    B, L, d = x.shape
    kc = w.shape[0]
    if hist is None:
        hist = np.zeros((B, kc - 1, d))
    hist = np.asarray(hist, np.float64)
    assert w.shape == (kc, d) and hist.shape == (B, kc - 1, d)
    full = np.concatenate([hist, x], axis=1)           # position l of x is kc - 1 + l here
    y = np.zeros((B, L, d))
    for j in range(kc):
        y += w[j] * full[:, kc - 1 - j: kc - 1 - j + L, :]
    return y


def query_linear(y, W_q) -> np.ndarray:
    """The query layer of eq. (2): y [T, d] times W_q [d, Q]."""
    return np.asarray(y, np.float64) @ np.asarray(W_q, np.float64)


def layer_norm(v, gamma, beta, eps: float) -> np.ndarray:
    """Trick 2: LayerNorm over the last axis (population variance), then gamma, beta."""
    v = np.asarray(v, np.float64)
    mu = v.mean(axis=-1, keepdims=True)
    var = ((v - mu) ** 2).mean(axis=-1, keepdims=True)
    return (v - mu) / np.sqrt(var + eps) * np.asarray(gamma, np.float64) + np.asarray(beta, np.float64)


def query_front_end(x, conv_w, W_q, gamma, beta, heads: int, dk: int, shared: bool, hist=None,
                    eps: float = 1e-5):
    """Hidden states x [B, L, d] -> (q_row, q_col), each [B * L, H, D_k].

    W_q [d, A * H * D_k] with A = 1 (shared) or 2 (row queries, then column queries);
    gamma, beta [A, H, D_k]."""
    x = np.asarray(x, np.float64)
    B, L, d = x.shape
    A = 1 if shared else 2
    y = causal_conv(x, conv_w, hist).reshape(B * L, d)
    q = query_linear(y, W_q).reshape(B * L, A, heads, dk)
    g = np.asarray(gamma, np.float64).reshape(A, heads, dk)
    b = np.asarray(beta, np.float64).reshape(A, heads, dk)
    q = layer_norm(q, g, b, eps)
    return (q[:, 0], q[:, 0]) if shared else (q[:, 0], q[:, 1])


def key_norm(K, gamma, beta, eps: float = 1e-5) -> np.ndarray:
    """Trick 2 on one key set: K [H, n, D_k], gamma, beta [H, D_k]."""
    K = np.asarray(K, np.float64)
    g = np.asarray(gamma, np.float64)[:, None, :]
    b = np.asarray(beta, np.float64)[:, None, :]
    return layer_norm(K, g, b, eps)
