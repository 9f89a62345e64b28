"""The query front-end oracle against its pins, and planted mistakes that the pins must catch.
CPU only."""
import numpy as np
import pytest

import oracle.query_oracle as Q
from tests.query_pins import QUERY_PINS

_orig = {name: getattr(Q, name) for name in ("causal_conv", "layer_norm", "query_front_end", "key_norm")}


@pytest.mark.parametrize("pin", QUERY_PINS, ids=lambda p: p.__name__)
def test_pin(pin):
    pin(Q)


def m_conv_future(x, w, hist=None):
    """Reads tap j from the token j steps ahead."""
    x = np.asarray(x, np.float64)
    rev = _orig["causal_conv"](x[:, ::-1], w, None)
    return rev[:, ::-1]


def m_conv_taps_reversed(x, w, hist=None):
    return _orig["causal_conv"](x, np.asarray(w)[::-1], hist)


def m_conv_no_history(x, w, hist=None):
    return _orig["causal_conv"](x, w, None)


def m_ln_sample_variance(v, gamma, beta, eps):
    """Divides the squared deviations by D_k - 1."""
    v = np.asarray(v, np.float64)
    sd = np.sqrt(v.var(axis=-1, ddof=1, keepdims=True) + eps)
    return (v - v.mean(axis=-1, keepdims=True)) / sd * np.asarray(gamma, np.float64) + np.asarray(beta, np.float64)


def m_ln_gamma_beta_swapped(v, gamma, beta, eps):
    return _orig["layer_norm"](v, beta, gamma, eps)


def m_front_end_axes_swapped(x, conv_w, W_q, gamma, beta, heads, dk, shared, hist=None, eps=1e-5):
    qr, qc = _orig["query_front_end"](x, conv_w, W_q, gamma, beta, heads, dk, shared, hist, eps)
    return qc, qr


def m_front_end_heads_interleaved(x, conv_w, W_q, gamma, beta, heads, dk, shared, hist=None, eps=1e-5):
    """Takes the D_k outputs of a head strided across the linear's output, not as a block."""
    W = np.asarray(W_q, np.float64)
    A = 1 if shared else 2
    perm = np.arange(A * heads * dk).reshape(dk, A * heads).T.reshape(-1)
    return _orig["query_front_end"](x, conv_w, W[:, perm], gamma, beta, heads, dk, shared, hist, eps)


def m_key_norm_shared_gamma(K, gamma, beta, eps=1e-5):
    g = np.asarray(gamma, np.float64)
    return _orig["key_norm"](K, np.broadcast_to(g[:1], g.shape), beta, eps)


MUTANTS = [
    ("causal_conv", m_conv_future), ("causal_conv", m_conv_taps_reversed),
    ("causal_conv", m_conv_no_history), ("layer_norm", m_ln_sample_variance),
    ("layer_norm", m_ln_gamma_beta_swapped), ("query_front_end", m_front_end_axes_swapped),
    ("query_front_end", m_front_end_heads_interleaved), ("key_norm", m_key_norm_shared_gamma),
]


@pytest.mark.parametrize("target,mutant", MUTANTS, ids=[m[1].__name__ for m in MUTANTS])
def test_mutant_is_caught(monkeypatch, target, mutant):
    monkeypatch.setattr(Q, target, mutant)
    failed = []
    for pin in QUERY_PINS:
        try:
            pin(Q)
        except AssertionError:
            failed.append(pin.__name__)
    assert failed, f"no pin catches {mutant.__name__}"
