"""Pins of the backward oracle (module ``B``): a hand-worked fixture, central finite
differences of the forward oracle (the gradient of L = <d_pooled, pooled> along random
directions, with the selection checked to stay fixed), and adjoint identities.

Each pin raises AssertionError on a mismatch and takes the backward module as an argument so
that the mutation tests can run it against copies with planted mistakes.
"""
from __future__ import annotations

import json
import os

import numpy as np

import oracle.umem_oracle as O

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def pin_golden_backward(B):
    with open(os.path.join(GOLDEN, "backward_additive_n2.json")) as f:
        g = json.load(f)
    arr = lambda k: np.asarray(g[k], dtype=np.float64)
    V = arr("values")
    sel = O.score_topk(arr("q_row"), arr("q_col"), arr("K_row"), arr("K_col"), 2, 2)
    assert list(sel["idx"][0, 0]) == g["expect_idx"]
    rows, dV, dw = B.gather_backward(lambda r: V[r], sel["idx"].reshape(1, 2), sel["w"].reshape(1, 2),
                                     arr("d_pooled")[:, None, :])
    assert list(rows) == g["expect_rows"]
    assert np.array_equal(dV, g["expect_dV"]) and np.array_equal(dw[0], g["expect_dw"])
    res = B.score_backward(arr("q_row"), arr("q_col"), arr("K_row"), arr("K_col"), sel["idx"],
                           dw.reshape(1, 1, 2))
    assert res["dq_row"][0, 0, 0] == g["expect_dq_row"] and res["dq_col"][0, 0, 0] == g["expect_dq_col"]
    assert np.array_equal(res["dK_row"][0, :, 0], g["expect_dK_row_col0"])
    assert np.array_equal(res["dK_col"][0, :, 0], g["expect_dK_col_col0"])


# ---------------------------------------------------------------- finite differences

def _layer(seed, grid, weight=O.W_RAW, rank=1, cores=1, expand=1):
    rng = np.random.default_rng(seed)
    T, H, n, dk, k, m, dv = 3, 2, 6, 4, 4, 5, 6
    layer = dict(
        q_row=rng.standard_normal((T, H, dk)), q_col=rng.standard_normal((T, H, dk)),
        K_row=rng.standard_normal((H, n, dk)), K_col=rng.standard_normal((H, n, dk)),
        d_pooled=rng.standard_normal((T, expand, dv)), topk=k, topm=m, grid=grid, weight=weight,
        rank=rank, expand=expand, n_values=n * n // expand)
    layer["V"] = rng.standard_normal((layer["n_values"], dv))
    layer["perm"] = rng.permutation(n * n) if expand > 1 else None
    if grid == O.GRID_TUCKER:
        if cores > 1:
            layer["core_parts"] = rng.standard_normal((H, cores, rank, rank))
        else:
            layer["core"] = rng.standard_normal((H, rank, rank))
    return layer


def _forward(L):
    out, sel, pooled = O.forward(L["q_row"], L["q_col"], L["K_row"], L["K_col"],
                                 lambda r: L["V"][r], L["topk"], L["topm"], L["grid"], L["weight"],
                                 L.get("core"), L["rank"], L["perm"], L["n_values"], L["expand"],
                                 core_parts=L.get("core_parts"))
    return float(np.sum(L["d_pooled"] * pooled)), sel


def _gradients(B, L):
    _, sel = _forward(L)
    T, H, m = sel["idx"].shape
    w = sel["w"].reshape(T, H * m) if sel["w_core"] is None else sel["w_core"].reshape(T, H * m, -1)
    rows, dV_rows, dw = B.gather_backward(lambda r: L["V"][r], sel["idx"].reshape(T, H * m), w,
                                          L["d_pooled"], L["perm"], L["n_values"], L["expand"])
    dV = np.zeros_like(L["V"])
    dV[rows] = dV_rows
    dw = dw.reshape((T, H, m) + dw.shape[2:])
    res = B.score_backward(L["q_row"], L["q_col"], L["K_row"], L["K_col"], sel["idx"], dw,
                           sel["w"], L["grid"], L["weight"], L.get("core"), L["rank"],
                           L.get("core_parts"))
    grads = dict(V=dV, q_row=res["dq_row"], q_col=res["dq_col"], K_row=res["dK_row"],
                 K_col=res["dK_col"])
    if "core" in L:
        grads["core"] = res["dC"]
    if "core_parts" in L:
        grads["core_parts"] = res["dC"]
    return grads, sel


def _check_fd(B, L, seed, eps=1e-6, rtol=1e-6):
    grads, sel = _gradients(B, L)
    rng = np.random.default_rng(1000 + seed)
    for name, gr in grads.items():
        d = rng.standard_normal(np.shape(L[name]))
        plus, minus = dict(L), dict(L)
        plus[name] = L[name] + eps * d
        minus[name] = L[name] - eps * d
        lp, sp = _forward(plus)
        lm, sm = _forward(minus)
        # the selection must not move under the perturbation, or the difference is not a derivative
        assert np.array_equal(sp["idx"], sel["idx"]) and np.array_equal(sm["idx"], sel["idx"]), name
        fd = (lp - lm) / (2 * eps)
        an = float(np.sum(gr * d))
        assert abs(fd - an) <= rtol * max(1.0, abs(fd)), (name, fd, an)


def pin_fd_additive(B):
    for seed in range(3):
        _check_fd(B, _layer(seed, O.GRID_ADD), seed)


def pin_fd_additive_softmax(B):
    for seed in range(3):
        _check_fd(B, _layer(10 + seed, O.GRID_ADD, O.W_SOFTMAX), seed)


def pin_fd_tucker(B):
    for seed in range(3):
        _check_fd(B, _layer(20 + seed, O.GRID_TUCKER, rank=2), seed)


def pin_fd_tucker_mcs(B):
    for seed in range(3):
        _check_fd(B, _layer(30 + seed, O.GRID_TUCKER, rank=2, cores=2), seed)


def pin_fd_ive(B):
    for seed in range(3):
        _check_fd(B, _layer(40 + seed, O.GRID_TUCKER, rank=2, expand=4), seed)


# ---------------------------------------------------------------- identities

def pin_adjoint_identities(B):
    """The pooled output is linear in V and in the weights: <d_pooled, pooled> equals both
    <dV, V> over the touched rows and sum(dw * w)."""
    rng = np.random.default_rng(5)
    T, bag, Np, dv, E = 4, 7, 11, 8, 2
    V = rng.standard_normal((Np, dv))
    idx = rng.integers(0, Np * E, size=(T, bag))
    perm = rng.permutation(Np * E)
    for w in (rng.standard_normal((T, bag)), rng.standard_normal((T, bag, 2))):
        dp = rng.standard_normal((T, E, dv))
        pooled = O.gather_sum(lambda r: V[r], idx, w, perm, Np, E)
        rows, dV, dw = B.gather_backward(lambda r: V[r], idx, w, dp, perm, Np, E)
        lhs = float(np.sum(dp * pooled))
        assert np.isclose(lhs, float(np.sum(dV * V[rows])), rtol=1e-12)
        assert np.isclose(lhs, float(np.sum(dw * w)), rtol=1e-12)


def pin_repeated_rows_add(B):
    """Two entries on one row: that row's gradient is the sum of both contributions."""
    V = np.arange(12.0).reshape(3, 4)
    idx = np.array([[1, 1, 2]])
    w = np.array([[0.5, 2.0, 1.0]])
    dp = np.array([[[1.0, -1.0, 2.0, 0.5]]])
    rows, dV, dw = B.gather_backward(lambda r: V[r], idx, w, dp)
    assert list(rows) == [1, 2]
    assert np.array_equal(dV[0], 2.5 * dp[0, 0]) and np.array_equal(dV[1], 1.0 * dp[0, 0])
    assert np.array_equal(dw[0], [np.dot(dp[0, 0], V[1]), np.dot(dp[0, 0], V[1]), np.dot(dp[0, 0], V[2])])


BACKWARD_PINS = [pin_golden_backward, pin_fd_additive, pin_fd_additive_softmax, pin_fd_tucker,
                 pin_fd_tucker_mcs, pin_fd_ive, pin_adjoint_identities, pin_repeated_rows_add]
