"""Plant plausible mistakes in the oracle (on the CPU) and check that the pins catch each one."""
import numpy as np
import pytest

import oracle.umem_oracle as O
from tests.pins import ALL_PINS

_orig = {name: getattr(O, name) for name in
         ("axis_scores", "rank1_factors", "selection_scores", "top_sorted", "grid_topm",
          "pooling_weights", "address_map", "gather_sum", "ive_project", "core_scores")}


def m_flat_transposed(S_row, S_col, I_row, I_col, n, m, grid=0, C=None):
    flat, g = _orig["grid_topm"](S_col, S_row, I_col, I_row, n, m, grid,
                                 None if C is None else np.asarray(C).T)
    return flat, g


def m_drop_col_term(S_row, S_col, I_row, I_col, n, m, grid=0, C=None):
    return _orig["grid_topm"](S_row, 0 * S_col, I_row, I_col, n, m, grid, C)


def m_core_transposed(S_row, S_col, I_row, I_col, n, m, grid=0, C=None):
    return _orig["grid_topm"](S_row, S_col, I_row, I_col, n, m, grid,
                              None if C is None else np.asarray(C).T)


def m_bottom_k(x, k):
    return _orig["top_sorted"](-np.asarray(x), k)


def m_ties_high_index(x, k):
    x = np.asarray(x, dtype=np.float64)
    order = np.argsort(-x[::-1], kind="stable")
    return (len(x) - 1 - order)[:k]


def m_sign_negative(C):
    u, t, s = _orig["rank1_factors"](C)
    return -u, -t, s


def m_t_from_C_not_CT(C):
    u, t, s = _orig["rank1_factors"](C)
    C = np.asarray(C, dtype=np.float64)
    return u, C @ u / s[0], s


def m_slices_interleaved(q, K, rank=1):
    q = np.asarray(q, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    dk = q.shape[2]
    perm = np.arange(dk).reshape(dk // rank, rank).T.reshape(-1)   # strided slices
    return _orig["axis_scores"](q[:, :, perm[::-1]] if rank == 1 else q[:, :, perm],
                                K[:, :, perm] if rank > 1 else K, rank)


def m_swap_factor_vectors(S, vecs):
    if vecs is None:
        return _orig["selection_scores"](S, vecs)
    return _orig["selection_scores"](S, [v[::-1] for v in vecs])


def m_repeats_overwrite(value_rows, idx, w, perm=None, n_values=None, expand=1):
    idx = np.asarray(idx)
    T, bag = idx.shape
    p, row = O.address_map(idx, perm, n_values, expand)
    out = None
    for t in range(T):
        vals = np.asarray(value_rows(row[t]), dtype=np.float64)
        if out is None:
            out = np.zeros((T, expand, vals.shape[1]))
        for b in range(bag):
            out[t, p[t, b]] = w[t, b] * vals[b]
    return out


def m_block_modulo(idx, perm=None, n_values=None, expand=1):
    idx = np.asarray(idx, dtype=np.int64)
    if perm is None and expand == 1:
        return np.zeros_like(idx), idx.copy()
    v = np.asarray(perm)[idx]
    return v % expand, v // expand


def m_project_transposed(pooled, W_proj=None, W_out=None):
    if W_proj is not None:
        W_proj = np.transpose(np.asarray(W_proj), (0, 2, 1))
        if W_proj.shape[1] != np.shape(pooled)[2]:
            W_proj = np.asarray(W_proj)[:, :np.shape(pooled)[2], :]
    return _orig["ive_project"](pooled, W_proj, W_out)


def m_softmax_no_normalise(g, weight=0):
    g = np.asarray(g, dtype=np.float64)
    return g.copy() if weight == 0 else np.exp(g - g.max())


def m_core_scores_reversed(S_row, S_col, flat, n, core_parts):
    return _orig["core_scores"](S_row, S_col, flat, n, core_parts)[:, ::-1]


def m_mcs_one_weight_for_all(value_rows, idx, w, perm=None, n_values=None, expand=1):
    w = np.asarray(w, dtype=np.float64)
    if w.ndim == 3:
        w = w.sum(axis=2)                       # the aggregated score on every slice
    return _orig["gather_sum"](value_rows, idx, w, perm, n_values, expand)


def m_mcs_slices_interleaved(value_rows, idx, w, perm=None, n_values=None, expand=1):
    w = np.asarray(w, dtype=np.float64)
    if w.ndim == 2:
        return _orig["gather_sum"](value_rows, idx, w, perm, n_values, expand)
    h = w.shape[2]
    out = None
    idx = np.asarray(idx)
    p, row = O.address_map(idx, perm, n_values, expand)
    for t in range(idx.shape[0]):
        vals = np.asarray(value_rows(row[t]), dtype=np.float64)
        if out is None:
            out = np.zeros((idx.shape[0], expand, vals.shape[1]))
        wt = np.tile(w[t], (1, vals.shape[1] // h))          # column c takes core c % h
        np.add.at(out[t], p[t], wt * vals)
    return out


MUTANTS = [
    ("core_scores", m_core_scores_reversed), ("gather_sum", m_mcs_one_weight_for_all),
    ("gather_sum", m_mcs_slices_interleaved),
    ("grid_topm", m_flat_transposed), ("grid_topm", m_drop_col_term),
    ("grid_topm", m_core_transposed), ("top_sorted", m_bottom_k),
    ("top_sorted", m_ties_high_index), ("rank1_factors", m_sign_negative),
    ("rank1_factors", m_t_from_C_not_CT), ("axis_scores", m_slices_interleaved),
    ("selection_scores", m_swap_factor_vectors), ("gather_sum", m_repeats_overwrite),
    ("address_map", m_block_modulo), ("ive_project", m_project_transposed),
    ("pooling_weights", m_softmax_no_normalise),
]


@pytest.mark.parametrize("target,mutant", MUTANTS, ids=[m[1].__name__ for m in MUTANTS])
def test_pins_catch_mutant(monkeypatch, target, mutant):
    monkeypatch.setattr(O, target, mutant)
    caught = []
    for pin in ALL_PINS:
        try:
            pin(O)
        except Exception as e:      # an assertion, or the mutant breaking a shape contract
            caught.append((getattr(pin, "__name__", "pin"), type(e).__name__))
    assert caught, f"no pin caught mutant {mutant.__name__}"
