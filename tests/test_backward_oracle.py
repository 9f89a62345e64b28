"""The backward oracle against its pins, and planted mistakes that the pins must catch.
CPU only."""
import numpy as np
import pytest

import oracle.backward_oracle as B
import oracle.umem_oracle as O
from tests.backward_pins import BACKWARD_PINS

_orig = {name: getattr(B, name) for name in ("gather_backward", "weights_backward", "score_backward")}


@pytest.mark.parametrize("pin", BACKWARD_PINS, ids=lambda p: p.__name__)
def test_pin(pin):
    pin(B)


def m_block0_gradient(value_rows, idx, w, d_pooled, perm=None, n_values=None, expand=1):
    """Every entry takes virtual block 0's output gradient."""
    dp = np.asarray(d_pooled, np.float64)
    return _orig["gather_backward"](value_rows, idx, w, np.repeat(dp[:, :1], dp.shape[1], axis=1),
                                    perm, n_values, expand)


def m_repeats_overwrite(value_rows, idx, w, d_pooled, perm=None, n_values=None, expand=1):
    """A row's gradient is the last entry's contribution, not the sum."""
    rows, dV, dw = _orig["gather_backward"](value_rows, idx, w, d_pooled, perm, n_values, expand)
    idx = np.asarray(idx, np.int64)
    p, row = O.address_map(idx, perm, n_values, expand)
    w = np.asarray(w, np.float64)
    dp = np.asarray(d_pooled, np.float64)
    pos = {int(r): k for k, r in enumerate(rows)}
    for t in range(idx.shape[0]):
        for b in range(idx.shape[1]):
            wb = w[t, b] if w.ndim == 2 else np.repeat(w[t, b], dp.shape[2] // w.shape[2])
            dV[pos[int(row[t, b])]] = wb * dp[t, p[t, b]]
    return rows, dV, dw


def m_mcs_whole_row_dots(value_rows, idx, w, d_pooled, perm=None, n_values=None, expand=1):
    """Each core's weight gradient taken over the whole row instead of its column slice."""
    rows, dV, dw = _orig["gather_backward"](value_rows, idx, w, d_pooled, perm, n_values, expand)
    if np.ndim(dw) == 3:
        dw = np.repeat(dw.sum(axis=2, keepdims=True), dw.shape[2], axis=2)
    return rows, dV, dw


def m_softmax_not_centred(dw, w, weight=0):
    if weight == O.W_RAW:
        return _orig["weights_backward"](dw, w, weight)
    return np.asarray(w, np.float64) * np.asarray(dw, np.float64)


def m_core_transposed(q_row, q_col, K_row, K_col, idx, dw, w=None, grid=0, weight=0, core=None,
                      rank=1, core_parts=None):
    tr = lambda c: None if c is None else np.swapaxes(np.asarray(c), -1, -2)
    res = _orig["score_backward"](q_row, q_col, K_row, K_col, idx, dw, w, grid, weight, tr(core),
                                  rank, tr(core_parts))
    if res["dC"] is not None:
        res["dC"] = np.swapaxes(res["dC"], -1, -2)
    return res


def m_dC_transposed(*a, **kw):
    res = _orig["score_backward"](*a, **kw)
    if res["dC"] is not None:
        res["dC"] = np.swapaxes(res["dC"], -1, -2)
    return res


def m_dq_axes_swapped(*a, **kw):
    res = _orig["score_backward"](*a, **kw)
    res["dq_row"], res["dq_col"] = res["dq_col"], res["dq_row"]
    return res


def m_dK_slices_swapped(q_row, q_col, K_row, K_col, idx, dw, w=None, grid=0, weight=0, core=None,
                        rank=1, core_parts=None):
    """The key gradient of slice rho takes the query of the other slice."""
    res = _orig["score_backward"](q_row, q_col, K_row, K_col, idx, dw, w, grid, weight, core, rank,
                                  core_parts)
    if rank > 1:
        width = np.shape(q_row)[2] // rank
        for name, q in (("dK_row", q_row), ("dK_col", q_col)):
            q = np.asarray(q, np.float64)
            qs = np.concatenate([q[:, :, width:], q[:, :, :width]], axis=2)
            dS = res["dS_row"] if name == "dK_row" else res["dS_col"]
            dK = np.zeros_like(res[name])
            for h in range(q.shape[1]):
                for rho in range(rank):
                    sl = slice(rho * width, (rho + 1) * width)
                    dK[h, :, sl] = dS[:, h, rho, :].T @ qs[:, h, sl]
            res[name] = dK
    return res


MUTANTS = [
    ("gather_backward", m_block0_gradient), ("gather_backward", m_repeats_overwrite),
    ("gather_backward", m_mcs_whole_row_dots), ("weights_backward", m_softmax_not_centred),
    ("score_backward", m_core_transposed), ("score_backward", m_dC_transposed),
    ("score_backward", m_dq_axes_swapped), ("score_backward", m_dK_slices_swapped),
]


@pytest.mark.parametrize("target,mutant", MUTANTS, ids=[m[1].__name__ for m in MUTANTS])
def test_mutant_is_caught(monkeypatch, target, mutant):
    monkeypatch.setattr(B, target, mutant)
    failed = []
    for pin in BACKWARD_PINS:
        try:
            pin(B)
        except AssertionError:
            failed.append(pin.__name__)
    assert failed, f"no pin catches {mutant.__name__}"
