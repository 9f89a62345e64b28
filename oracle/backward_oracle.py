"""Backward of the UltraMem memory layer: a plain CPU oracle in fp64.  TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline leg may use this
module.  It shares no code with the GPU library.

The layer is trained end to end with the transformer around it (Sec. 4).  Its forward is
piecewise differentiable: the per-axis top-k and the global top-m are piecewise constant in the
scores, so the gradient reaches the queries, keys and core only through the scores of the
selected slots.  This module is the exact derivative of ``umem_oracle.forward`` with the
selection held fixed, step by step in reverse:

1. pooling        eq. (1) / eq. (15) per virtual block / eq. (17) per column slice:
                  dw[t, b] = <d_pooled[t, p_b, slice], V[row_b, slice]>,
                  dV[row_b, slice] += w[t, b] d_pooled[t, p_b, slice]  (repeats add)
2. weights        raw scores (Trick 1): dg = dw; eq. (3)'s SoftMax over the m selected:
                  dg = w * (dw - sum_j w_j dw_j)
3. grid scores    eq. (3): dS_row[0, i] += dg, dS_col[0, j] += dg;
                  eq. (10) (and eq. (16) per component core C^(c) with its own dg^(c)):
                  dS_row[:, i] += dg C S_col[:, j], dS_col[:, j] += dg C^T S_row[:, i],
                  dC += dg S_row[:, i] S_col[:, j]^T
4. axis scores    eq. (2) / eq. (4): dq[t, h, slice rho] = sum_i dS[rho, i] K[h, i, slice rho],
                  dK[h, i, slice rho] += dS[rho, i] q[t, h, slice rho]

Readings:

* The selection is held fixed.  Its derivative is zero wherever it is defined, and the rank-1
  factors u, t of eqs. (8), (9) only choose the candidates, so no gradient reaches them; C is
  trained through the exact candidate scores of eq. (10) (and the auxiliary loss of eq. (12),
  which is separate).
* Repeated slots (two heads choosing one value row) add, as they do in the forward.
"""
from __future__ import annotations

import numpy as np

import oracle.umem_oracle as O

__all__ = ["gather_backward", "weights_backward", "score_backward"]


def gather_backward(value_rows, idx, w, d_pooled, perm=None, n_values: int | None = None,
                    expand: int = 1):
    """Step 1.  idx [T, bag]; w [T, bag] or [T, bag, h] (multi-core scoring); d_pooled
    [T, E, Dv].  Returns (rows, dV, dw): the distinct physical rows touched (ascending), their
    gradients dV [len(rows), Dv], and dw shaped like w."""
    idx = np.asarray(idx, dtype=np.int64)
    w = np.asarray(w, dtype=np.float64)
    d_pooled = np.asarray(d_pooled, dtype=np.float64)
    T, bag = idx.shape
    p, row = O.address_map(idx, perm, n_values, expand)
    rows = np.unique(row)
    pos = {int(r): k for k, r in enumerate(rows)}
    dv = d_pooled.shape[2]
    h = 1 if w.ndim == 2 else w.shape[2]
    width = dv // h
    dV = np.zeros((len(rows), dv))
    dw = np.zeros_like(w)
    for t in range(T):
        vals = np.asarray(value_rows(row[t]), dtype=np.float64)
        for b in range(bag):
            g = d_pooled[t, p[t, b]]
            for c in range(h):
                sl = slice(c * width, (c + 1) * width)
                wb = w[t, b] if w.ndim == 2 else w[t, b, c]
                dot = float(np.dot(g[sl], vals[b, sl]))
                if w.ndim == 2:
                    dw[t, b] += dot
                else:
                    dw[t, b, c] = dot
                dV[pos[int(row[t, b])], sl] += wb * g[sl]
    return rows, dV, dw


def weights_backward(dw, w, weight: int = O.W_RAW) -> np.ndarray:
    """Step 2 for the m slots of one (token, head): the gradient of the grid scores."""
    dw = np.asarray(dw, dtype=np.float64)
    if weight == O.W_RAW:
        return dw.copy()
    w = np.asarray(w, dtype=np.float64)
    return w * (dw - np.dot(w, dw))


def score_backward(q_row, q_col, K_row, K_col, idx, dw, w=None, grid: int = O.GRID_ADD,
                   weight: int = O.W_RAW, core=None, rank: int = 1, core_parts=None) -> dict:
    """Steps 2-4 for the selections idx [T, H, m] and weight gradients dw [T, H, m] (or
    [T, H, m, h] with multi-core scoring; w [T, H, m] is needed for the SoftMax).

    Returns dq_row, dq_col [T, H, Dk]; dK_row, dK_col [H, n, Dk]; dC [H, r, r] (Tucker) or
    [H, h, r, r] (multi-core scoring), else None."""
    q_row = np.asarray(q_row, dtype=np.float64)
    q_col = np.asarray(q_col, dtype=np.float64)
    K_row = np.asarray(K_row, dtype=np.float64)
    K_col = np.asarray(K_col, dtype=np.float64)
    idx = np.asarray(idx, dtype=np.int64)
    dw = np.asarray(dw, dtype=np.float64)
    T, H, dk = q_row.shape
    n = K_row.shape[1]
    m = idx.shape[2]
    S_row = O.axis_scores(q_row, K_row, rank)          # [T, H, r, n]
    S_col = O.axis_scores(q_col, K_col, rank)
    if core_parts is not None:
        parts = np.asarray(core_parts, dtype=np.float64)          # [H, h, r, r]
    elif grid == O.GRID_TUCKER:
        parts = np.asarray(core, dtype=np.float64)[:, None]      # one component: [H, 1, r, r]
    else:
        parts = None
    dS_row = np.zeros_like(S_row)
    dS_col = np.zeros_like(S_col)
    dC = None if parts is None else np.zeros_like(parts)
    for t in range(T):
        for h in range(H):
            if parts is None:
                dg = weights_backward(dw[t, h], None if w is None else w[t, h], weight)
                for s in range(m):
                    i, j = divmod(int(idx[t, h, s]), n)
                    dS_row[t, h, 0, i] += dg[s]
                    dS_col[t, h, 0, j] += dg[s]
                continue
            dgc = dw[t, h] if dw.ndim == 4 else weights_backward(
                dw[t, h], None if w is None else w[t, h], weight)[:, None]
            for s in range(m):
                i, j = divmod(int(idx[t, h, s]), n)
                for c in range(parts.shape[1]):
                    C = parts[h, c]
                    g = dgc[s, c]
                    dS_row[t, h, :, i] += g * (C @ S_col[t, h, :, j])
                    dS_col[t, h, :, j] += g * (C.T @ S_row[t, h, :, i])
                    dC[h, c] += g * np.outer(S_row[t, h, :, i], S_col[t, h, :, j])
    width = dk // rank
    dq_row, dq_col = np.zeros_like(q_row), np.zeros_like(q_col)
    dK_row, dK_col = np.zeros_like(K_row), np.zeros_like(K_col)
    for dS, q, K, dq, dK in ((dS_row, q_row, K_row, dq_row, dK_row),
                             (dS_col, q_col, K_col, dq_col, dK_col)):
        for h in range(H):
            for rho in range(rank):
                sl = slice(rho * width, (rho + 1) * width)
                dq[:, h, sl] = dS[:, h, rho, :] @ K[h, :, sl]
                dK[h, :, sl] += dS[:, h, rho, :].T @ q[:, h, sl]
    if dC is not None and core_parts is None:
        dC = dC[:, 0]
    return dict(dq_row=dq_row, dq_col=dq_col, dK_row=dK_row, dK_col=dK_col, dC=dC,
                dS_row=dS_row, dS_col=dS_col)
