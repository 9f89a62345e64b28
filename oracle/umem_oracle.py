"""UltraMem memory-layer forward: a plain, slow CPU oracle in fp64.  TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline leg may use this
module.  It shares no code with the GPU library; inputs come from :mod:`synth`.

It follows the paper ("Ultra-Sparse Memory Network", Huang et al.) step by step:

1. axis scores      Sec. 3.1 eq. (2) (product keys); Sec. 3.2 TDQKR eq. (4) (rank-r slices)
2. rank-1 factors   Sec. 3.2 TDQKR eqs. (6), (7), (11): leading singular pair of the core C
3. per-axis top-k   eq. (2) sigma_TopM; eqs. (8), (9) I_TopM on u^T S_row and t^T S_col
4. grid scores      eq. (3) s_row + s_col^T (additive); eq. (10) S~_row^T C S~_col (Tucker)
5. global top-m     eq. (3) / eq. (10) sigma_TopM over the candidates; weights raw (Trick 1 of
                    Sec. 3.2 removes the softmax) or eq. (3)'s SoftMax
6. address map      Sec. 3.1 (physical address n*i + j); Sec. 3.2 IVE eq. (14) Shuffle and the
                    block concatenation of eq. (13)
7. gather-sum       eq. (1) o = V^T s; eq. (15) V^T s_p per virtual block; heads add (Sec. 3.1);
                    with multi-core scoring (Sec. 3.2 MCS), eq. (17): column slice i of the
                    values pooled with core i's scores
8. projection       eq. (15) sum_p W_p^T (.); output linear of Trick 6 (Sec. 3.2)

Readings where the paper is silent or ambiguous (each is also a test):

* Ties: order is (score desc, index asc) -- the per-axis key index, or on the grid the logical
  flat index i*n + j (before any shuffle); -0.0 equals +0.0; NaN inputs are rejected.  Outputs
  are sorted in that order.
* Names: the paper writes m for both the per-axis and the global top; here k is per axis and m
  global, with 1 <= m <= k*k.
* Masked Tucker grid, eqs. (8)-(10): entries outside I_row x I_col are excluded from the final
  top-m (they are -inf, as sigma_TopM defines), not scored 0 by the 0/1 mask.
* Singular-vector sign: u and t are fixed only up to a joint flip, which would turn the per-axis
  top-k into a bottom-k.  The component of u of largest magnitude (lowest index among equal
  magnitudes) is made positive and t = C^T u / sigma_1, so C ~ sigma_1 u t^T; sigma_1 > 0 is
  dropped since it does not change any order.  A core with sigma_1 - sigma_2 <= 1e-9 sigma_1 is
  rejected (its leading pair is not unique).
* IVE layout: blocks p = 0..E-1; virtual slot v = p * N_p + physical row (the concatenation
  order of eq. (13)); the shuffle sends the score of logical slot x to virtual slot perm[x].
* Heads: each head has its own keys and core, all heads share V, and their pooled outputs add.
* Multi-core scoring (Sec. 3.2, eqs. (16), (17)): the Tucker core of each head is given as h
  component cores; selection runs on their sum (eq. (16)), and each selected slot carries h
  scores, S_row^T C^(i) S_col, that weight column slice i (of Dv / h columns) of its value row.
  With IVE the physical rows are split.  Only raw scores are defined for it (the paper pairs
  MCS with Trick 1's removal of the softmax).
* Precision: everything in fp64 from the stored fp32 / bf16 inputs (a product of two fp32 numbers
  is exact in fp64).
"""
from __future__ import annotations

import numpy as np

GRID_ADD = 0
GRID_TUCKER = 1
W_RAW = 0
W_SOFTMAX = 1

DEGENERATE_GAP = 1e-9

__all__ = [
    "GRID_ADD", "GRID_TUCKER", "W_RAW", "W_SOFTMAX", "axis_scores", "rank1_factors",
    "selection_scores", "top_sorted", "grid_topm", "core_scores", "pooling_weights", "score_topk",
    "address_map", "gather_sum", "ive_project", "forward",
]


def axis_scores(q, K, rank: int = 1) -> np.ndarray:
    """Scores of one axis (row or column) -- eq. (2); with rank r, eq. (4).

    q: [T, H, Dk] this axis's query; K: [H, n, Dk] this axis's keys.  With rank r the Dk axis is
    read as r contiguous slices of Dk/r, the reshape to K in R^{r x n x Dk/r} and
    q in R^{r x Dk/r} of eq. (4).  Returns S [T, H, r, n], fp64, with
    S[t, h, rho, i] = sum_{d in slice rho} K[h, i, d] * q[t, h, d].
    """
    q = np.asarray(q, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    T, H, dk = q.shape
    n = K.shape[1]
    assert K.shape == (H, n, dk) and dk % rank == 0
    width = dk // rank
    S = np.empty((T, H, rank, n))
    for h in range(H):
        for rho in range(rank):
            sl = slice(rho * width, (rho + 1) * width)
            S[:, h, rho, :] = q[:, h, sl] @ K[h, :, sl].T
    return S


def rank1_factors(C):
    """Leading left/right singular vectors (u, t) of one Tucker core C [r, r] -- eqs. (6), (11).

    Returns (u, t, singular values in descending order).  Sign reading as in the module header.
    """
    C = np.asarray(C, dtype=np.float64)
    U, sig, _ = np.linalg.svd(C)
    if C.shape[0] > 1 and sig[0] - sig[1] <= DEGENERATE_GAP * sig[0]:
        raise ValueError("degenerate Tucker core: leading singular value is not simple")
    if sig[0] == 0.0:
        raise ValueError("zero Tucker core")
    u = U[:, 0].copy()
    j = int(np.argmax(np.abs(u)))          # first maximum: lowest index among equal magnitudes
    if u[j] < 0:
        u = -u
    t = C.T @ u / sig[0]
    return u, t, sig


def selection_scores(S: np.ndarray, vecs) -> np.ndarray:
    """The per-axis score that the top-k runs on: u^T S_row or t^T S_col of eqs. (6), (8), (9).

    S: [T, H, r, n]; vecs: [H, r] (one factor vector per head), or None for the additive grid,
    where the score is the axis score itself (eq. (2)).  Returns [T, H, n].
    """
    if vecs is None:
        assert S.shape[2] == 1
        return S[:, :, 0, :].copy()
    T, H, r, n = S.shape
    a = np.zeros((T, H, n))
    for h in range(H):
        for rho in range(r):
            a[:, h, :] += vecs[h][rho] * S[:, h, rho, :]
    return a


def top_sorted(x, k: int) -> np.ndarray:
    """Indices of the k largest entries of the 1-D array x, ordered by (value desc, index asc).

    This is the keep-set of sigma_TopM (eq. (2)) and of I_TopM (eqs. (8), (9)).
    """
    x = np.asarray(x, dtype=np.float64)
    if np.isnan(x).any():
        raise ValueError("NaN score")
    order = np.argsort(-x, kind="stable")  # a stable sort keeps lower indices first among ties
    return order[:k]


def grid_topm(S_row, S_col, I_row, I_col, n: int, m: int, grid: int = GRID_ADD, C=None):
    """Candidate scores on I_row x I_col and the global top-m of one (token, head).

    S_row, S_col: [r, n] axis scores of this token and head.  Additive grid (eq. (3)): candidate
    (i, j) scores S_row[0, i] + S_col[0, j].  Tucker grid (eq. (10)): it scores
    sum_{rho, sigma} S_row[rho, i] * C[rho, sigma] * S_col[sigma, j].  Entries outside the
    candidate set are excluded.  Returns (flat logical indices i*n + j, their scores), m of each,
    ordered by (score desc, flat index asc).
    """
    I_row = np.asarray(I_row, dtype=np.int64)
    I_col = np.asarray(I_col, dtype=np.int64)
    ii = np.repeat(I_row, len(I_col))
    jj = np.tile(I_col, len(I_row))
    if grid == GRID_ADD:
        g = S_row[0, ii] + S_col[0, jj]
    else:
        C = np.asarray(C, dtype=np.float64)
        r = C.shape[0]
        g = np.zeros(len(ii))
        for rho in range(r):
            for sig in range(r):
                g += S_row[rho, ii] * C[rho, sig] * S_col[sig, jj]
    flat = ii * n + jj
    if np.isnan(g).any():
        raise ValueError("NaN grid score")
    order = np.lexsort((flat, -g))[:m]     # primary key -g, secondary key flat
    return flat[order], g[order]


def core_scores(S_row, S_col, flat, n: int, core_parts) -> np.ndarray:
    """Per-core scores of the selected slots -- multi-core scoring, Sec. 3.2, eq. (16):
    S^(i) = S_row^T C^(i) S_col at slot (i_row, j_col) = divmod(flat, n).

    S_row, S_col: [r, n] of one (token, head); core_parts: [h, r, r].  Returns [len(flat), h].
    """
    flat = np.asarray(flat, dtype=np.int64)
    ii, jj = flat // n, flat % n
    parts = np.asarray(core_parts, dtype=np.float64)
    h, r, _ = parts.shape
    out = np.zeros((len(flat), h))
    for c in range(h):
        for rho in range(r):
            for sig in range(r):
                out[:, c] += S_row[rho, ii] * parts[c, rho, sig] * S_col[sig, jj]
    return out


def pooling_weights(g, weight: int = W_RAW) -> np.ndarray:
    """Weights of the m selected slots of one (token, head).

    W_RAW: the selected scores themselves (Trick 1 of Sec. 3.2 removes the softmax).
    W_SOFTMAX: eq. (3)'s SoftMax over vec(S_grid), whose unselected entries are -inf and so get
    weight 0; computed with the maximum subtracted.
    """
    g = np.asarray(g, dtype=np.float64)
    if weight == W_RAW:
        return g.copy()
    e = np.exp(g - g.max())
    return e / e.sum()


def score_topk(q_row, q_col, K_row, K_col, topk: int, topm: int, grid: int = GRID_ADD,
               weight: int = W_RAW, core=None, rank: int = 1, core_parts=None):
    """Steps 1-5 for every token and head.  Returns a dict with

    idx [T, H, m] logical flat indices (sorted), w [T, H, m] weights, g [T, H, m] grid scores,
    axis_idx [2, T, H, k] per-axis top-k (row, col; sorted), sel_row / sel_col [T, H, n] the
    per-axis selection scores, S_row / S_col [T, H, r, n], factors [(u, t, sig)] per head.

    Multi-core scoring: core_parts [H, h, r, r] are the component cores (core must then be None);
    selection runs on their sum, and w_core [T, H, m, h] holds each core's score of every
    selected slot (raw weights only).
    """
    if core_parts is not None:
        if core is not None or grid != GRID_TUCKER or weight != W_RAW:
            raise ValueError("multi-core scoring takes component cores, the Tucker grid, raw weights")
        core = np.asarray(core_parts, dtype=np.float64).sum(axis=1)     # eq. (16)
    T, H, dk = np.shape(q_row)
    n = np.shape(K_row)[1]
    if grid == GRID_ADD:
        assert rank == 1
    if not (1 <= topk <= n and 1 <= topm <= topk * topk):
        raise ValueError("need 1 <= k <= n and 1 <= m <= k*k")
    S_row = axis_scores(q_row, K_row, rank)
    S_col = axis_scores(q_col, K_col, rank)
    if grid == GRID_TUCKER:
        factors = [rank1_factors(core[h]) for h in range(H)]
        sel_row = selection_scores(S_row, [f[0] for f in factors])
        sel_col = selection_scores(S_col, [f[1] for f in factors])
    else:
        factors = None
        sel_row = selection_scores(S_row, None)
        sel_col = selection_scores(S_col, None)
    idx = np.empty((T, H, topm), dtype=np.int64)
    w = np.empty((T, H, topm))
    g = np.empty((T, H, topm))
    axis_idx = np.empty((2, T, H, topk), dtype=np.int64)
    w_core = None if core_parts is None else np.empty((T, H, topm, np.shape(core_parts)[1]))
    for t in range(T):
        for h in range(H):
            I_row = top_sorted(sel_row[t, h], topk)
            I_col = top_sorted(sel_col[t, h], topk)
            flat, gs = grid_topm(S_row[t, h], S_col[t, h], I_row, I_col, n, topm, grid,
                                 None if core is None else core[h])
            idx[t, h], g[t, h] = flat, gs
            w[t, h] = pooling_weights(gs, weight)
            axis_idx[0, t, h], axis_idx[1, t, h] = I_row, I_col
            if core_parts is not None:
                w_core[t, h] = core_scores(S_row[t, h], S_col[t, h], flat, n, core_parts[h])
    return dict(idx=idx, w=w, g=g, axis_idx=axis_idx, sel_row=sel_row, sel_col=sel_col,
                S_row=S_row, S_col=S_col, factors=factors, w_core=w_core)


def address_map(idx, perm=None, n_values: int | None = None, expand: int = 1):
    """Logical slot -> (virtual block p, physical row).

    Without expansion the slot (i, j) lives at physical row n*i + j (Sec. 3.1), i.e. row = idx.
    With IVE (eq. (14)) the shuffle sends logical slot x to virtual slot v = perm[x]; the virtual
    table is the concatenation of the E blocks V W_p (eq. (13)), so p = v // N_p and the physical
    row is v % N_p.
    """
    idx = np.asarray(idx, dtype=np.int64)
    if perm is None and expand == 1:
        return np.zeros_like(idx), idx.copy()
    v = np.asarray(perm, dtype=np.int64)[idx] if perm is not None else idx
    return v // n_values, v % n_values


def gather_sum(value_rows, idx, w, perm=None, n_values: int | None = None, expand: int = 1):
    """Score-weighted pooling of the selected value rows -- eq. (1) o = V^T s, eq. (3), and
    eq. (15)'s per-block V^T s_p.

    value_rows(rows) returns the stored rows [len(rows), Dv] (any float type); idx: [T, bag] (a
    bag is all heads' m selections of a token); w: [T, bag], or [T, bag, h] with multi-core
    scoring, where column slice i (Dv / h columns) of each row takes weight w[..., i] (eq. (17)).
    Returns out [T, E, Dv] in fp64 with out[t, p, :] = sum over entries b of block p of
    w[t, b] * V[row[t, b], :]; repeats add.
    """
    idx = np.asarray(idx, dtype=np.int64)
    w = np.asarray(w, dtype=np.float64)
    T, bag = idx.shape
    p, row = address_map(idx, perm, n_values, expand)
    out = None
    for t in range(T):
        vals = np.asarray(value_rows(row[t]), dtype=np.float64)
        if out is None:
            out = np.zeros((T, expand, vals.shape[1]))
        if w.ndim == 2:
            wt = w[t][:, None]
        else:
            h = w.shape[2]
            wt = np.repeat(w[t], vals.shape[1] // h, axis=1)   # weight of each column
        np.add.at(out[t], p[t], wt * vals)
    return out


def ive_project(pooled, W_proj=None, W_out=None) -> np.ndarray:
    """sum_p W_p^T (V^T s_p) of eq. (15), then the output linear of Trick 6 (Sec. 3.2).

    pooled: [T, E, Dv]; W_proj: [E, Dv, D'v] or None (E must then be 1); W_out: [D'v, d_out] or
    None.  Returns [T, D'v] or [T, d_out] in fp64.
    """
    pooled = np.asarray(pooled, dtype=np.float64)
    T, E, dv = pooled.shape
    if W_proj is None:
        assert E == 1
        y = pooled[:, 0, :]
    else:
        W_proj = np.asarray(W_proj, dtype=np.float64)
        y = np.zeros((T, W_proj.shape[2]))
        for p in range(E):
            y += pooled[:, p, :] @ W_proj[p]
    if W_out is not None:
        y = y @ np.asarray(W_out, dtype=np.float64)
    return y


def forward(q_row, q_col, K_row, K_col, value_rows, topk: int, topm: int, grid: int = GRID_ADD,
            weight: int = W_RAW, core=None, rank: int = 1, perm=None, n_values=None,
            expand: int = 1, W_proj=None, W_out=None, core_parts=None):
    """The whole layer (steps 1-8).  Returns (output, score_topk dict, pooled [T, E, Dv])."""
    sel = score_topk(q_row, q_col, K_row, K_col, topk, topm, grid, weight, core, rank, core_parts)
    T, H, m = sel["idx"].shape
    w = sel["w"].reshape(T, H * m) if core_parts is None else sel["w_core"].reshape(T, H * m, -1)
    pooled = gather_sum(value_rows, sel["idx"].reshape(T, H * m), w, perm, n_values, expand)
    if W_proj is None and W_out is None:
        out = pooled[:, 0, :] if expand == 1 else pooled
    else:
        out = ive_project(pooled, W_proj, W_out)
    return out, sel, pooled
