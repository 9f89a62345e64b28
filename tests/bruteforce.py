"""Brute-force references that pin the oracle: they compute the layer the long way round, from
the general memory layer (eq. (1)) over all N slots, and share no code with the oracle.

* Additive product keys: slot (i, j) has the full key [K_row[i], K_col[j]] and the full query
  is [q_row, q_col], so its eq. (1) score is one dot product of length 2 Dk (Sec. 3.1).
* Tucker grid: the exact score of slot (i, j) is the bilinear form
  sum_{rho, sigma} (K_row[rho, i] . q_row[rho]) C[rho, sigma] (K_col[sigma, j] . q_col[sigma])
  of eqs. (4)-(5), evaluated term by term per slot.
* Pooling: a dense [T, N] weight matrix times V (eq. (1), o = V^T s).
* IVE: the materialised virtual table V~ = [V W_0; ...; V W_{E-1}] of eq. (13) and the shuffled
  score vector of eq. (14) -- the "naive reparameterisation" that eq. (15) avoids.
Sizes are tiny; the ordering uses Python's own sort on (-score, index) tuples.
"""
from __future__ import annotations

import numpy as np


def full_keys_additive(K_row, K_col):
    """[H, n*n, 2*Dk] table of full keys: row i*n + j is [K_row[h, i], K_col[h, j]]."""
    H, n, dk = K_row.shape
    full = np.empty((H, n * n, 2 * dk))
    for h in range(H):
        for i in range(n):
            for j in range(n):
                full[h, i * n + j, :dk] = K_row[h, i]
                full[h, i * n + j, dk:] = K_col[h, j]
    return full


def exhaustive_scores_additive(q_row, q_col, K_row, K_col):
    """eq. (1) scores K q of every slot, [T, H, N], from the full keys and the full query."""
    full = full_keys_additive(np.asarray(K_row, np.float64), np.asarray(K_col, np.float64))
    T, H, dk = q_row.shape
    s = np.empty((T, H, full.shape[1]))
    for t in range(T):
        for h in range(H):
            qf = np.concatenate([np.asarray(q_row[t, h], np.float64), np.asarray(q_col[t, h], np.float64)])
            s[t, h] = full[h] @ qf
    return s


def exhaustive_scores_tucker(q_row, q_col, K_row, K_col, core, rank):
    """Exact Tucker score of every slot, [T, H, N], term by term."""
    T, H, dk = q_row.shape
    n = K_row.shape[1]
    w = dk // rank
    s = np.zeros((T, H, n * n))
    for t in range(T):
        for h in range(H):
            for i in range(n):
                for j in range(n):
                    acc = 0.0
                    for rho in range(rank):
                        a = sum(float(K_row[h, i, rho * w + d]) * float(q_row[t, h, rho * w + d]) for d in range(w))
                        for sig in range(rank):
                            b = sum(float(K_col[h, j, sig * w + d]) * float(q_col[t, h, sig * w + d]) for d in range(w))
                            acc += a * float(core[h, rho, sig]) * b
                    s[t, h, i * n + j] = acc
    return s


def ranked(scores, m):
    """Indices of the m best entries under (score desc, index asc), by Python's sort."""
    order = sorted(range(len(scores)), key=lambda x: (-float(scores[x]), x))
    return np.array(order[:m], dtype=np.int64)


def dense_pool(V, idx, w, n_rows):
    """out = W_dense @ V with W_dense[t, row] = sum of the weights selecting that row."""
    T, bag = idx.shape
    W = np.zeros((T, n_rows))
    for t in range(T):
        for b in range(bag):
            W[t, idx[t, b]] += w[t, b]
    return W @ np.asarray(V, np.float64)


def naive_ive(V, W_proj, perm, idx, w, W_out=None):
    """o = V~^T s^ with V~ materialised (eq. (13)) and s^ = Shuffle(vec(S_grid)) (eq. (14))."""
    E, dv, dvv = W_proj.shape
    Np = V.shape[0]
    Vt = np.concatenate([np.asarray(V, np.float64) @ np.asarray(W_proj[p], np.float64) for p in range(E)], axis=0)
    T, bag = idx.shape
    out = np.zeros((T, dvv))
    for t in range(T):
        s_hat = np.zeros(E * Np)
        for b in range(bag):
            s_hat[perm[idx[t, b]]] += w[t, b]
        out[t] = Vt.T @ s_hat
    if W_out is not None:
        out = out @ np.asarray(W_out, np.float64)
    return out


def svd2_closed_form(C):
    """Singular values of a 2x2 matrix from the eigenvalues of C^T C (quadratic formula)."""
    M = np.asarray(C, np.float64).T @ np.asarray(C, np.float64)
    tr = M[0, 0] + M[1, 1]
    det = M[0, 0] * M[1, 1] - M[0, 1] * M[1, 0]
    disc = np.sqrt(max(tr * tr / 4 - det, 0.0))
    return np.sqrt(tr / 2 + disc), np.sqrt(max(tr / 2 - disc, 0.0))
