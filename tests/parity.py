"""Staged comparison of the GPU path with the oracle.

Index results must match exactly, except where the oracle's own fp64 scores put an element
within ``gap`` (1e-6) of the selection threshold: there the fp32 rounding of the GPU scores may
legitimately decide the other way.  Such exemptions are counted and reported.

* Stage A: per-axis top-k sets, against the oracle's threshold theta_k.
* Stage B: the oracle's grid top-m computed on the GPU's own axis sets, against theta_m.
* Stage C: each GPU weight against the exact fp64 score of the slot the GPU chose.
* Stage D: pooling, the oracle's gather-sum on the GPU's own (idx, w).
"""
from __future__ import annotations

import numpy as np

import oracle.umem_oracle as O

GAP = 1e-6


def exact_grid_scores(S_row, S_col, flat, n, grid, C):
    """fp64 grid score of logical slots ``flat`` of one (token, head)."""
    i, j = np.asarray(flat) // n, np.asarray(flat) % n
    if grid == O.GRID_ADD:
        return S_row[0, i] + S_col[0, j]
    C = np.asarray(C, np.float64)
    g = np.zeros(len(i))
    for rho in range(C.shape[0]):
        for sig in range(C.shape[0]):
            g += S_row[rho, i] * C[rho, sig] * S_col[sig, j]
    return g


def _check_sorted(scores, ids, gap, what):
    for a in range(len(ids) - 1):
        assert scores[a] >= scores[a + 1] - gap, f"{what}: not sorted at {a}"
        if scores[a] == scores[a + 1]:
            assert ids[a] < ids[a + 1], f"{what}: tie not broken by index at {a}"


def check_selection(cfg, q_row, q_col, K_row, K_col, core, gpu_idx, gpu_w, gpu_axis=None,
                    gap=GAP, w_rtol=1e-5):
    """Stages A-C for tokens whose queries are q_row/q_col [T, H, Dk].  gpu_idx: [T, H, m];
    gpu_w: [T, H, m], or [T, H, m, h] with multi-core scoring (core then holds the component
    cores [H, h, r, r]); gpu_axis: [2, T, H, k] or None.  Returns (oracle result, report)."""
    parts = None
    if cfg.cores > 1:
        parts, core = np.asarray(core, np.float64), np.asarray(core, np.float64).sum(axis=1)
        ref = O.score_topk(q_row, q_col, K_row, K_col, cfg.topk, cfg.topm, cfg.grid, cfg.weight,
                           None, cfg.rank, core_parts=parts)
    else:
        ref = O.score_topk(q_row, q_col, K_row, K_col, cfg.topk, cfg.topm, cfg.grid, cfg.weight,
                           core, cfg.rank)
    T, H, m = gpu_idx.shape
    n, k = cfg.n_keys, cfg.topk
    rep = dict(tokens=T, axis_exempt=0, grid_exempt=0, e2e_slot_mismatch=0, max_w_err=0.0)
    for t in range(T):
        for h in range(H):
            C = None if core is None else core[h]
            if gpu_axis is not None:
                for axis, sel in ((0, ref["sel_row"][t, h]), (1, ref["sel_col"][t, h])):
                    g_list = [int(x) for x in gpu_axis[axis, t, h]]
                    r_list = [int(x) for x in ref["axis_idx"][axis, t, h]]
                    assert len(set(g_list)) == k and all(0 <= x < n for x in g_list), (t, h, axis)
                    theta = sel[r_list[-1]]
                    for x in set(g_list) ^ set(r_list):
                        assert abs(sel[x] - theta) < gap, ("stage A", t, h, axis, x, sel[x], theta)
                        rep["axis_exempt"] += 1
                    _check_sorted(sel[g_list], g_list, gap, f"axis order t={t} h={h} axis={axis}")
                I_row, I_col = gpu_axis[0, t, h], gpu_axis[1, t, h]
            else:
                I_row, I_col = ref["axis_idx"][0, t, h], ref["axis_idx"][1, t, h]
            gi = [int(x) for x in gpu_idx[t, h]]
            assert len(set(gi)) == m, ("duplicate slots", t, h)
            rows, cols = set(int(x) for x in I_row), set(int(x) for x in I_col)
            assert all(x // n in rows and x % n in cols for x in gi), ("slot outside candidates", t, h)
            flat_b, g_b = O.grid_topm(ref["S_row"][t, h], ref["S_col"][t, h], I_row, I_col, n, m,
                                      cfg.grid, C)
            theta_m = g_b[-1]
            g_gpu = exact_grid_scores(ref["S_row"][t, h], ref["S_col"][t, h], gi, n, cfg.grid, C)
            g_of = dict(zip(gi, g_gpu))
            for x in set(gi) ^ set(int(f) for f in flat_b):
                gx = g_of[x] if x in g_of else exact_grid_scores(ref["S_row"][t, h], ref["S_col"][t, h], [x], n, cfg.grid, C)[0]
                assert abs(gx - theta_m) < gap, ("stage B", t, h, x, gx, theta_m)
                rep["grid_exempt"] += 1
            _check_sorted(g_gpu, gi, gap, f"grid order t={t} h={h}")
            if parts is not None:
                # eq. (16): each core's exact score of the GPU's slots
                w_ref = O.core_scores(ref["S_row"][t, h], ref["S_col"][t, h], gi, n, parts[h])
                scale = max(np.abs(w_ref).max(), 1e-30)
            elif cfg.weight == O.W_RAW:
                w_ref = g_gpu
                scale = max(np.abs(g_gpu).max(), 1e-30)
            else:
                w_ref = O.pooling_weights(g_gpu, O.W_SOFTMAX)
                scale = 1.0
            err = np.abs(np.asarray(gpu_w[t, h], np.float64) - w_ref).max() / scale
            assert err <= w_rtol, ("stage C", t, h, err)
            rep["max_w_err"] = max(rep["max_w_err"], float(err))
            rep["e2e_slot_mismatch"] += m - len(set(gi) & set(int(x) for x in ref["idx"][t, h]))
    return ref, rep


def check_pooled(cfg, value_rows, gpu_idx, gpu_w, gpu_pooled, perm=None, rtol=1e-5):
    """Stage D: oracle gather-sum on the GPU's (idx, w) vs the GPU's pooled [T, E, Dv].
    Error per token: max |diff| / max |reference|."""
    T = gpu_idx.shape[0]
    idx = np.asarray(gpu_idx).reshape(T, -1)
    w = np.asarray(gpu_w, np.float64)
    w = w.reshape(T, idx.shape[1], -1) if cfg.cores > 1 else w.reshape(T, -1)
    ref = O.gather_sum(value_rows, idx, w, perm, cfg.n_values, cfg.expand)
    got = np.asarray(gpu_pooled, np.float64).reshape(ref.shape)
    worst = 0.0
    for t in range(T):
        den = max(np.abs(ref[t]).max(), 1e-30)
        err = np.abs(got[t] - ref[t]).max() / den
        worst = max(worst, float(err))
        assert err <= rtol, ("stage D", t, err)
    return ref, worst
