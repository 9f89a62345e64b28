"""Pins of the oracle: each function checks one part of the oracle module ``O`` against something
other than itself -- hand-worked fixtures under tests/golden/, the exhaustive eq. (1) scoring of
all N slots, closed forms, invariants the paper states, or brute force on tiny inputs.

Each pin raises AssertionError on a mismatch.  They take the oracle module as an argument so that
the mutation tests can run them against copies with planted mistakes.
"""
from __future__ import annotations

import json
import math
import os

import numpy as np

from tests import bruteforce as BF

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _arr(x):
    return np.asarray(x, dtype=np.float64)


def _grid(O, name):
    return O.GRID_ADD if name == "add" else O.GRID_TUCKER


# ---------------------------------------------------------------- golden (hand-worked) fixtures

def pin_golden_additive(O):
    g = _golden("additive_ties_n3.json")
    res = O.score_topk(_arr(g["q_row"]), _arr(g["q_col"]), _arr(g["K_row"]), _arr(g["K_col"]),
                       g["topk"], g["topm"], O.GRID_ADD, O.W_RAW)
    assert list(res["axis_idx"][0, 0, 0]) == g["expect_axis_row"]
    assert list(res["axis_idx"][1, 0, 0]) == g["expect_axis_col"]
    assert list(res["idx"][0, 0]) == g["expect_idx"]
    assert np.array_equal(res["w"][0, 0], g["expect_scores"])
    sm = O.score_topk(_arr(g["q_row"]), _arr(g["q_col"]), _arr(g["K_row"]), _arr(g["K_col"]),
                      g["topk"], g["topm"], O.GRID_ADD, O.W_SOFTMAX)
    e = math.e
    assert np.allclose(sm["w"][0, 0], np.array([e, e, 1.0]) / (2 * e + 1), rtol=1e-14, atol=0)
    V = _arr(g["values"])
    out, _, _ = O.forward(_arr(g["q_row"]), _arr(g["q_col"]), _arr(g["K_row"]), _arr(g["K_col"]),
                          lambda r: V[r], g["topk"], g["topm"])
    assert np.array_equal(out[0], g["expect_out_raw"])


def pin_golden_tucker(O):
    g = _golden("tucker_masked_n3.json")
    C = _arr(g["core"])
    u, t, _ = O.rank1_factors(C[0])
    assert np.allclose(u, g["expect_u"], atol=1e-15) and np.allclose(t, g["expect_t"], atol=1e-15)
    res = O.score_topk(_arr(g["q_row"]), _arr(g["q_col"]), _arr(g["K_row"]), _arr(g["K_col"]),
                       g["topk"], g["topm"], O.GRID_TUCKER, O.W_RAW, core=C, rank=g["rank"])
    assert list(res["axis_idx"][0, 0, 0]) == g["expect_axis_row"]
    assert list(res["axis_idx"][1, 0, 0]) == g["expect_axis_col"]
    assert list(res["idx"][0, 0]) == g["expect_idx"]
    assert np.array_equal(res["w"][0, 0], g["expect_scores"])
    V = _arr(g["values"])
    out, _, _ = O.forward(_arr(g["q_row"]), _arr(g["q_col"]), _arr(g["K_row"]), _arr(g["K_col"]),
                          lambda r: V[r], g["topk"], g["topm"], O.GRID_TUCKER, O.W_RAW, core=C,
                          rank=g["rank"])
    assert np.array_equal(out[0], g["expect_out_raw"])


def pin_golden_signed_zero(O):
    g = _golden("signed_zero_ties_n4.json")
    res = O.score_topk(_arr(g["q_row"]), _arr(g["q_col"]), _arr(g["K_row"]), _arr(g["K_col"]),
                       g["topk"], g["topm"])
    assert list(res["axis_idx"][0, 0, 0]) == g["expect_axis_row"]
    assert list(res["axis_idx"][1, 0, 0]) == g["expect_axis_col"]
    assert list(res["idx"][0, 0]) == g["expect_idx"]


def pin_golden_ive(O):
    g = _golden("ive_reversal_e4.json")
    V = _arr(g["values"])
    idx = np.array(g["idx"])
    pooled = O.gather_sum(lambda r: V[r], idx, _arr(g["w"]), np.array(g["perm"]), g["n_values"],
                          g["expand"])
    assert np.array_equal(pooled, g["expect_pooled"])
    assert np.array_equal(O.ive_project(pooled, _arr(g["W_proj"])), g["expect_projected"])
    assert np.array_equal(O.ive_project(pooled, _arr(g["W_proj"]), _arr(g["W_out"])), g["expect_out"])


def pin_golden_svd(O):
    g = _golden("svd_core_3045.json")
    C = _arr(g["core"])
    u, t, sig = O.rank1_factors(C)
    assert np.allclose(sig, [3 * math.sqrt(5), math.sqrt(5)], rtol=1e-14)
    assert np.allclose(u, [1 / math.sqrt(10), 3 / math.sqrt(10)], rtol=1e-14)
    assert np.allclose(t, [1 / math.sqrt(2), 1 / math.sqrt(2)], rtol=1e-14)
    u2, t2, _ = O.rank1_factors(-C)
    assert np.allclose(u2, u, rtol=1e-14) and np.allclose(t2, -t, rtol=1e-14)


# ---------------------------------------------------------------- exhaustive eq. (1) scoring

def _rand_layer(rng, n, dk, T, H, quantise=False):
    def draw(shape):
        x = rng.standard_normal(shape)
        return np.round(x * 2) if quantise else x
    return draw((T, H, dk)), draw((T, H, dk)), draw((H, n, dk)), draw((H, n, dk))


def pin_scores_full_keys(O, seeds=range(6)):
    """s_row[i] + s_col[j] is the eq. (1) score of slot i*n + j under the full key table."""
    for seed in seeds:
        rng = np.random.default_rng(seed)
        n, dk, T, H = int(rng.integers(2, 9)), int(rng.integers(1, 7)), 2, int(rng.integers(1, 4))
        qr, qc, Kr, Kc = _rand_layer(rng, n, dk, T, H)
        ex = BF.exhaustive_scores_additive(qr, qc, Kr, Kc)
        Sr, Sc = O.axis_scores(qr, Kr, 1), O.axis_scores(qc, Kc, 1)
        for t in range(T):
            for h in range(H):
                grid = Sr[t, h, 0][:, None] + Sc[t, h, 0][None, :]
                assert np.allclose(grid.reshape(-1), ex[t, h], rtol=1e-12, atol=1e-12)


def pin_exhaustive_topm_additive(O, seeds=range(12), quantise=False):
    """Two-phase top-m equals the top-m of all N slots when k >= m (Sec. 3.1)."""
    for seed in seeds:
        rng = np.random.default_rng(1000 + seed)
        n = int(rng.integers(2, 13))
        dk, T, H = int(rng.integers(1, 6)), 3, int(rng.integers(1, 4))
        m = int(rng.integers(1, n + 1))
        k = int(rng.integers(m, n + 1))
        qr, qc, Kr, Kc = _rand_layer(rng, n, dk, T, H, quantise)
        res = O.score_topk(qr, qc, Kr, Kc, k, m)
        ex = BF.exhaustive_scores_additive(qr, qc, Kr, Kc)
        for t in range(T):
            for h in range(H):
                want = BF.ranked(ex[t, h], m)
                assert np.array_equal(res["idx"][t, h], want), (seed, t, h)
                assert np.allclose(res["w"][t, h], ex[t, h][want], rtol=1e-12, atol=1e-12)


def pin_topology_bias(O, seeds=range(8)):
    """With additive scores the second-best slot shares a row or a column with the best (Sec. 3.2)."""
    for seed in seeds:
        rng = np.random.default_rng(2000 + seed)
        n, dk, T, H = 9, 4, 4, 2
        qr, qc, Kr, Kc = _rand_layer(rng, n, dk, T, H)
        res = O.score_topk(qr, qc, Kr, Kc, 4, 2)
        for t in range(T):
            for h in range(H):
                a, b = res["idx"][t, h]
                assert a // n == b // n or a % n == b % n


def pin_softmax_full_vector(O, seeds=range(4)):
    """eq. (3): SoftMax of vec(S_grid) with -inf outside the top-m; weights sum to 1."""
    for seed in seeds:
        rng = np.random.default_rng(3000 + seed)
        n, dk, T, H, k, m = 7, 3, 3, 2, 6, 4
        qr, qc, Kr, Kc = _rand_layer(rng, n, dk, T, H)
        res = O.score_topk(qr, qc, Kr, Kc, k, m, O.GRID_ADD, O.W_SOFTMAX)
        ex = BF.exhaustive_scores_additive(qr, qc, Kr, Kc)
        for t in range(T):
            for h in range(H):
                full = np.full(n * n, -np.inf)
                sel = BF.ranked(ex[t, h], m)
                full[sel] = ex[t, h][sel]
                e = np.exp(full - full.max())
                sm = e / e.sum()
                assert np.allclose(res["w"][t, h], sm[res["idx"][t, h]], rtol=1e-12, atol=1e-15)
                assert abs(res["w"][t, h].sum() - 1.0) < 1e-12


def pin_gather_dense(O, seeds=range(4)):
    """Pooling equals the dense product W @ V (eq. (1) o = V^T s); repeated rows add."""
    for seed in seeds:
        rng = np.random.default_rng(4000 + seed)
        N, dv, T, bag = 50, 7, 5, 12
        V = rng.standard_normal((N, dv))
        idx = rng.integers(0, N, size=(T, bag))
        idx[:, 1] = idx[:, 0]                 # force repeats
        w = rng.standard_normal((T, bag))
        out = O.gather_sum(lambda r: V[r], idx, w)
        assert out.shape == (T, 1, dv)
        assert np.allclose(out[:, 0], BF.dense_pool(V, idx, w, N), rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------- Tucker (TDQKR)

def pin_svd_closed_form(O, seeds=range(20)):
    """2x2 cores: sigma from C^T C's eigenvalues; C t = sigma_1 u; sign rule; unit vectors."""
    for seed in seeds:
        rng = np.random.default_rng(5000 + seed)
        C = rng.standard_normal((2, 2))
        u, t, sig = O.rank1_factors(C)
        s1, s2 = BF.svd2_closed_form(C)
        assert np.allclose(sig, [s1, s2], rtol=1e-10, atol=1e-12)
        assert abs(np.linalg.norm(u) - 1) < 1e-12 and abs(np.linalg.norm(t) - 1) < 1e-12
        assert np.allclose(C @ t, s1 * u, atol=1e-10)
        assert np.allclose(C.T @ u, s1 * t, atol=1e-10)
        j = int(np.argmax(np.abs(u)))
        assert u[j] > 0


def pin_svd_power_iteration(O, seeds=range(8)):
    """r = 3, 4: the leading pair agrees with plain power iteration on C^T C."""
    for seed in seeds:
        rng = np.random.default_rng(6000 + seed)
        r = 3 + seed % 2
        C = rng.standard_normal((r, r))
        x = np.ones(r)
        for _ in range(5000):
            x = C.T @ (C @ x)
            x /= np.linalg.norm(x)
        s1 = np.linalg.norm(C @ x)
        u_pi = C @ x / s1
        if u_pi[int(np.argmax(np.abs(u_pi)))] < 0:
            u_pi = -u_pi
        u, t, sig = O.rank1_factors(C)
        assert abs(sig[0] - s1) < 1e-9 * s1
        assert np.allclose(u, u_pi, atol=1e-7)


def _positive_layer(rng, n, dk, T, H):
    qr = rng.uniform(0.1, 1.0, (T, H, dk))
    qc = rng.uniform(0.1, 1.0, (T, H, dk))
    Kr = rng.uniform(0.1, 1.0, (H, n, dk))
    Kc = rng.uniform(0.1, 1.0, (H, n, dk))
    return qr, qc, Kr, Kc


def pin_tucker_rank1_core_exact(O, seeds=range(6)):
    """A rank-1 core a b^T with a, b > 0 and positive axis scores makes the approximate
    retrieval exact: it equals the exhaustive top-m of the exact Tucker score (k >= m)."""
    for seed in seeds:
        rng = np.random.default_rng(7000 + seed)
        n, r, T, H = 6, 2, 2, 2
        dk = 2 * r
        qr, qc, Kr, Kc = _positive_layer(rng, n, dk, T, H)
        core = np.stack([np.outer(rng.uniform(0.5, 2, r), rng.uniform(0.5, 2, r)) for _ in range(H)])
        m = int(rng.integers(1, 6))
        k = int(rng.integers(m, n + 1))
        res = O.score_topk(qr, qc, Kr, Kc, k, m, O.GRID_TUCKER, O.W_RAW, core=core, rank=r)
        ex = BF.exhaustive_scores_tucker(qr, qc, Kr, Kc, core, r)
        for t in range(T):
            for h in range(H):
                want = BF.ranked(ex[t, h], m)
                assert np.array_equal(res["idx"][t, h], want), (seed, t, h)
                assert np.allclose(res["w"][t, h], ex[t, h][want], rtol=1e-12)


def pin_tucker_exact_scores(O, seeds=range(4)):
    """For any core, each selected slot's weight is its exact Tucker score (eqs. (5), (10)), and
    every selected slot lies in I_row x I_col."""
    for seed in seeds:
        rng = np.random.default_rng(8000 + seed)
        n, r, T, H, k, m = 7, 2, 2, 2, 3, 4
        qr, qc, Kr, Kc = _rand_layer(rng, n, 2 * r, T, H)
        core = rng.standard_normal((H, r, r))
        res = O.score_topk(qr, qc, Kr, Kc, k, m, O.GRID_TUCKER, O.W_RAW, core=core, rank=r)
        ex = BF.exhaustive_scores_tucker(qr, qc, Kr, Kc, core, r)
        for t in range(T):
            for h in range(H):
                idx = res["idx"][t, h]
                assert np.allclose(res["w"][t, h], ex[t, h][idx], rtol=1e-12, atol=1e-12)
                assert set(idx // n) <= set(res["axis_idx"][0, t, h])
                assert set(idx % n) <= set(res["axis_idx"][1, t, h])
                # the selected set is the best m of the candidate set, by brute force
                cand = [i * n + j for i in res["axis_idx"][0, t, h] for j in res["axis_idx"][1, t, h]]
                best = sorted(cand, key=lambda x: (-ex[t, h][x], x))[:m]
                assert list(idx) == best


def pin_tucker_rank_one_slices(O, seeds=range(4)):
    """r = 1 with a positive 1x1 core: the score is c * s_row[i] * s_col[j]; with positive axis
    scores the two-phase result equals the exhaustive top-m of that product (k >= m)."""
    for seed in seeds:
        rng = np.random.default_rng(9000 + seed)
        n, dk, T, H = 8, 3, 2, 1
        qr, qc, Kr, Kc = _positive_layer(rng, n, dk, T, H)
        core = np.array([[[rng.uniform(0.5, 2.0)]]])
        res = O.score_topk(qr, qc, Kr, Kc, 5, 5, O.GRID_TUCKER, O.W_RAW, core=core, rank=1)
        for t in range(T):
            sr = [sum(Kr[0, i, d] * qr[t, 0, d] for d in range(dk)) for i in range(n)]
            sc = [sum(Kc[0, j, d] * qc[t, 0, d] for d in range(dk)) for j in range(n)]
            prod = [core[0, 0, 0] * sr[i] * sc[j] for i in range(n) for j in range(n)]
            assert np.array_equal(res["idx"][t, 0], BF.ranked(prod, 5))


# ---------------------------------------------------------------- IVE

def pin_ive_materialised(O, seeds=range(4)):
    """Pool-per-block then project (eq. (15)) equals pooling the materialised, shuffled virtual
    table (eqs. (13)-(14))."""
    for seed in seeds:
        rng = np.random.default_rng(10000 + seed)
        E, n_p, dv, dvv, T, bag = 4, 3, 5, 6, 3, 10
        Np = n_p * n_p
        V = rng.standard_normal((Np, dv))
        Wp = rng.standard_normal((E, dv, dvv))
        Wo = rng.standard_normal((dvv, 4))
        perm = rng.permutation(E * Np)
        idx = rng.integers(0, E * Np, size=(T, bag))
        w = rng.standard_normal((T, bag))
        pooled = O.gather_sum(lambda r: V[r], idx, w, perm, Np, E)
        got = O.ive_project(pooled, Wp, Wo)
        assert np.allclose(got, BF.naive_ive(V, Wp, perm, idx, w, Wo), rtol=1e-10, atol=1e-10)


def pin_ive_concat_same_column(O):
    """Without the shuffle, a physical row's E virtual copies sit in one logical column -- the
    topology the paper's shuffle removes (Sec. 3.2 IVE).  n_v = sqrt(E) n_p, n_p even."""
    for E, n_p in ((4, 2), (4, 6), (16, 4)):
        n_v = int(math.isqrt(E)) * n_p
        Np = n_p * n_p
        x = np.arange(n_v * n_v)
        p, row = O.address_map(x.reshape(1, -1), np.arange(E * Np), Np, E)
        p, row = p[0], row[0]
        assert set(p) == set(range(E))
        for r in range(Np):
            cols = set((x[row == r] % n_v).tolist())
            assert len(cols) == 1 and len(x[row == r]) == E


# ---------------------------------------------------------------- multi-core scoring

def pin_golden_mcs(O):
    g = _golden("mcs_two_cores_n2.json")
    args = (_arr(g["q_row"]), _arr(g["q_col"]), _arr(g["K_row"]), _arr(g["K_col"]), g["topk"])
    V = _arr(g["values"])
    res = O.score_topk(*args, 2, O.GRID_TUCKER, O.W_RAW, rank=g["rank"], core_parts=_arr(g["core_parts"]))
    assert list(res["idx"][0, 0]) == g["expect_idx_m2"]
    assert np.allclose(res["g"][0, 0], g["expect_g_m2"], rtol=0, atol=1e-12)
    assert np.allclose(res["w_core"][0, 0], g["expect_w_core_m2"], rtol=0, atol=1e-12)
    out, _, _ = O.forward(*args[:4], lambda r: V[r], g["topk"], 2, O.GRID_TUCKER, O.W_RAW,
                          rank=g["rank"], core_parts=_arr(g["core_parts"]))
    assert np.allclose(out[0], g["expect_out_m2"], rtol=0, atol=1e-12)
    res3 = O.score_topk(*args, 3, O.GRID_TUCKER, O.W_RAW, rank=g["rank"], core_parts=_arr(g["core_parts"]))
    assert list(res3["idx"][0, 0]) == g["expect_idx_m3"]
    assert np.allclose(res3["w_core"][0, 0], g["expect_w_core_m3"], rtol=0, atol=1e-12)


def pin_mcs_scores_add_up(O, seeds=range(4)):
    """eq. (16): the component scores of every selected slot add up to its grid score, and the
    selection is the one the summed core makes; one component reproduces the plain grid."""
    for seed in seeds:
        rng = np.random.default_rng(11000 + seed)
        n, r, T, H, k, m, h = 7, 2, 2, 2, 4, 6, 3
        qr, qc, Kr, Kc = _rand_layer(rng, n, 2 * r, T, H)
        parts = rng.standard_normal((H, h, r, r))
        res = O.score_topk(qr, qc, Kr, Kc, k, m, O.GRID_TUCKER, O.W_RAW, rank=r, core_parts=parts)
        whole = O.score_topk(qr, qc, Kr, Kc, k, m, O.GRID_TUCKER, O.W_RAW, core=parts.sum(axis=1), rank=r)
        assert np.array_equal(res["idx"], whole["idx"])
        assert np.allclose(res["w_core"].sum(axis=3), whole["g"], rtol=1e-12, atol=1e-12)
        ex = BF.exhaustive_scores_tucker(qr, qc, Kr, Kc, parts[:, 1], r)   # core 1 alone, all slots
        for t in range(T):
            for hd in range(H):
                assert np.allclose(res["w_core"][t, hd, :, 1], ex[t, hd][res["idx"][t, hd]],
                                   rtol=1e-12, atol=1e-12)
        one = O.score_topk(qr, qc, Kr, Kc, k, m, O.GRID_TUCKER, O.W_RAW, rank=r, core_parts=parts[:, :1])
        assert np.array_equal(one["w_core"][..., 0], one["g"])


def pin_mcs_dense_pool(O, seeds=range(3)):
    """eq. (17) as written: dense score vectors s^(i) over all N slots, o = [s^(1)T V^(1), ...];
    with IVE, the physical rows split, per virtual block (eq. (15))."""
    for seed in seeds:
        rng = np.random.default_rng(12000 + seed)
        h, dv, T, bag, Np = 2, 6, 3, 9, 16
        V = rng.standard_normal((Np, dv))
        idx = rng.integers(0, Np, size=(T, bag))
        idx[:, 1] = idx[:, 0]                      # a repeated slot adds
        w = rng.standard_normal((T, bag, h))
        got = O.gather_sum(lambda r: V[r], idx, w, None, Np, 1)[:, 0, :]
        want = np.concatenate([BF.dense_pool(V[:, c * dv // h:(c + 1) * dv // h], idx, w[:, :, c], Np)
                               for c in range(h)], axis=1)
        assert np.allclose(got, want, rtol=1e-12, atol=1e-12)
        E = 4
        perm = rng.permutation(E * Np)
        idx = rng.integers(0, E * Np, size=(T, bag))
        pooled = O.gather_sum(lambda r: V[r], idx, w, perm, Np, E)
        v = perm[idx]
        for p in range(E):
            wp = np.where((v // Np) == p, 1.0, 0.0)[:, :, None] * w
            want = np.concatenate([BF.dense_pool(V[:, c * dv // h:(c + 1) * dv // h], v % Np, wp[:, :, c], Np)
                                   for c in range(h)], axis=1)
            assert np.allclose(pooled[:, p, :], want, rtol=1e-12, atol=1e-12)


ALL_PINS = [
    pin_golden_additive, pin_golden_tucker, pin_golden_signed_zero, pin_golden_ive, pin_golden_svd,
    pin_scores_full_keys, pin_exhaustive_topm_additive,
    lambda O: pin_exhaustive_topm_additive(O, seeds=range(12, 20), quantise=True),
    pin_topology_bias, pin_softmax_full_vector, pin_gather_dense, pin_svd_closed_form,
    pin_svd_power_iteration, pin_tucker_rank1_core_exact, pin_tucker_exact_scores,
    pin_tucker_rank_one_slices, pin_ive_materialised, pin_ive_concat_same_column,
    pin_golden_mcs, pin_mcs_scores_add_up, pin_mcs_dense_pool,
]


# ---------------------------------------------------------------- the oracle at paper scale

def exhaustive_topm_product_keys(q_row, q_col, K_row, K_col, m):
    """The m best of all n*n slots of one (token, head) under eq. (1) with product keys: slot
    (i, j) has the full key [K_row[i], K_col[j]], so its score against the full query
    [q_row, q_col] is K_row[i].q_row + K_col[j].q_col.  The whole n x n grid is materialised in
    fp64 and ordered by (score desc, flat index i*n + j asc).  Returns (flat indices, scores)."""
    a = np.asarray(K_row, np.float64) @ np.asarray(q_row, np.float64)
    b = np.asarray(K_col, np.float64) @ np.asarray(q_col, np.float64)
    return _exhaustive_topm((a[:, None] + b[None, :]).reshape(-1), m)


def exhaustive_topm_tucker(q_row, q_col, K_row, K_col, C, m):
    """The m best of all n*n slots under the exact Tucker score of eqs. (4)-(5): with the r
    slices of the query/key dim, S_row[rho, i] = K_row[i, slice rho] . q_row[slice rho] (the same
    for columns) and g(i, j) = sum_{rho, sigma} S_row[rho, i] C[rho, sigma] S_col[sigma, j], the
    whole n x n grid in fp64.  Returns (flat indices, scores)."""
    C = np.asarray(C, np.float64)
    r = C.shape[0]
    w = len(q_row) // r
    Sr = np.stack([np.asarray(K_row, np.float64)[:, s * w:(s + 1) * w] @ np.asarray(q_row[s * w:(s + 1) * w], np.float64)
                   for s in range(r)])
    Sc = np.stack([np.asarray(K_col, np.float64)[:, s * w:(s + 1) * w] @ np.asarray(q_col[s * w:(s + 1) * w], np.float64)
                   for s in range(r)])
    return _exhaustive_topm((Sr.T @ C @ Sc).reshape(-1), m)


def _exhaustive_topm(g, m):
    part = np.argpartition(-g, m - 1)[:m]
    cut = g[part].min()                          # the m-th largest score
    cand = np.flatnonzero(g >= cut)              # every slot that can rank among the m best
    order = np.lexsort((cand, -g[cand]))         # score desc, then flat index asc
    best = cand[order[:m]]
    return best, g[best]


def pin_exhaustive_topm_paper_scale(O, cfg_names=("decode-20M", "prefill-1M"), tokens=(0, 1, 2)):
    """Sec. 3.1: with k >= m the two-phase top-m (per-axis top-k, then the grid) is the top-m of
    all N slots.  Checked on the paper-scale layers the oracle is used at: 4480^2 = 20,070,400
    slots of the decode layer and 1024^2 of the prefill layer (k = m = 32, two heads), against
    the whole grid of eq. (1) scores.  Also the raw weights are the exact slot scores."""
    from synth import configs as CF
    for name in cfg_names:
        cfg = CF.CONFIGS[name]
        qr, qc = CF.queries(cfg, batch=0, tokens=np.asarray(tokens))
        kr, kc = CF.keys(cfg)
        res = O.score_topk(qr, qc, kr, kc, cfg.topk, cfg.topm)
        for t in range(len(tokens)):
            for h in range(cfg.heads):
                want, g = exhaustive_topm_product_keys(qr[t, h], qc[t, h], kr[h], kc[h], cfg.topm)
                assert np.array_equal(res["idx"][t, h], want), (name, t, h)
                assert np.allclose(res["w"][t, h], g, rtol=1e-12, atol=1e-15), (name, t, h)


SCALE_PINS = [pin_exhaustive_topm_paper_scale]


def tucker_recall(O, cfg, tokens):
    """Recall@m of the paper's rank-1 retrieval (eqs. (7)-(10): per-axis top-k on the leading
    singular pair's factors, then the exact score of the k*k candidates) against the exhaustive
    exact-Tucker top-m of all n*n slots (the core a head uses; with multi-core scoring, the sum
    of its components, eq. (16)).  Not a pass/fail property: the rank-1 factors only approximate
    the bilinear score (their product has either sign).  Returns per-(token, head) recalls."""
    from synth import configs as CF
    qr, qc = CF.queries(cfg, batch=0, tokens=np.asarray(tokens))
    kr, kc = CF.keys(cfg)
    core = np.asarray(CF.core(cfg), np.float64)
    if cfg.cores > 1:
        core = core.sum(axis=1)
    res = O.score_topk(qr, qc, kr, kc, cfg.topk, cfg.topm, O.GRID_TUCKER, O.W_RAW, core, cfg.rank)
    rec = np.zeros((len(tokens), cfg.heads))
    for t in range(len(tokens)):
        for h in range(cfg.heads):
            want, _ = exhaustive_topm_tucker(qr[t, h], qc[t, h], kr[h], kc[h], core[h], cfg.topm)
            rec[t, h] = len(set(want.tolist()) & set(res["idx"][t, h].tolist())) / cfg.topm
    return rec
