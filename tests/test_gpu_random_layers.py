"""Seeded random layer shapes through the whole forward, against the oracle (Sec. 3.1 eqs.
(1)-(3); Sec. 3.2 eqs. (4)-(17)).

Each case draws one valid layer inside the library's limits: grid (additive or Tucker of rank
1-4), key count, key width, k and m, heads, SoftMax or raw weights, value width and dtype,
multi-core scoring, implicit value expansion with its projection or the output linear alone, the
token count (across the single-wave, wide and plane scoring kernels and the pooling selection),
and Gaussian or clustered queries.  The shapes are fixed by the seeds; `random_layer` is plain
host code, so the same draws are checked on the CPU (tests/test_abi_host.py) to be accepted by
the descriptor checks.
"""
import numpy as np
import pytest

from synth import configs as CF

N_CASES = 64


def _additive_candidates(k, m):
    return sum(min(k, m // (a + 1)) for a in range(min(k, m)))


def random_layer(i: int) -> CF.Layer:
    rng = np.random.default_rng(9000 + i)
    tucker = bool(rng.random() < 0.5)
    rank = int(rng.choice([1, 2, 3, 4])) if tucker else 1
    if rng.random() < 0.5:                                    # (dk / rank) % 4 == 0, <= 256
        dk = rank * 4 * int(rng.integers(1, 17))
    else:                                                     # also a plane-scoring width
        dk = int(rng.choice([d for d in (32, 64, 96, 128, 192, 256) if (d // rank) % 8 == 0 and d % rank == 0]))
    n = int(rng.integers(8, 257))
    if rng.random() < 0.5:
        n -= n % 4
    k = int(rng.integers(1, min(n, 64 if tucker else 90) + 1))
    m = int(rng.integers(1, min(k * k, 256) + 1))
    while not tucker and _additive_candidates(k, m) > 2048:
        m = max(1, m // 2)
    heads = int(rng.integers(1, 5))
    vdtype = CF.F32 if rng.random() < 0.5 else CF.BF16
    esize = 4 if vdtype == CF.F32 else 2
    row_bytes = int(rng.choice([16, 64, 256, 1024, 2048, 4096]))
    dv = row_bytes // esize
    cores = 1
    if tucker and rng.random() < 0.6:
        for h in (2, 4, 3):
            if dv % h == 0 and (dv // h) * esize % 16 == 0:
                cores = h
                break
    softmax = cores == 1 and bool(rng.random() < 0.3)
    expand, dv_virt, d_out = 1, 0, 0
    r = rng.random()
    if r < 0.25 and n % 2 == 0 and dv % 8 == 0:
        expand = 4
        dv_virt = 8 * int(rng.integers(1, 33))
        d_out = 8 * int(rng.integers(0, 33))
    elif r < 0.4 and dv % 8 == 0:
        d_out = 8 * int(rng.integers(1, 33))                # the output linear alone
    T = int(rng.choice([1, 3, 17, 40, 64, 65, 130, 300]))
    queries = "clusters" if rng.random() < 0.25 else "gauss"
    return CF.Layer(f"random-{i}", T=T, heads=heads, dk=dk, n_keys=n, topk=k, topm=m, dv=dv,
                    vdtype=vdtype, seed=500 + i, rank=rank,
                    grid=CF.GRID_TUCKER if tucker else CF.GRID_ADD,
                    weight=CF.W_SOFTMAX if softmax else CF.W_RAW, expand=expand,
                    dv_virt=dv_virt, d_out=d_out, queries=queries, cores=cores)


N_FRONT_ENDS = 16


def random_front_end(i: int) -> CF.FrontEnd:
    """A query front-end inside the library's limits (Sec. 3.2 Tricks 2, 4, 5): hidden width a
    multiple of 8, up to eight taps, 1-4 heads of Dk up to 1024, shared or separate queries, with
    or without history."""
    rng = np.random.default_rng(9500 + i)
    shared = bool(rng.random() < 0.5)
    heads = int(rng.integers(1, 5))
    while True:
        dk = int(rng.choice([int(rng.integers(1, 129)), int(rng.integers(129, 1025))]))
        if ((1 if shared else 2) * heads * dk) % 8 == 0:
            break
    return CF.FrontEnd(f"random-fe-{i}", B=int(rng.integers(1, 9)), L=int(rng.integers(1, 65)),
                       d_model=8 * int(rng.integers(1, 257)), conv_k=int(rng.integers(1, 9)),
                       heads=heads, dk=dk, shared=shared, seed=600 + i,
                       history=bool(rng.random() < 0.7))


@pytest.mark.gpu
@pytest.mark.parametrize("i", range(N_CASES))
def test_random_layer(i):
    from tests.test_gpu_parity import run_and_check
    cfg = random_layer(i)
    run_and_check(cfg, tokens=None if cfg.T <= 64 else np.arange(0, cfg.T, 5))


@pytest.mark.gpu
@pytest.mark.parametrize("i", range(0, N_CASES, 2))
def test_random_layer_backward(i):
    """The backward of every other random layer at the GPU forward's own selection, against the
    backward oracle: the value-row and weight gradients (eqs. (1), (15), (17) differentiated, in
    the dense and the compact form), then the query, key and core gradients (eqs. (2)-(4), (10),
    (16) differentiated)."""
    import torch
    import oracle.backward_oracle as B
    from synth import device as SD
    from tests import gpu_util as G
    from tests.test_gpu_backward import (RTOL, rel, run_gather_backward, run_gather_backward_rows,
                                         run_score_backward)
    cfg = random_layer(i)
    print(f"[case] random backward {cfg}", flush=True)
    dl = SD.make_layer(cfg)
    T = cfg.T
    idx, w, _ = G.score_topk(dl, T, 0)
    rng = np.random.default_rng(700 + i)
    # b1: value rows and weights
    dp = rng.standard_normal((T, cfg.expand, cfg.dv)).astype(np.float32)
    dV = torch.zeros((cfg.n_values, cfg.dv), dtype=torch.float32, device="cuda")
    wshape = (T, cfg.bag) + ((cfg.cores,) if cfg.cores > 1 else ())
    dw_g = run_gather_backward(cfg.n_values, cfg.dv, cfg.vdtype, dl.values, T, cfg.bag,
                               idx.reshape(T, cfg.bag), w.reshape(wshape), dl.perm, cfg.expand,
                               cfg.cores, torch.from_numpy(dp).cuda(), dV)
    # b1 in compact form: the distinct rows, each equal bit for bit to the dense (zeroed) row
    rows_c, d_rows, n_rows, dw_c = run_gather_backward_rows(
        cfg.n_values, cfg.dv, cfg.vdtype, dl.values, T, cfg.bag, idx.reshape(T, cfg.bag),
        w.reshape(wshape), dl.perm, cfg.expand, cfg.cores, torch.from_numpy(dp).cuda())
    # b2: queries, keys, core
    dw_s = rng.standard_normal(tuple(w.shape)).astype(np.float32)
    dq_row, dq_col, dk_row, dk_col, dcore = run_score_backward(cfg, dl, idx, w, torch.from_numpy(dw_s).cuda())
    torch.cuda.synchronize()
    idx_h, w_h = G.host(idx), G.host(w)
    rows, dV_ref, dw_ref = B.gather_backward(G.value_rows_fn(cfg), idx_h.reshape(T, cfg.bag),
                                             w_h.reshape(wshape), dp, CF.perm(cfg), cfg.n_values,
                                             cfg.expand)
    errs = dict(dV=rel(G.host(dV)[rows], dV_ref), dw=rel(G.host(dw_g), dw_ref))
    n = int(n_rows.item())
    assert n == len(rows) and np.array_equal(rows_c[:n].cpu().numpy(), np.sort(rows))
    assert torch.equal(d_rows[:n], dV[rows_c[:n].long()]) and torch.equal(dw_c, dw_g)
    qr, qc = CF.queries(cfg)
    kr, kc = CF.keys(cfg)
    core = CF.core(cfg)
    res = B.score_backward(qr, qc, kr, kc, idx_h, dw_s, w_h, cfg.grid, cfg.weight,
                           None if cfg.cores > 1 else core, cfg.rank,
                           core if cfg.cores > 1 else None)
    errs.update(dq_row=rel(G.host(dq_row), res["dq_row"]), dq_col=rel(G.host(dq_col), res["dq_col"]),
                dk_row=rel(G.host(dk_row), res["dK_row"]), dk_col=rel(G.host(dk_col), res["dK_col"]))
    if dcore is not None:
        errs["dcore"] = rel(G.host(dcore), res["dC"])
    print(f"[report] random backward {cfg.name}: {errs}", flush=True)
    assert max(errs.values()) <= RTOL, errs


@pytest.mark.gpu
@pytest.mark.parametrize("i", range(N_FRONT_ENDS))
def test_random_front_end(i):
    """Random query front-ends against the front-end oracle (causal convolution, query linear,
    per-head LayerNorm), to the tolerance of the bf16 query linear."""
    from tests.test_gpu_query import (Q_RTOL, ROUNDED_RTOL, oracle_queries, rounded_rows_queries,
                                      row_err, run_query)
    fe = random_front_end(i)
    inp, q_row, q_col, _ = run_query(fe)
    got = (q_row.cpu().numpy(), q_col.cpu().numpy())
    # 1. against the oracle's steps with the query linear's documented input rounding
    ref16 = rounded_rows_queries(fe, inp)
    e16 = max(row_err(got[a], ref16[:, 0 if fe.shared else a]) for a in (0, 1))
    # 2. against the plain fp64 oracle, to the query tolerance; a LayerNorm over a handful of
    # values (Dk < 16) can divide the linear's rounding by a spread far below the values' size,
    # so there the first check stands alone
    qr_ref, qc_ref = oracle_queries(fe, inp)
    er, ec = row_err(got[0], qr_ref), row_err(got[1], qc_ref)
    print(f"[report] {fe}: against bf16-rounded rows {e16:.2e}; against fp64 q_row {er:.2e}, "
          f"q_col {ec:.2e}", flush=True)
    assert e16 <= ROUNDED_RTOL
    if fe.dk >= 16:
        assert er <= Q_RTOL and ec <= Q_RTOL
