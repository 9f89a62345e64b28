"""GPU parity of the backward (value-row and weight gradients; query, key and core gradients)
through the C ABI, against the backward oracle on the same seeded inputs and the GPU forward's
own selection."""
from __future__ import annotations

import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():     # collected on CPU hosts too; every test here is gpu-marked
    pytest.skip("no GPU", allow_module_level=True)

import oracle.backward_oracle as B                  # noqa: E402
import oracle.umem_oracle as O                      # noqa: E402
import paper_2411_12364_amd as U                    # noqa: E402
import synth as S                                   # noqa: E402
from synth import configs as CF                     # noqa: E402
from synth import device as SD                      # noqa: E402
from tests import gpu_util as G                     # noqa: E402

RTOL = 1e-5          # fp32 sums of fp32 products against fp64


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def rel(got, ref):
    ref = np.asarray(ref, np.float64)
    return float(np.abs(np.asarray(got, np.float64) - ref).max() / max(np.abs(ref).max(), 1e-30))


def run_gather_backward(n_values, dv, vdtype, values, T, bag, idx, w, perm, expand, cores, dp, dV):
    st, nws = U.umem_gather_backward_workspace_size(T, bag, dv)
    U.check(st)
    ws = torch.empty(max(nws, 256), dtype=torch.uint8, device="cuda")
    dw = torch.empty(w.shape, dtype=torch.float32, device="cuda")
    U.check(U.umem_gather_backward(n_values, dv, vdtype, values, T, bag, idx, w, perm, expand, cores,
                                   dp, dV, dw, ws, ws.numel()), "umem_gather_backward")
    return dw


def run_gather_backward_rows(n_values, dv, vdtype, values, T, bag, idx, w, perm, expand, cores, dp):
    """The compact form; rows past the count keep their sentinels (-1 / NaN)."""
    st, nws = U.umem_gather_backward_workspace_size(T, bag, dv)
    U.check(st)
    ws = torch.empty(max(nws, 256), dtype=torch.uint8, device="cuda")
    M = T * bag
    rows = torch.full((M,), -1, dtype=torch.int32, device="cuda")
    d_rows = torch.full((M, dv), float("nan"), dtype=torch.float32, device="cuda")
    n_rows = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    dw = torch.empty(w.shape, dtype=torch.float32, device="cuda")
    U.check(U.umem_gather_backward_rows(n_values, dv, vdtype, values, T, bag, idx, w, perm, expand,
                                        cores, dp, rows, d_rows, n_rows, dw, ws, ws.numel()),
            "umem_gather_backward_rows")
    return rows, d_rows, n_rows, dw


GATHER_BWD_CASES = [
    (512, CF.BF16, 1, 64, 37, 1, 300),        # many repeated rows
    (256, CF.F32, 1, 33, 20, 1, 5000),        # few repeats
    (512, CF.BF16, 4, 96, 25, 2, 200),        # IVE blocks, two cores
    (4096, CF.BF16, 4, 84, 9, 2, 500),        # 8 KiB rows (eight row chunks)
    (64, CF.BF16, 1, 40, 50, 4, 60),          # rows narrower than a wave's chunk, four cores
    (1024, CF.F32, 1, 7, 3, 8, 50000),        # eight cores of fp32 slices
    # d_pooled beyond one XCD's L2 (4 MB)
    (256, CF.F32, 1, 16, 4200, 1, 500),
    (512, CF.BF16, 4, 32, 600, 2, 300),       # IVE blocks, two cores
    # the library's limits: a bag of 2048, E = 64, eight cores
    (64, CF.BF16, 64, 2048, 5, 8, 4096),
]


def gather_backward_inputs(dv, vdtype, expand, bag, T, cores, Np):
    """Seeded bags over min(Np, 4096) rows (forcing repeats), weights, d_pooled; the value
    table from torch's generator."""
    rng = np.random.default_rng(dv + bag + T + cores)
    torch_dt = torch.float32 if vdtype == CF.F32 else torch.bfloat16
    rows_used = min(Np, 4096)
    V = torch.randn((Np, dv), dtype=torch.float32, device="cuda").to(torch_dt)
    idx = rng.integers(0, rows_used * expand, size=(T, bag)).astype(np.int32)
    perm = None
    if expand > 1:
        perm = rng.permutation(Np * expand).astype(np.int32)
        # map the chosen virtual slots onto rows_used physical rows only, to force repeats
        perm = (perm % (rows_used * expand)).astype(np.int32) if Np > rows_used else perm
    w = rng.standard_normal((T, bag) + ((cores,) if cores > 1 else ())).astype(np.float32)
    dp = rng.standard_normal((T, expand, dv)).astype(np.float32)
    dev = dict(idx=torch.from_numpy(idx).cuda(), w=torch.from_numpy(w).cuda(),
               perm=None if perm is None else torch.from_numpy(perm).cuda(), dp=torch.from_numpy(dp).cuda())
    return V, idx, perm, w, dp, dev


@pytest.mark.parametrize("dv,vdtype,expand,bag,T,cores,Np", GATHER_BWD_CASES)
def test_gather_backward(dv, vdtype, expand, bag, T, cores, Np):
    log(f"[case] gather backward dv={dv} E={expand} bag={bag} T={T} cores={cores} Np={Np}")
    V, idx, perm, w, dp, dev = gather_backward_inputs(dv, vdtype, expand, bag, T, cores, Np)
    dV0 = torch.randn((Np, dv), dtype=torch.float32, device="cuda")
    dV = dV0.clone()
    dw = run_gather_backward(Np, dv, vdtype, V, T, bag, dev["idx"], dev["w"], dev["perm"], expand,
                             cores, dev["dp"], dV)
    torch.cuda.synchronize()
    Vh = V.float().cpu().numpy()
    rows, dV_ref, dw_ref = B.gather_backward(lambda r: Vh[r], idx, w, dp, perm, Np, expand)
    got = (dV - dV0).cpu().numpy()
    e_dw = rel(dw.cpu().numpy(), dw_ref)
    e_dv = rel(got[rows], dV_ref)
    untouched = np.setdiff1d(np.arange(Np), rows)
    assert np.array_equal(dV.cpu().numpy()[untouched], dV0.cpu().numpy()[untouched])
    log(f"[report] gather backward dv={dv} E={expand} cores={cores}: {len(rows)} rows, "
        f"dw err {e_dw:.2e}, dV err {e_dv:.2e}")
    assert e_dw <= RTOL and e_dv <= RTOL


@pytest.mark.parametrize("dv,vdtype,expand,bag,T,cores,Np", GATHER_BWD_CASES)
def test_gather_backward_rows(dv, vdtype, expand, bag, T, cores, Np):
    """The compact form: the distinct rows ascending and their count, each row's gradient equal
    bit for bit to what the dense form adds into a zeroed row, the same dw, nothing written past
    the count; and against the backward oracle."""
    log(f"[case] gather backward rows dv={dv} E={expand} bag={bag} T={T} cores={cores} Np={Np}")
    V, idx, perm, w, dp, dev = gather_backward_inputs(dv, vdtype, expand, bag, T, cores, Np)
    dV = torch.zeros((Np, dv), dtype=torch.float32, device="cuda")
    dw_dense = run_gather_backward(Np, dv, vdtype, V, T, bag, dev["idx"], dev["w"], dev["perm"],
                                   expand, cores, dev["dp"], dV)
    rows, d_rows, n_rows, dw = run_gather_backward_rows(Np, dv, vdtype, V, T, bag, dev["idx"], dev["w"],
                                                        dev["perm"], expand, cores, dev["dp"])
    torch.cuda.synchronize()
    Vh = V.float().cpu().numpy()
    rows_ref, dV_ref, dw_ref = B.gather_backward(lambda r: Vh[r], idx, w, dp, perm, Np, expand)
    order = np.argsort(rows_ref)
    n = int(n_rows.item())
    assert n == len(rows_ref)
    got_rows = rows.cpu().numpy()
    assert np.array_equal(got_rows[:n], np.asarray(rows_ref)[order])
    assert (got_rows[n:] == -1).all()
    assert torch.equal(d_rows[:n], dV[rows[:n].long()])
    assert torch.isnan(d_rows[n:]).all()
    assert torch.equal(dw, dw_dense)
    e_dv = rel(d_rows[:n].cpu().numpy(), np.asarray(dV_ref)[order])
    log(f"[report] gather backward rows dv={dv} E={expand} cores={cores}: {n} rows, dV err {e_dv:.2e}")
    assert e_dv <= RTOL


def test_gather_backward_rows_tucker_ive():
    """The compact form at the 4M-slot Tucker + IVE layer's 4096-token batch (clustered queries:
    runs of hundreds of entries spanning many segments), against the dense form bit for bit."""
    cfg = CF.C5
    dl = SD.make_layer(cfg)
    idx, w, _ = G.score_topk(dl, cfg.T, 0)
    rng = np.random.default_rng(6)
    dp = torch.from_numpy(rng.standard_normal((cfg.T, cfg.expand, cfg.dv)).astype(np.float32)).cuda()
    idx2, w2 = idx.reshape(cfg.T, cfg.bag), w.reshape(cfg.T, cfg.bag)
    dV = torch.zeros((cfg.n_values, cfg.dv), dtype=torch.float32, device="cuda")
    dw_dense = run_gather_backward(cfg.n_values, cfg.dv, cfg.vdtype, dl.values, cfg.T, cfg.bag, idx2,
                                   w2, dl.perm, cfg.expand, 1, dp, dV)
    rows, d_rows, n_rows, dw = run_gather_backward_rows(cfg.n_values, cfg.dv, cfg.vdtype, dl.values,
                                                        cfg.T, cfg.bag, idx2, w2, dl.perm, cfg.expand,
                                                        1, dp)
    torch.cuda.synchronize()
    n = int(n_rows.item())
    idx_h = G.host(idx2).astype(np.int64)
    _, row = O.address_map(idx_h, CF.perm(cfg), cfg.n_values, cfg.expand)
    uniq = np.unique(row)
    log(f"[report] gather backward rows tucker-ive-4M: {n} distinct rows of {row.size} entries")
    assert n == len(uniq)
    assert np.array_equal(rows[:n].cpu().numpy(), uniq)
    assert torch.equal(d_rows[:n], dV[rows[:n].long()])
    assert torch.equal(dw, dw_dense)


def test_gather_backward_deterministic():
    cfg = CF.C5.with_tokens(512)
    dl = SD.make_layer(cfg)
    idx, w, _ = G.score_topk(dl, cfg.T, 0)
    dp = torch.randn((cfg.T, cfg.expand, cfg.dv), dtype=torch.float32, device="cuda")
    outs = []
    for _ in range(2):
        dV = torch.zeros((cfg.n_values, cfg.dv), dtype=torch.float32, device="cuda")
        dw = run_gather_backward(cfg.n_values, cfg.dv, cfg.vdtype, dl.values, cfg.T, cfg.bag,
                                 idx.reshape(cfg.T, cfg.bag), w.reshape(cfg.T, cfg.bag), dl.perm,
                                 cfg.expand, 1, dp, dV)
        torch.cuda.synchronize()
        outs.append((dV, dw))
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])


def test_gather_backward_tucker_ive_sampled():
    """The 4M-slot Tucker + IVE layer's 4096-token batch (clustered queries: rows shared by many
    tokens), on sampled rows: the oracle gets exactly the entries on those rows."""
    cfg = CF.C5
    dl = SD.make_layer(cfg)
    idx, w, _ = G.score_topk(dl, cfg.T, 0)
    rng = np.random.default_rng(5)
    dp = torch.from_numpy(rng.standard_normal((cfg.T, cfg.expand, cfg.dv)).astype(np.float32)).cuda()
    dV = torch.zeros((cfg.n_values, cfg.dv), dtype=torch.float32, device="cuda")
    idx2, w2 = idx.reshape(cfg.T, cfg.bag), w.reshape(cfg.T, cfg.bag)
    dw = run_gather_backward(cfg.n_values, cfg.dv, cfg.vdtype, dl.values, cfg.T, cfg.bag, idx2, w2,
                             dl.perm, cfg.expand, 1, dp, dV)
    torch.cuda.synchronize()
    idx_h, w_h, dp_h = G.host(idx2).astype(np.int64), G.host(w2), dp.cpu().numpy()
    perm = CF.perm(cfg)
    _, row = O.address_map(idx_h, perm, cfg.n_values, cfg.expand)
    sample = np.unique(row)[rng.choice(len(np.unique(row)), 24, replace=False)]
    sel = np.argwhere(np.isin(row, sample))                  # (t, b) entries on sampled rows, in order
    sub_idx = idx_h[sel[:, 0], sel[:, 1]][:, None]
    sub_w = w_h[sel[:, 0], sel[:, 1]][:, None]
    sub_dp = dp_h[sel[:, 0]]
    vrows = G.value_rows_fn(cfg)
    rows, dV_ref, dw_ref = B.gather_backward(vrows, sub_idx, sub_w, sub_dp, perm, cfg.n_values, cfg.expand)
    e_dv = rel(dV[torch.from_numpy(rows).cuda()].cpu().numpy(), dV_ref)
    e_dw = rel(G.host(dw)[sel[:, 0], sel[:, 1]], dw_ref[:, 0])
    log(f"[report] tucker-ive-4M gather backward: {len(sel)} entries on 24 sampled rows, "
        f"dV err {e_dv:.2e}, dw err {e_dw:.2e}")
    assert e_dv <= RTOL and e_dw <= RTOL


# ---------------------------------------------------------------- score backward

SCORE_CASES = [
    CF.Layer("add-raw", T=24, heads=2, dk=64, n_keys=80, topk=12, topm=20, dv=8, vdtype=CF.F32, seed=51),
    CF.Layer("add-softmax", T=16, heads=1, dk=32, n_keys=50, topk=8, topm=16, dv=8, vdtype=CF.F32,
             seed=52, weight=CF.W_SOFTMAX),
    CF.Layer("tucker", T=20, heads=3, dk=64, n_keys=70, topk=10, topm=24, dv=8, vdtype=CF.F32, seed=53,
             rank=2, grid=CF.GRID_TUCKER),
    CF.Layer("tucker-mcs", T=18, heads=2, dk=128, n_keys=64, topk=16, topm=32, dv=8, vdtype=CF.F32,
             seed=54, rank=2, grid=CF.GRID_TUCKER, cores=2),
    # more than 64 slots per (token, head): two and four slots per lane; one slot
    CF.Layer("tucker-m100", T=40, heads=2, dk=64, n_keys=96, topk=16, topm=100, dv=8, vdtype=CF.F32,
             seed=56, rank=2, grid=CF.GRID_TUCKER),
    CF.Layer("add-softmax-m200", T=12, heads=1, dk=32, n_keys=120, topk=20, topm=200, dv=8,
             vdtype=CF.F32, seed=57, weight=CF.W_SOFTMAX),
    CF.Layer("tucker-mcs-m256", T=10, heads=2, dk=64, n_keys=64, topk=16, topm=256, dv=8,
             vdtype=CF.F32, seed=58, rank=2, grid=CF.GRID_TUCKER, cores=2),
    CF.Layer("add-m1", T=9, heads=3, dk=16, n_keys=30, topk=2, topm=1, dv=8, vdtype=CF.F32, seed=59),
    CF.Layer("tucker-r4-wide", T=256, heads=2, dk=128, n_keys=512, topk=32, topm=64, dv=8,
             vdtype=CF.F32, seed=55, rank=4, grid=CF.GRID_TUCKER),
    # the per-slice recompute's other lane splits: four lanes on one slice; rank 3 (one idle lane,
    # 7-piece slices)
    CF.Layer("tucker-r1", T=14, heads=2, dk=64, n_keys=60, topk=12, topm=30, dv=8, vdtype=CF.F32,
             seed=60, rank=1, grid=CF.GRID_TUCKER),
    CF.Layer("tucker-r3", T=11, heads=1, dk=84, n_keys=70, topk=14, topm=40, dv=8, vdtype=CF.F32,
             seed=61, rank=3, grid=CF.GRID_TUCKER),
    # the library's limits: n = 8192, Dk = 1024, k = 90, m = 256; 64 heads
    CF.Layer("add-limits", T=3, heads=1, dk=1024, n_keys=8192, topk=90, topm=256, dv=8,
             vdtype=CF.F32, seed=62),
    CF.Layer("tucker-h64", T=3, heads=64, dk=64, n_keys=128, topk=16, topm=32, dv=8, vdtype=CF.F32,
             seed=63, rank=2, grid=CF.GRID_TUCKER),
    # key rows of 4 and 8 dims (64 and 32 key entries per wave in the key gradients and dq), and
    # the paper's Kdim 448 (dq in passes of 256 dims)
    CF.Layer("add-dk4", T=30, heads=2, dk=4, n_keys=40, topk=6, topm=10, dv=8, vdtype=CF.F32, seed=64),
    CF.Layer("tucker-dk8", T=25, heads=2, dk=8, n_keys=48, topk=8, topm=16, dv=8, vdtype=CF.F32,
             seed=65, rank=2, grid=CF.GRID_TUCKER),
    CF.Layer("tucker-dk448", T=12, heads=2, dk=448, n_keys=96, topk=14, topm=42, dv=8,
             vdtype=CF.F32, seed=66, rank=2, grid=CF.GRID_TUCKER, cores=2),
]


SCORE_CASE = {c.name: c for c in SCORE_CASES}


def run_score_backward(cfg, dl, idx, w, dw, dk_init=None, dc_init=None, dq_offset=0):
    """dq_offset: floats by which dq_row and dq_col start past a 256-byte boundary (the API asks
    4-byte alignment of them only)."""
    d = G.desc_for(cfg)
    st, nws = U.umem_score_backward_workspace_size(d, cfg.T)
    U.check(st)
    ws = torch.empty(max(nws, 256), dtype=torch.uint8, device="cuda")
    nq = dl.q_row[0].numel()
    dq_row = torch.empty(nq + dq_offset, dtype=torch.float32, device="cuda")[dq_offset:].view_as(dl.q_row[0])
    dq_col = torch.empty(nq + dq_offset, dtype=torch.float32, device="cuda")[dq_offset:].view_as(dl.q_col[0])
    dk_row = torch.zeros_like(dl.k_row) if dk_init is None else dk_init[0].clone()
    dk_col = torch.zeros_like(dl.k_col) if dk_init is None else dk_init[1].clone()
    dcore = None
    if cfg.grid == CF.GRID_TUCKER:
        dcore = torch.zeros_like(dl.core) if dc_init is None else dc_init.clone()
    U.check(U.umem_score_backward(d, cfg.T, dl.q_row[0], dl.q_col[0], dl.k_row, dl.k_col, dl.core,
                                  idx, w, dw, dq_row, dq_col, dk_row, dk_col, dcore, ws, ws.numel()),
            "umem_score_backward")
    return dq_row, dq_col, dk_row, dk_col, dcore


@pytest.mark.parametrize("cfg", SCORE_CASES, ids=[c.name for c in SCORE_CASES])
def test_score_backward(cfg):
    log(f"[case] score backward {cfg.name}")
    dl = SD.make_layer(cfg)
    idx, w, _ = G.score_topk(dl, cfg.T, 0)
    rng = np.random.default_rng(cfg.seed)
    dw_h = rng.standard_normal(tuple(w.shape)).astype(np.float32)
    dk0 = (torch.randn_like(dl.k_row), torch.randn_like(dl.k_col))
    dc0 = None if dl.core is None else torch.randn_like(dl.core)
    dq_row, dq_col, dk_row, dk_col, dcore = run_score_backward(
        cfg, dl, idx, w, torch.from_numpy(dw_h).cuda(), dk0, dc0)
    torch.cuda.synchronize()
    qr, qc = CF.queries(cfg)
    kr, kc = CF.keys(cfg)
    core = CF.core(cfg)
    res = B.score_backward(qr, qc, kr, kc, G.host(idx), dw_h, G.host(w), cfg.grid, cfg.weight,
                           None if cfg.cores > 1 else core, cfg.rank,
                           core if cfg.cores > 1 else None)
    errs = dict(dq_row=rel(G.host(dq_row), res["dq_row"]), dq_col=rel(G.host(dq_col), res["dq_col"]),
                dk_row=rel(G.host(dk_row) - G.host(dk0[0]), res["dK_row"]),
                dk_col=rel(G.host(dk_col) - G.host(dk0[1]), res["dK_col"]))
    if dcore is not None:
        errs["dcore"] = rel(G.host(dcore) - G.host(dc0), res["dC"])
    log(f"[report] score backward {cfg.name}: {errs}")
    assert max(errs.values()) <= RTOL, errs


@pytest.mark.parametrize("offset", [1, 2])
def test_score_backward_dq_unaligned(offset):
    """dq rows that are 4-byte but not 16-byte aligned take the one-dim-per-lane form of dq: the
    same result, to the tolerance, as the 16-byte form on aligned rows."""
    cfg = SCORE_CASE["tucker"]                                     # Tucker, Dk = 64
    dl = SD.make_layer(cfg)
    idx, w, _ = G.score_topk(dl, cfg.T, 0)
    rng = np.random.default_rng(7)
    dw = torch.from_numpy(rng.standard_normal(tuple(w.shape)).astype(np.float32)).cuda()
    a = run_score_backward(cfg, dl, idx, w, dw)
    b = run_score_backward(cfg, dl, idx, w, dw, dq_offset=offset)
    torch.cuda.synchronize()
    assert b[0].data_ptr() % 16 != 0
    for x, y in zip(a[:4], b[:4]):
        assert rel(G.host(y), G.host(x)) <= RTOL
    assert torch.equal(a[2], b[2]) and torch.equal(a[3], b[3])      # dK does not involve dq


def test_score_backward_deterministic():
    cfg = SCORE_CASE["tucker-h64"]
    dl = SD.make_layer(cfg)
    idx, w, _ = G.score_topk(dl, cfg.T, 0)
    dw = torch.randn_like(w)
    a = run_score_backward(cfg, dl, idx, w, dw)
    b = run_score_backward(cfg, dl, idx, w, dw)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x, y)


def test_backward_graph_replay_matches_eager():
    """Both backward entry points captured in a HIP graph (with the clearing of their accumulated
    outputs by fill kernels), replayed several times with eager work in between, give the eager
    results bit for bit: their piece counters and lists are rebuilt by kernels on every call."""
    cfg = SCORE_CASE["tucker-h64"]        # Tucker r = 2, 64 heads, rows shared by many tokens
    dl = SD.make_layer(cfg)
    idx, w, _ = G.score_topk(dl, cfg.T, 0)
    torch.cuda.synchronize()
    T, bag = cfg.T, cfg.heads * cfg.topm
    desc = G.desc_for(cfg)
    dp = torch.randn((T, cfg.expand, cfg.dv), dtype=torch.float32, device="cuda")
    dwin = torch.randn_like(w)
    st, n1 = U.umem_gather_backward_workspace_size(T, bag, cfg.dv)
    U.check(st)
    st, n2 = U.umem_score_backward_workspace_size(desc, T)
    U.check(st)
    ws1 = torch.empty(max(n1, 256), dtype=torch.uint8, device="cuda")
    ws2 = torch.empty(max(n2, 256), dtype=torch.uint8, device="cuda")
    dV = torch.empty((cfg.n_values, cfg.dv), dtype=torch.float32, device="cuda")
    dw = torch.empty((T, bag), dtype=torch.float32, device="cuda")
    dq_r, dq_c = torch.empty_like(dl.q_row[0]), torch.empty_like(dl.q_col[0])
    dk_r, dk_c = torch.empty_like(dl.k_row), torch.empty_like(dl.k_col)
    dc = torch.empty_like(dl.core)
    outs = (dV, dw, dq_r, dq_c, dk_r, dk_c, dc)

    def step():
        for t in (dV, dk_r, dk_c, dc):          # accumulated outputs start from zero
            t.zero_()
        U.check(U.umem_gather_backward(cfg.n_values, cfg.dv, cfg.vdtype, dl.values, T, bag,
                                       idx.reshape(T, bag), w.reshape(T, bag), dl.perm, cfg.expand,
                                       cfg.cores, dp, dV, dw, ws1, ws1.numel()), "umem_gather_backward")
        U.check(U.umem_score_backward(desc, T, dl.q_row[0], dl.q_col[0], dl.k_row, dl.k_col, dl.core,
                                      idx, w, dwin, dq_r, dq_c, dk_r, dk_c, dc, ws2, ws2.numel()),
                "umem_score_backward")

    step()
    torch.cuda.synchronize()
    want = [t.clone() for t in outs]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for rep in range(4):
        for t in outs:
            t.fill_(-1.0)
        ws1.fill_(0xAB)                      # stale counters and lists from any earlier call
        ws2.fill_(0xCD)
        g.replay()
        torch.cuda.synchronize()
        for got, ref in zip(outs, want):
            assert torch.equal(got, ref), rep
        step()                               # eager work between replays
        torch.cuda.synchronize()
