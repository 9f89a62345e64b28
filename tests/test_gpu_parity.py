"""GPU parity: the HIP path through the C ABI against the oracle, on the same seeded inputs."""
from __future__ import annotations

import dataclasses
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():     # collected on CPU hosts too; every test here is gpu-marked
    pytest.skip("no GPU", allow_module_level=True)

import oracle.umem_oracle as O                      # noqa: E402
import paper_2411_12364_amd as U                    # noqa: E402
import synth as S                                   # noqa: E402
from synth import configs as CF                     # noqa: E402
from synth import device as SD                      # noqa: E402
from tests import gpu_util as G                     # noqa: E402
from tests import parity as P                       # noqa: E402


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def small(name, **kw):
    base = dict(T=8, heads=1, dk=64, n_keys=64, topk=8, topm=8, dv=256, vdtype=CF.F32, seed=11)
    base.update(kw)
    return CF.Layer(name, **base)


# The GPU's fp32 first GEMM and the oracle's fp64 one round a few of the intermediate values to
# bf16 differently (a value within its fp32 error of a rounding boundary: about one in 400 at
# K = 2048); each such value moves by one bf16 step, 2^-8 of itself.  Measured at most 9.8e-4
# of a row (the two-core Tucker + IVE layer), against 2e-2 for the plain oracle.
PROJ_ROUNDED_RTOL = 4e-3


def _round_bf16(a):
    a = np.asarray(a, np.float32)
    return S.bf16_bits_to_f32(S.f32_to_bf16_bits(a)).reshape(a.shape).astype(np.float64)


def projection_of_rounded(pooled, wp, wo):
    """eq. (15) and the output linear on the oracle's pooled rows [T, E, Dv], with each GEMM's
    A operand rounded to bf16 as the GPU's GEMM takes it (bf16 weights as given)."""
    Wp = None if wp is None else S.bf16_bits_to_f32(wp).reshape(wp.shape).astype(np.float64)
    Wo = None if wo is None else S.bf16_bits_to_f32(wo).reshape(wo.shape).astype(np.float64)
    y = O.ive_project(_round_bf16(pooled), Wp, None)      # without W_p: the rounded rows
    if Wo is None:
        return y
    return (_round_bf16(y) if Wp is not None else y) @ Wo


def run_and_check(cfg, batch=0, tokens=None, gap=P.GAP, expect_no_exempt=False, dl=None):
    """Full staged check of one configuration; ``tokens`` samples the tokens the oracle checks."""
    log(f"[case] {cfg.name} T={cfg.T} H={cfg.heads} n={cfg.n_keys} k={cfg.topk} m={cfg.topm} "
        f"dv={cfg.dv} E={cfg.expand} grid={cfg.grid}")
    dl = dl or SD.make_layer(cfg, batches=batch + 1)
    T = cfg.T
    idx, w, ax = G.score_topk(dl, T, batch)
    pooled = G.gather(dl, idx, w, T)
    out_f, idx_f, w_f = G.forward(dl, T, batch)
    torch.cuda.synchronize()
    idx_h, w_h, ax_h = G.host(idx), G.host(w), G.host(ax)
    # umem_forward runs the same kernels: identical bits
    assert np.array_equal(G.host(idx_f), idx_h) and np.array_equal(G.host(w_f), w_h)
    t_sel = np.arange(T) if tokens is None else np.asarray(tokens)
    qr, qc = CF.queries(cfg, batch=batch, tokens=t_sel)
    kr, kc = CF.keys(cfg)
    core = CF.core(cfg)
    _, rep = P.check_selection(cfg, qr, qc, kr, kc, core, idx_h[t_sel], w_h[t_sel], ax_h[:, t_sel],
                               gap=gap)
    perm = CF.perm(cfg)
    ref_pooled, err = P.check_pooled(cfg, G.value_rows_fn(cfg), idx_h[t_sel], w_h[t_sel],
                                     G.host(pooled)[t_sel], perm)
    rep["pooled_err"] = err
    if cfg.dv_virt or cfg.d_out:
        wp, wo = CF.projections(cfg)
        y_ref = O.ive_project(ref_pooled, None if wp is None else S.bf16_bits_to_f32(wp).reshape(wp.shape),
                              None if wo is None else S.bf16_bits_to_f32(wo).reshape(wo.shape))
        got = G.host(out_f)[t_sel].astype(np.float64)
        perr = np.abs(got - y_ref).max(axis=1) / np.abs(y_ref).max(axis=1)
        rep["proj_err"] = float(perr.max())
        assert perr.max() <= 2e-2, ("projection", perr.max())
        # the GEMMs' documented operand roundings (the pooled rows, and the projection's output
        # before the output linear, to bf16 nearest even from fp32) applied to the oracle's own
        # values: what is left is fp32 accumulation and a rare rounding decided the other way
        y16 = projection_of_rounded(ref_pooled, wp, wo)
        perr16 = np.abs(got - y16).max(axis=1) / np.abs(y16).max(axis=1)
        rep["proj_err_rounded"] = float(perr16.max())
        assert perr16.max() <= PROJ_ROUNDED_RTOL, ("projection of rounded operands", perr16.max())
    else:
        # the forward may pool inside the selection kernel (another summation order): both it
        # and the standalone gather are held to the oracle
        fwd = G.host(out_f).reshape(G.host(pooled).shape)[t_sel].astype(np.float64)
        den = np.abs(ref_pooled).reshape(len(t_sel), -1).max(axis=1) + 1e-30
        ferr = (np.abs(fwd - ref_pooled).reshape(len(t_sel), -1).max(axis=1) / den).max()
        rep["forward_pooled_err"] = float(ferr)
        assert ferr <= 1e-5, ("forward pooled", ferr)
    log(f"[report] {cfg.name}: {rep}")
    if expect_no_exempt:
        assert rep["axis_exempt"] == 0 and rep["grid_exempt"] == 0 and rep["e2e_slot_mismatch"] == 0
    return rep


# ---------------------------------------------------------------- generator twin

@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_device_generator_matches_host(dtype):
    rows, width = 1003, 72
    t = torch.empty((rows, width), dtype=torch.float32 if dtype == "f32" else torch.bfloat16, device="cuda")
    SD.fill_normal_(t, 5, S.TID_VALUES, 0.125, chunk=4096 * 7 + 8)
    torch.cuda.synchronize()
    pick = np.array([0, 1, 500, 999, 1002])
    want = S.rows_f32(5, S.TID_VALUES, pick, width, 0.125)
    if dtype == "f32":
        got = t.cpu().numpy()[pick]
        assert np.array_equal(got.view(np.uint32), want.view(np.uint32))
    else:
        got = t.view(torch.int16).cpu().numpy()[pick].view(np.uint16)
        assert np.array_equal(got, S.f32_to_bf16_bits(want).reshape(got.shape))


# ---------------------------------------------------------------- small shapes, every token

def test_c1_tiny_pkm():
    rep = run_and_check(CF.C1)
    assert rep["pooled_err"] <= 1e-5


def test_c1_softmax():
    run_and_check(dataclasses.replace(CF.C1, weight=CF.W_SOFTMAX, name="tiny-softmax"))


def test_tiles_and_ragged_tails():
    # 3 token tiles (ragged), 4 key tiles (ragged), 3 heads, bag not a multiple of 64
    run_and_check(small("ragged", T=70, heads=3, n_keys=200, topk=16, topm=24, dv=256,
                        vdtype=CF.BF16, seed=12))


@pytest.mark.parametrize("kw", [
    dict(T=1, n_keys=1, topk=1, topm=1, dk=4),
    dict(T=5, n_keys=7, topk=7, topm=49, dk=8),             # k = n, m = k^2: the whole grid
    dict(T=3, n_keys=33, topk=1, topm=1),                   # argmax only
    dict(T=9, n_keys=130, topk=20, topm=3, heads=2, dk=12),
    dict(T=33, n_keys=64, topk=8, topm=8, dv=64, vdtype=CF.BF16),   # 128-byte rows
    dict(T=4, n_keys=64, topk=8, topm=8, dv=8, vdtype=CF.BF16),     # 16-byte rows
], ids=["n1", "whole-grid", "argmax", "odd-sizes", "row128B", "row16B"])
def test_edge_shapes(kw):
    run_and_check(small("edge", **kw))


# The library's own limits (`umem_internal.h`), each at its maximum in one case: n = 8192 keys per
# axis, k = 90 and m = 256 (additive); Dk = 1024 with the Tucker rank 4 (the query rows fill
# the 512 threads); a bag of 2048 rows of 8 KiB; the Tucker k = 64 with E = 64 and h = 8 cores.
# With k > 64 the additive grid's candidate table is built in two passes of a wave; the k = 70
# case runs that over 16 (token, head) pairs.
@pytest.mark.parametrize("kw", [
    dict(T=3, heads=1, dk=64, n_keys=8192, topk=90, topm=256, dv=8, vdtype=CF.BF16),
    dict(T=8, heads=2, dk=64, n_keys=2048, topk=70, topm=256, dv=8, vdtype=CF.BF16),
    dict(T=5, heads=2, dk=1024, n_keys=300, rank=4, grid=CF.GRID_TUCKER, topk=16, topm=64,
         dv=256, vdtype=CF.F32),
    dict(T=4, heads=8, dk=64, n_keys=256, topk=32, topm=256, dv=4096, vdtype=CF.BF16),
    dict(T=5, heads=2, dk=256, n_keys=512, rank=4, grid=CF.GRID_TUCKER, topk=64, topm=256, dv=64,
         vdtype=CF.BF16, expand=64, dv_virt=64, cores=8),
    # 64 heads (one factor pair each), the Tucker grid
    dict(T=3, heads=64, dk=64, n_keys=128, rank=2, grid=CF.GRID_TUCKER, topk=16, topm=32, dv=64,
         vdtype=CF.BF16),
    # the selection pooling the rows itself at its limits: 128 tokens, m = 64, rows of 2 KiB
    dict(T=128, heads=2, dk=128, n_keys=256, topk=32, topm=64, dv=1024, vdtype=CF.BF16),
    # n not a multiple of 4 at the largest per-thread share: 32 keys per thread and axis
    dict(T=2, heads=1, dk=64, n_keys=8191, topk=32, topm=32, dv=8, vdtype=CF.BF16),
], ids=["n-8192-k-90-m-256", "k-70-m-256", "dk-1024-rank-4", "bag-2048-rows-8KiB",
        "tucker-k-64-E-64-h-8", "heads-64", "pooled-T-128-m-64-2KiB", "n-8191"])
def test_library_limits(kw):
    cfg = small("limit", **kw)
    run_and_check(cfg, tokens=None if cfg.T <= 64 else np.arange(0, cfg.T, 7))


# The Tucker grid's exact per-slice scores (eq. (4)) split each key row over G = 16, 8 or 4 lanes
# (by 2k) and those over the slices (G, G/2 or G/4 lanes per slice for rank 1, 2, 3-4); these
# cases take every split, the idle lanes of rank 3, a slice of 7 pieces over 2 lanes, and rows
# of 112 pieces that need four batches of loads.
@pytest.mark.parametrize("kw", [
    dict(T=6, heads=2, dk=64, n_keys=120, rank=1, topk=12, topm=20),
    dict(T=5, heads=1, dk=84, n_keys=90, rank=3, topk=30, topm=40),
    dict(T=4, heads=2, dk=128, n_keys=100, rank=4, topk=50, topm=64),
    dict(T=3, heads=1, dk=448, n_keys=80, rank=2, topk=64, topm=64),
], ids=["rank1-G16", "rank3-G8", "rank4-G4", "dk448-G4"])
def test_tucker_exact_slice_splits(kw):
    run_and_check(small("tucker-slices", grid=CF.GRID_TUCKER, seed=17, **kw))


def _tie_layer(cfg):
    """Integer-valued queries and keys (0, +-1, +-2): many exact ties in fp32 and fp64 alike."""
    dl = SD.make_layer(cfg)
    q = [np.round(CF.queries(cfg)[a] * 8).clip(-2, 2).astype(np.float32) for a in (0, 1)]
    kr, kc = [np.round(k * 8).clip(-2, 2).astype(np.float32) for k in CF.keys(cfg)]
    dl.q_row = torch.from_numpy(q[0][None]).cuda()
    dl.q_col = torch.from_numpy(q[1][None]).cuda()
    dl.k_row, dl.k_col = torch.from_numpy(kr).cuda(), torch.from_numpy(kc).cuda()
    return dl, q, kr, kc


@pytest.mark.parametrize("kw", [dict(T=16, n_keys=300, topk=24, topm=40, heads=2, dk=8),
                                dict(T=8, n_keys=64, topk=8, topm=8, dk=4)], ids=["wide", "narrow"])
def test_exact_ties_lower_index(kw):
    cfg = small("ties", **kw)
    dl, q, kr, kc = _tie_layer(cfg)
    idx, w, ax = G.score_topk(dl, cfg.T)
    torch.cuda.synchronize()
    _, rep = P.check_selection(cfg, q[0], q[1], kr, kc, None, G.host(idx), G.host(w), G.host(ax),
                               gap=0.0)
    log(f"[report] ties: {rep}")
    assert rep["e2e_slot_mismatch"] == 0


# ---------------------------------------------------------------- a1 + a2 alone, every kernel

@pytest.mark.parametrize("kw", [
    # 16 < T <= 64: 32 x 32 tiles, eight waves splitting Dk (Dk / 64 loads per lane and operand)
    dict(T=40, heads=2, dk=128, n_keys=200),                                  # wide, 2 token tiles
    dict(T=40, heads=2, dk=128, n_keys=200, rank=2, grid=CF.GRID_TUCKER),     # wide + fold
    dict(T=64, heads=1, dk=256, n_keys=33),                                   # wide, dk = 256
    dict(T=33, heads=2, dk=64, n_keys=100),                                   # wide, dk = 64
    dict(T=50, heads=1, dk=128, n_keys=96, rank=4, grid=CF.GRID_TUCKER),      # wide + rank-4 fold
    # T <= 16: 16 x 16 tiles, four waves splitting Dk
    dict(T=9, heads=1, dk=64, n_keys=70, rank=4, grid=CF.GRID_TUCKER),        # split, 1 chunk
    dict(T=12, heads=2, dk=128, n_keys=150, rank=2, grid=CF.GRID_TUCKER),     # split, 2 chunks
    dict(T=100, heads=1, dk=256, n_keys=130, rank=2, grid=CF.GRID_TUCKER),    # tiled MFMA
    dict(T=70, heads=3, dk=64, n_keys=200),                                   # tiled MFMA
    dict(T=5, heads=2, dk=12, n_keys=33, rank=3, grid=CF.GRID_TUCKER),        # vector ALU
    # many tokens on fp16 planes: ragged token and key tiles, three dk steps; dk = 448
    dict(T=200, heads=3, dk=96, n_keys=300, rank=2, grid=CF.GRID_TUCKER),
    dict(T=130, heads=1, dk=448, n_keys=260),
], ids=["wide", "wide-tucker2", "wide-dk256", "wide-dk64", "wide-tucker4", "split-tucker4",
        "split-tucker2", "tiled-tucker2", "tiled", "valu-tucker3", "planes-tucker2", "planes-dk448"])
def test_axis_scores_kernels(kw):
    cfg = small("scores", topk=4, topm=4, **kw)
    log(f"[case] axis scores {kw}")
    dl = SD.make_layer(cfg)
    desc = G.desc_for(cfg)
    T, H, n = cfg.T, cfg.heads, cfg.n_keys
    sel = torch.empty((2, T, H, n), dtype=torch.float32, device="cuda")
    ws = G.workspace(desc, T)
    U.check(U.umem_axis_scores(desc, T, dl.q_row[0], dl.q_col[0], dl.k_row, dl.k_col, dl.core, sel,
                               ws, ws.numel()), "umem_axis_scores")
    torch.cuda.synchronize()
    got = G.host(sel).astype(np.float64)
    qr, qc = CF.queries(cfg)
    kr, kc = CF.keys(cfg)
    core = CF.core(cfg)
    vr = vc = None
    if core is not None:
        f = [O.rank1_factors(core[h].astype(np.float64)) for h in range(H)]
        vr, vc = [x[0] for x in f], [x[1] for x in f]
    for a, (q, K, v) in enumerate(((qr, kr, vr), (qc, kc, vc))):
        want = O.selection_scores(O.axis_scores(q, K, cfg.rank), v)
        # fp32 products and sums against fp64: bound by the size of the terms
        scale = np.einsum("thd,hnd->thn", np.abs(q.astype(np.float64)), np.abs(K.astype(np.float64)))
        err = np.abs(got[a] - want) / (scale + 1e-30)
        log(f"[report] axis {a}: max err / sum|q k| = {err.max():.2e}")
        assert err.max() <= 1e-5, (a, err.max())


def _special_cores(rank, rng):
    """Cores whose leading singular pair the fp64 Jacobi sweeps must find in edge conditions: a
    diagonal core (nothing to rotate), a zero column (rank-deficient), leading singular values
    1e-3 apart, scales of 1e-20 and 1e18, and all entries negative."""
    r = rank
    cores = [np.diag(np.arange(r, 0, -1)).astype(np.float32)]
    z = rng.standard_normal((r, r)).astype(np.float32)
    z[:, -1] = 0.0
    cores.append(z)
    u_, _ = np.linalg.qr(rng.standard_normal((r, r)))
    v_, _ = np.linalg.qr(rng.standard_normal((r, r)))
    s = np.linspace(1.0, 0.4, r)
    s[1] = 1.0 - 1e-3
    cores.append((u_ @ np.diag(s) @ v_.T).astype(np.float32))
    cores.append(rng.standard_normal((r, r)).astype(np.float32) * np.float32(1e-20))
    cores.append(rng.standard_normal((r, r)).astype(np.float32) * np.float32(1e18))
    cores.append(-np.abs(rng.standard_normal((r, r))).astype(np.float32))
    return np.stack(cores)


@pytest.mark.parametrize("T,rank,dk", [(12, 2, 128), (12, 4, 64), (130, 2, 96), (40, 2, 128)],
                         ids=["split-r2", "split-r4", "planes-r2", "wide-r2"])
def test_rank1_fold_special_cores(T, rank, dk):
    """The rank-1 factors of the Tucker core (eqs. (8)-(10)) folded into the axis scores, for the
    cores of _special_cores (one per head), against the oracle's factors."""
    cores = _special_cores(rank, np.random.default_rng(31 + rank))
    H = cores.shape[0]
    cfg = small("rank1", T=T, heads=H, dk=dk, n_keys=100, topk=4, topm=4, rank=rank,
                grid=CF.GRID_TUCKER)
    log(f"[case] rank-1 fold T={T} rank={rank} dk={dk}")
    dl = SD.make_layer(cfg)
    dl.core = torch.from_numpy(cores).cuda()
    desc = G.desc_for(cfg)
    n = cfg.n_keys
    sel = torch.empty((2, T, H, n), dtype=torch.float32, device="cuda")
    ws = G.workspace(desc, T)
    U.check(U.umem_axis_scores(desc, T, dl.q_row[0], dl.q_col[0], dl.k_row, dl.k_col, dl.core, sel,
                               ws, ws.numel()), "umem_axis_scores")
    torch.cuda.synchronize()
    got = G.host(sel).astype(np.float64)
    qr, qc = CF.queries(cfg)
    kr, kc = CF.keys(cfg)
    f = [O.rank1_factors(cores[h].astype(np.float64)) for h in range(H)]
    for a, (q, K, v) in enumerate(((qr, kr, [x[0] for x in f]), (qc, kc, [x[1] for x in f]))):
        want = O.selection_scores(O.axis_scores(q, K, rank), v)
        scale = np.einsum("thd,hnd->thn", np.abs(q.astype(np.float64)), np.abs(K.astype(np.float64)))
        err = np.abs(got[a] - want) / (scale + 1e-30)
        log(f"[report] axis {a}: max err / sum|q k| = {err.max():.2e}")
        assert err.max() <= 1e-5, (a, err.max())


def test_planes_row_exponents():
    """The fp16-plane scoring scales every query and key row by its own power of two before the
    split: rows scaled by 2^-40 .. 2^40, a zero row, a row with one nonzero element and a row whose
    elements span 2^-40 .. 1 all keep their scores within 1e-6 of sum |q_d k_d| of the fp64
    value."""
    cfg = small("exps", T=130, heads=2, dk=64, n_keys=256, topk=4, topm=4, dv=8, vdtype=CF.BF16)
    desc = G.desc_for(cfg)
    T, H, n, dk = cfg.T, cfg.heads, cfg.n_keys, cfg.dk
    rng = np.random.default_rng(77)
    qr, qc = CF.queries(cfg)
    kr, kc = CF.keys(cfg)
    qr = qr * np.exp2(rng.integers(-40, 41, size=(T, H, 1))).astype(np.float32)
    kr = kr * np.exp2(rng.integers(-40, 41, size=(H, n, 1))).astype(np.float32)
    qr[0] = 0.0
    kr[:, 0] = 0.0
    qr[1] = 0.0
    qr[1, :, 5] = 1.0
    qr[2] = (rng.standard_normal((H, dk)) * np.exp2(-np.linspace(0, 40, dk))).astype(np.float32)
    kc[:, 3] = kc[:, 3] * np.float32(2.0 ** 40)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()
    sel = torch.empty((2, T, H, n), dtype=torch.float32, device="cuda")
    ws = G.workspace(desc, T)
    U.check(U.umem_axis_scores(desc, T, dev(qr), dev(qc), dev(kr), dev(kc), None, sel, ws,
                               ws.numel()), "umem_axis_scores")
    torch.cuda.synchronize()
    got = G.host(sel).astype(np.float64)
    for a, (q, K) in enumerate(((qr, kr), (qc, kc))):
        want = O.axis_scores(q, K, 1)[:, :, 0, :]
        scale = np.einsum("thd,hnd->thn", np.abs(q.astype(np.float64)), np.abs(K.astype(np.float64)))
        err = np.abs(got[a] - want) / (scale + 1e-300)
        log(f"[report] row exponents, axis {a}: max err / sum|q k| = {err.max():.2e}")
        assert err.max() <= 1e-6, (a, err.max())
        assert np.all(got[a][(scale == 0)] == 0.0)


# ---------------------------------------------------------------- multi-core scoring

@pytest.mark.parametrize("kw", [
    # pooled inside the selection (two heads, 1 KiB rows)
    dict(T=40, heads=2, dk=128, n_keys=150, rank=2, grid=CF.GRID_TUCKER, topk=16, topm=24,
         dv=512, vdtype=CF.BF16, cores=2),
    # the gather kernel (three heads), four cores, fp32 rows
    dict(T=20, heads=3, dk=64, n_keys=90, rank=2, grid=CF.GRID_TUCKER, topk=10, topm=30, dv=256,
         vdtype=CF.F32, cores=4),
    # with IVE and the projection: the physical rows are split
    dict(T=24, heads=2, dk=128, n_keys=128, rank=2, grid=CF.GRID_TUCKER, topk=16, topm=32,
         dv=512, vdtype=CF.BF16, expand=4, dv_virt=256, d_out=192, cores=2),
], ids=["pooled-in-select", "gather-4-cores", "ive-projection"])
def test_multi_core_scoring(kw):
    run_and_check(small("mcs", **kw))


def test_paper_model_layer_sampled():
    """One memory layer of the paper's UltraMem-1.6B-x12 model (Kdim 448, 1792^2 slots, top-42 of
    2 heads, r = 2, h = 2, E = 4, 8 KiB rows) at a 512-token decode batch: 256 of its tokens."""
    rng = np.random.default_rng(6)
    run_and_check(CF.C6, tokens=np.sort(rng.choice(CF.C6.T, 256, replace=False)))


def test_c5_tucker_ive_mcs_sampled():
    """The rank-2 Tucker + IVE layer with the paper's default two component cores: 256 tokens,
    the first and last among them."""
    cfg = dataclasses.replace(CF.C5, cores=2, name="tucker-ive-mcs-4M")
    rng = np.random.default_rng(55)
    tokens = np.union1d([0, 1, 2, 1023, 2048, 4095], rng.choice(cfg.T, 250, replace=False))
    run_and_check(cfg, tokens=tokens)


# ---------------------------------------------------------------- a7 inside the selection

@pytest.mark.parametrize("kw", [
    dict(T=37, heads=1, dk=64, n_keys=100, topk=8, topm=8, dv=256, vdtype=CF.F32),
    dict(T=37, heads=2, dk=128, n_keys=300, topk=16, topm=40, dv=1024, vdtype=CF.BF16),
    dict(T=20, heads=2, dk=128, n_keys=150, topk=12, topm=64, dv=512, vdtype=CF.BF16,
         weight=CF.W_SOFTMAX),
    dict(T=9, heads=2, dk=128, n_keys=90, rank=2, grid=CF.GRID_TUCKER, topk=10, topm=20, dv=512,
         vdtype=CF.BF16),
    dict(T=20, heads=2, dk=64, n_keys=128, topk=16, topm=32, dv=512, vdtype=CF.F32),
    # multi-core weights on 2 KiB rows: each lane's two chunks take their own slices' weights
    dict(T=24, heads=2, dk=128, n_keys=128, rank=2, grid=CF.GRID_TUCKER, topk=16, topm=48,
         dv=1024, vdtype=CF.BF16, cores=4),
], ids=["f32-1KiB", "bf16-2KiB-m40", "softmax-m64", "tucker", "f32-2KiB", "mcs4-2KiB"])
def test_select_pools_like_gather(kw):
    """umem_select with values/pooled: the same idx and w as without, and pooled rows that match
    the oracle's gather of them."""
    cfg = small("pool", **kw)
    log(f"[case] select pooling {kw}")
    dl = SD.make_layer(cfg)
    desc = G.desc_for(cfg)
    T, H, n, m = cfg.T, cfg.heads, cfg.n_keys, cfg.topm
    ws = G.workspace(desc, T)
    sel = torch.empty((2, T, H, n), dtype=torch.float32, device="cuda")
    U.check(U.umem_axis_scores(desc, T, dl.q_row[0], dl.q_col[0], dl.k_row, dl.k_col, dl.core, sel,
                               ws, ws.numel()), "umem_axis_scores")
    outs = []
    for pool in (False, True):
        idx = torch.empty((T, H, m), dtype=torch.int32, device="cuda")
        w = torch.empty(G.weights_shape(cfg, T), dtype=torch.float32, device="cuda")
        pooled = torch.zeros((T, cfg.dv), dtype=torch.float32, device="cuda")
        U.check(U.umem_select(desc, T, sel, dl.q_row[0], dl.q_col[0], dl.k_row, dl.k_col, dl.core,
                              idx, w, None, dl.values if pool else None, pooled if pool else None),
                "umem_select")
        outs.append((idx, w, pooled))
    torch.cuda.synchronize()
    (i0, w0, _), (i1, w1, p1) = outs
    assert torch.equal(i0, i1) and torch.equal(w0, w1)
    _, err = P.check_pooled(cfg, G.value_rows_fn(cfg), G.host(i0), G.host(w0),
                            G.host(p1)[:, None, :], None)
    log(f"[report] select pooling {kw}: err={err:.2e}")


# ---------------------------------------------------------------- gather and projection alone

@pytest.mark.parametrize("dv,vdtype,expand,bag,T,cores", [
    (512, CF.BF16, 1, 64, 37, 1), (1024, CF.BF16, 1, 77, 37, 1), (256, CF.F32, 1, 5, 37, 1),
    (512, CF.BF16, 4, 256, 37, 1), (128, CF.BF16, 9, 40, 37, 1), (3072, CF.BF16, 1, 33, 37, 1),
    (8, CF.BF16, 4, 130, 37, 1),
    # thousands of tokens: a wave per token (ragged last workgroup, sub-rows, long rows)
    (512, CF.BF16, 1, 64, 4099, 1), (64, CF.BF16, 1, 33, 4100, 1), (2048, CF.BF16, 1, 20, 4096, 1),
    (256, CF.F32, 1, 7, 5001, 1),
    # ... with rows of 16 and 32 bytes: 64 and 32 rows at once per wave
    (8, CF.BF16, 1, 70, 2100, 1), (16, CF.BF16, 1, 33, 2050, 1),
    # multi-core weights (eq. (17)): column slices, with IVE, sub-rows, many tokens
    (512, CF.BF16, 1, 64, 37, 2), (1024, CF.BF16, 4, 100, 37, 4), (64, CF.BF16, 1, 33, 70, 4),
    (256, CF.F32, 1, 33, 4099, 2), (3072, CF.BF16, 1, 20, 9, 8),
    # 8 KiB rows with IVE and two cores (the paper's 1.6B-x12 layer)
    (4096, CF.BF16, 4, 84, 37, 2),
    # whole virtual blocks per wave: four blocks each (E = 16), sixteen with sub-rows and two
    # cores (E = 64), and a bag of one entry (three empty blocks)
    (256, CF.F32, 16, 50, 37, 1), (64, CF.BF16, 64, 200, 37, 2), (512, CF.BF16, 4, 1, 37, 1)])
def test_gather_standalone(dv, vdtype, expand, bag, T, cores):
    rng = np.random.default_rng(dv + bag + T + cores)
    Np = 5000
    vdt = torch.float32 if vdtype == CF.F32 else torch.bfloat16
    values = torch.empty((Np, dv), dtype=vdt, device="cuda")
    SD.fill_normal_(values, 21, S.TID_VALUES, 1 / np.sqrt(dv))
    idx = rng.integers(0, Np * expand, size=(T, bag)).astype(np.int32)
    if bag > 1:
        idx[:, 1] = idx[:, 0]
    w = rng.standard_normal((T, bag) + ((cores,) if cores > 1 else ())).astype(np.float32)
    perm = rng.permutation(Np * expand).astype(np.int32) if expand > 1 else None
    out = torch.empty((T, expand, dv), dtype=torch.float32, device="cuda")
    U.check(U.umem_gather_sum(Np, dv, vdtype, values, T, bag, torch.from_numpy(idx).cuda(),
                              torch.from_numpy(w).cuda(),
                              None if perm is None else torch.from_numpy(perm).cuda(), expand,
                              cores, out))
    torch.cuda.synchronize()
    vals = values.float().cpu().numpy().astype(np.float64)
    ref = O.gather_sum(lambda r: vals[r], idx, w, perm, Np, expand)
    err = np.abs(out.cpu().numpy() - ref).max() / np.abs(ref).max()
    log(f"[report] gather T={T} dv={dv} E={expand} bag={bag} cores={cores}: err={err:.2e}")
    assert err <= 1e-5


@pytest.mark.parametrize("T,E,dv,dvv,dout", [(70, 4, 512, 512, 2048), (5, 1, 256, 0, 96),
                                              (130, 9, 64, 80, 0),
                                              # long K over few tiles: split reductions
                                              (37, 4, 4096, 1024, 2048), (200, 1, 2048, 0, 64)])
def test_project_standalone(T, E, dv, dvv, dout):
    rng = np.random.default_rng(T)
    pooled = rng.standard_normal((T, E, dv)).astype(np.float32)
    kin = dv if dvv == 0 else dvv
    wp = S.f32_to_bf16_bits(rng.standard_normal((E, dv, dvv)) / np.sqrt(dv)).reshape(E, dv, dvv) if dvv else None
    wo = S.f32_to_bf16_bits(rng.standard_normal((kin, dout)) / np.sqrt(kin)).reshape(kin, dout) if dout else None
    width = dout if dout else dvv
    out = torch.empty((T, width), dtype=torch.float32, device="cuda")
    st, nws = U.umem_project_workspace_size(T, E, dv, dvv, dout)
    U.check(st)
    ws = torch.empty(max(nws, 256), dtype=torch.uint8, device="cuda")
    # the GPU takes the weights output-major ([out, in]), as a linear layer stores them
    dev = lambda a: None if a is None else torch.from_numpy(CF.output_major(a).view(np.int16)).cuda()
    U.check(U.umem_project(T, E, dv, dvv, dout, torch.from_numpy(pooled).cuda(), dev(wp), dev(wo), out,
                           ws, ws.numel()))
    torch.cuda.synchronize()
    f = lambda a: None if a is None else S.bf16_bits_to_f32(a).reshape(a.shape)
    ref = O.ive_project(pooled, f(wp), f(wo)) if dvv else pooled[:, 0, :].astype(np.float64) @ f(wo)
    err = (np.abs(out.cpu().numpy() - ref).max(axis=1) / np.abs(ref).max(axis=1)).max()
    log(f"[report] project T={T} E={E}: err={err:.2e}")
    assert err <= 2e-2


def test_project_banded_split_k_stays_in_workspace():
    """An output linear whose fp32 input (400 x 2^20, 1.68 GB) is launched in two bands of rows
    (384 and 16) with K split per band: the partial sums stay inside the workspace the library
    asked for (a guard region behind it keeps its fill), and sampled rows match the oracle."""
    T, dv, dout = 400, 1 << 20, 8
    log(f"[case] banded project T={T} K={dv} N={dout}")
    st, nws = U.umem_project_workspace_size(T, 1, dv, 0, dout)
    U.check(st)
    guard = 1 << 20
    ws = torch.full((nws + guard,), 0x5A, dtype=torch.uint8, device="cuda")
    gen = torch.Generator(device="cuda").manual_seed(40)
    pooled = torch.randn((T, 1, dv), generator=gen, dtype=torch.float32, device="cuda")
    rng = np.random.default_rng(40)
    wo = S.f32_to_bf16_bits(rng.standard_normal((dv, dout)) / np.sqrt(dv)).reshape(dv, dout)
    out = torch.empty((T, dout), dtype=torch.float32, device="cuda")
    U.check(U.umem_project(T, 1, dv, 0, dout, pooled, None,
                           torch.from_numpy(CF.output_major(wo).view(np.int16)).cuda(), out, ws, nws))
    torch.cuda.synchronize()
    assert bool((ws[nws:] == 0x5A).all()), "split-K partials written past the workspace"
    rows = np.array([0, 1, 200, 383, 384, 390, 399])
    a = pooled[torch.from_numpy(rows).cuda(), 0].cpu().numpy().astype(np.float64)
    ref = a @ S.bf16_bits_to_f32(wo).reshape(wo.shape).astype(np.float64)
    got = out.cpu().numpy()[rows]
    err = (np.abs(got - ref).max(axis=1) / np.abs(ref).max(axis=1)).max()
    log(f"[report] banded project: err={err:.2e}")
    assert err <= 2e-2
    del pooled, ws


# ---------------------------------------------------------------- the paper-scale workloads

@pytest.mark.parametrize("kw", [
    # expansion, both GEMMs, the projection's K split
    dict(T=70, heads=2, dk=64, n_keys=96, topk=16, topm=24, dv=512, vdtype=CF.BF16, rank=2,
         grid=CF.GRID_TUCKER, expand=4, dv_virt=64, d_out=128),
    # the output linear alone, fp32 rows
    dict(T=33, heads=1, dk=64, n_keys=64, topk=8, topm=8, dv=256, vdtype=CF.F32, d_out=96),
    # a wave per token (2,100 tokens), the projectors alone
    dict(T=2100, heads=1, dk=64, n_keys=64, topk=8, topm=8, dv=256, vdtype=CF.BF16, dv_virt=64),
    # multi-core weights with expansion
    dict(T=24, heads=2, dk=128, n_keys=128, rank=2, grid=CF.GRID_TUCKER, topk=16, topm=32,
         dv=512, vdtype=CF.BF16, expand=4, dv_virt=256, d_out=192, cores=2),
], ids=["ive-two-gemms", "output-linear", "wave-per-token", "multi-core"])
def test_forward_projection_is_gather_then_project(kw):
    """The forward hands its projection the pooled rows in bf16, rounded as the projection's GEMM
    rounds an fp32 operand: its output equals umem_gather_sum (fp32 rows) followed by
    umem_project, bit for bit."""
    cfg = small("fwd-parts", **kw)
    log(f"[case] forward = gather + project: {kw}")
    dl = SD.make_layer(cfg)
    T = cfg.T
    w_proj, w_out = dl.w_proj, dl.w_out      # the output linear alone: w_out [d_out, dv]
    desc = G.desc_for(cfg)
    out_f = torch.empty((T, cfg.d_out or cfg.dv_virt), dtype=torch.float32, device="cuda")
    idx_f = torch.empty((T, cfg.heads, cfg.topm), dtype=torch.int32, device="cuda")
    w_f = torch.empty(G.weights_shape(cfg, T), dtype=torch.float32, device="cuda")
    ws = G.workspace(desc, T)
    U.check(U.umem_forward(desc, T, dl.q_row[0], dl.q_col[0], dl.k_row, dl.k_col, dl.core,
                           dl.values, dl.perm, w_proj, w_out, out_f, idx_f, w_f, ws, ws.numel()),
            "umem_forward")
    pooled = G.gather(dl, idx_f, w_f, T)
    st, nws = U.umem_project_workspace_size(T, cfg.expand, cfg.dv, cfg.dv_virt, cfg.d_out)
    U.check(st)
    ws_p = torch.empty(max(nws, 256), dtype=torch.uint8, device="cuda")
    out_p = torch.empty_like(out_f)
    U.check(U.umem_project(T, cfg.expand, cfg.dv, cfg.dv_virt, cfg.d_out, pooled, w_proj, w_out,
                           out_p, ws_p, ws_p.numel()), "umem_project")
    torch.cuda.synchronize()
    assert torch.equal(out_f, out_p)


def test_c2_prefill_sampled():
    rng = np.random.default_rng(2)
    run_and_check(CF.C2, tokens=np.sort(rng.choice(CF.C2.T, 256, replace=False)))


@pytest.fixture(scope="module")
def c3_values():
    """The 20.07M x 512 bf16 value table of the decode layer (20.55 GB), drawn once for the decode
    tests of this module."""
    cfg = CF.C3
    v = torch.empty((cfg.n_values, cfg.dv), dtype=torch.bfloat16, device="cuda")
    SD.fill_normal_(v, cfg.seed, S.TID_VALUES, CF.value_std(cfg))
    yield v
    del v
    torch.cuda.empty_cache()


def test_c3_decode_20m_full_size(c3_values):
    # every token of the 32-token decode batch, 20.07M-slot table
    run_and_check(CF.C3, dl=SD.make_layer(CF.C3, values=c3_values))


@pytest.mark.parametrize("T", CF.C4_BATCHES)
def test_c4_decode_batches(T, c3_values):
    """The decode batch sweep on the 20.07M-slot layer.  Up to 128 tokens the selection pools the
    rows itself (scoring clears the output first: the split and the 32 x 32 kernel); at 256 and
    1024 the gather kernel pools them.  Every token up to 256, 256 of 1024."""
    rng = np.random.default_rng(T)
    tokens = None if T <= 256 else np.sort(rng.choice(T, 256, replace=False))
    cfg = CF.C3.with_tokens(T)
    run_and_check(cfg, batch=1, tokens=tokens, dl=SD.make_layer(cfg, batches=2, values=c3_values))


@pytest.mark.parametrize("n_keys", [300, 301], ids=["planes", "tiled"])
def test_fused_forward_many_tokens(n_keys):
    """The forward with the selection pooling the rows for 64 < T <= 128 tokens (two heads, 1 KiB
    bf16 rows, no projection): the scoring kernel, here the fp16-plane one (n % 4 == 0) or the
    tiled fp32 MFMA one (n % 4 != 0), clears the output with its grid before the selection adds
    both heads' rows into it.  A ragged token tile (100 of 128)."""
    cfg = small("fused-many", T=100, heads=2, dk=128, n_keys=n_keys, topk=16, topm=24, dv=512,
                vdtype=CF.BF16, seed=31)
    run_and_check(cfg)


def test_c5_tucker_ive_sampled():
    rng = np.random.default_rng(5)
    run_and_check(CF.C5, tokens=np.sort(rng.choice(CF.C5.T, 256, replace=False)))


@pytest.mark.parametrize("heads", [1, 2])
def test_deterministic(heads):
    # two heads pool into the same rows with atomic adds: two adds onto zero commute exactly
    cfg = CF.C1 if heads == 1 else small("det2", T=40, heads=2, n_keys=200, topk=16, topm=24,
                                         dv=512, vdtype=CF.BF16)
    dl = SD.make_layer(cfg)
    a = G.forward(dl, cfg.T)
    b = G.forward(dl, cfg.T)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x, y)


def test_two_streams_concurrently():
    """Forwards of two layers (one pooling inside the selection, one with expansion and the
    projection) issued alternately on two streams, each with its own workspace, give the results
    each gives alone: every launch goes to the caller's stream and the library holds no state
    between calls."""
    cfgs = [small("s1", T=40, heads=2, n_keys=200, topk=16, topm=24, dv=512, vdtype=CF.BF16),
            small("s2", T=130, heads=2, dk=64, n_keys=96, topk=16, topm=24, dv=512, vdtype=CF.BF16,
                  rank=2, grid=CF.GRID_TUCKER, expand=4, dv_virt=64, d_out=128)]
    dls = [SD.make_layer(c, batches=2) for c in cfgs]
    want = []
    for dl, c in zip(dls, cfgs):
        want.append([G.forward(dl, c.T, b) for b in range(2)])
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    got = [[None, None], [None, None]]
    for rep in range(3):
        for b in range(2):
            for i, (dl, c) in enumerate(zip(dls, cfgs)):
                with torch.cuda.stream(streams[i]):
                    got[i][b] = G.forward(dl, c.T, b)
        torch.cuda.synchronize()
        for i in range(2):
            for b in range(2):
                for x, y in zip(got[i][b], want[i][b]):
                    assert torch.equal(x, y), (rep, i, b)


def test_hip_graph_replay_matches_eager():
    """Forwards captured in a HIP graph, replayed several times with eager work in between, give
    the eager results bit for bit."""
    cfg = CF.C1
    dl = SD.make_layer(cfg, batches=3)
    desc = G.desc_for(cfg)
    T = cfg.T
    ws = G.workspace(desc, T)
    outs = [torch.empty((T, cfg.dv), dtype=torch.float32, device="cuda") for _ in range(3)]
    idxs = [torch.empty((T, cfg.heads, cfg.topm), dtype=torch.int32, device="cuda") for _ in range(3)]
    wts = [torch.empty((T, cfg.heads, cfg.topm), dtype=torch.float32, device="cuda") for _ in range(3)]

    def step(b):
        U.check(U.umem_forward(desc, T, dl.q_row[b], dl.q_col[b], dl.k_row, dl.k_col, None, dl.values,
                               None, None, None, outs[b], idxs[b], wts[b], ws, ws.numel()))

    for b in range(3):
        step(b)
    torch.cuda.synchronize()
    want = [(o.clone(), i.clone(), w.clone()) for o, i, w in zip(outs, idxs, wts)]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for b in range(3):
            step(b)
    for rep in range(4):
        for t in outs + wts:
            t.fill_(-1.0)
        for t in idxs:
            t.fill_(-1)
        g.replay()
        torch.cuda.synchronize()
        for b in range(3):
            assert torch.equal(outs[b], want[b][0]) and torch.equal(idxs[b], want[b][1])
            assert torch.equal(wts[b], want[b][2])
        step(0)                     # eager work between replays
        torch.cuda.synchronize()


def test_graph_replay_projected_layer_stale_workspace():
    """A Tucker + IVE layer with projection at 130 tokens (scoring on fp16 planes, the expanded
    gather, the projection with a split K) captured in a HIP graph and replayed with a
    garbage-filled workspace and eager work between replays gives the eager results bit for
    bit: nothing reads the workspace before writing it."""
    cfg = small("graph-ive", T=130, heads=2, dk=64, n_keys=96, topk=16, topm=24, dv=512,
                vdtype=CF.BF16, rank=2, grid=CF.GRID_TUCKER, expand=4, dv_virt=64, d_out=128)
    dl = SD.make_layer(cfg)
    desc = G.desc_for(cfg)
    T = cfg.T
    ws = G.workspace(desc, T)
    out = torch.empty((T, cfg.d_out), dtype=torch.float32, device="cuda")
    idx = torch.empty((T, cfg.heads, cfg.topm), dtype=torch.int32, device="cuda")
    w = torch.empty((T, cfg.heads, cfg.topm), dtype=torch.float32, device="cuda")

    def step():
        U.check(U.umem_forward(desc, T, dl.q_row[0], dl.q_col[0], dl.k_row, dl.k_col, dl.core,
                               dl.values, dl.perm, dl.w_proj, dl.w_out, out, idx, w, ws, ws.numel()),
                "umem_forward")

    step()
    torch.cuda.synchronize()
    want = (out.clone(), idx.clone(), w.clone())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for rep in range(4):
        out.fill_(-1.0)
        w.fill_(-1.0)
        idx.fill_(-1)
        ws.fill_(0x5A)
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, want[0]) and torch.equal(idx, want[1]) and torch.equal(w, want[2]), rep
        step()
        torch.cuda.synchronize()


@pytest.mark.parametrize("kw", [
    dict(T=3, heads=2, n_keys=2048, topk=32, topm=32, dv=8, vdtype=CF.BF16),        # float4 loads
    dict(T=2, heads=1, n_keys=1001, topk=20, topm=50, dv=8, vdtype=CF.BF16),        # scalar loads
    dict(T=2, heads=2, n_keys=200, dk=64, rank=2, grid=CF.GRID_TUCKER, topk=40, topm=64, dv=8,
         vdtype=CF.BF16),                                                            # 1600 tied candidates
], ids=["axis-vec4", "axis-scalar", "tucker-grid"])
def test_massive_ties_fallbacks(kw):
    """All-zero queries: every score ties (as +0.0 or -0.0), far more survivors than the
    threshold filter's buffers hold, so the exact fallbacks decide; ties go to lower indices."""
    cfg = small("massive-ties", **kw)
    dl = SD.make_layer(cfg)
    z = np.zeros((cfg.T, cfg.heads, cfg.dk), np.float32)
    dl.q_row = torch.from_numpy(z[None]).cuda()
    dl.q_col = torch.from_numpy(z[None]).cuda()
    idx, w, ax = G.score_topk(dl, cfg.T)
    torch.cuda.synchronize()
    kr, kc = CF.keys(cfg)
    _, rep = P.check_selection(cfg, z, z, kr, kc, CF.core(cfg), G.host(idx), G.host(w), G.host(ax),
                               gap=0.0)
    log(f"[report] massive ties {kw}: {rep}")
    assert rep["e2e_slot_mismatch"] == 0
    # the lowest indices win: axis lists are 0..k-1
    assert np.array_equal(G.host(ax)[:, :, :, :], np.broadcast_to(np.arange(cfg.topk), G.host(ax).shape))
