"""GPU parity of the query front-end and the key LayerNorm through the C ABI, against the
front-end oracle on the same seeded inputs; and the layer fed end to end with the queries and
keys they produce."""
from __future__ import annotations

import dataclasses
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():     # collected on CPU hosts too; every test here is gpu-marked
    pytest.skip("no GPU", allow_module_level=True)

import oracle.query_oracle as Q                     # noqa: E402
import paper_2411_12364_amd as U                    # noqa: E402
import synth as S                                   # noqa: E402
from synth import configs as CF                     # noqa: E402
from synth import device as SD                      # noqa: E402
from tests import gpu_util as G                     # noqa: E402
from tests import parity as P                       # noqa: E402

# Query rows: bf16 rounding of the convolved rows before the linear (relative 2^-9 per element)
# gives about 1e-3 of a row's scale after the LayerNorm; the bound leaves a 10x margin.
Q_RTOL = 1e-2


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def qdesc(fe):
    d = U.umem_query_desc()
    d.d_model, d.conv_k, d.heads, d.dk = fe.d_model, fe.conv_k, fe.heads, fe.dk
    d.shared, d.eps = int(fe.shared), fe.eps
    return d


def run_query(fe, inp=None):
    inp = inp or CF.front_end_inputs(fe)
    qd = qdesc(fe)
    st, nws = U.umem_query_workspace_size(qd, fe.B, fe.L)
    U.check(st)
    ws = torch.empty(max(nws, 256), dtype=torch.uint8, device="cuda")
    dev = lambda a: None if a is None else torch.from_numpy(np.ascontiguousarray(a)).cuda()
    q_row = torch.empty((fe.T, fe.heads, fe.dk), dtype=torch.float32, device="cuda")
    q_col = None if fe.shared else torch.empty_like(q_row)
    log(f"[case] query front-end {fe.name}: B={fe.B} L={fe.L} d={fe.d_model} K_c={fe.conv_k} "
        f"H={fe.heads} Dk={fe.dk} shared={fe.shared}")
    U.check(U.umem_query(qd, fe.B, fe.L, dev(inp["x"]), dev(inp["hist"]), dev(inp["conv_w"]),
                         dev(CF.output_major(inp["w_q"]).view(np.int16)), dev(inp["gamma"]), dev(inp["beta"]),
                         q_row, q_col, ws, ws.numel()), "umem_query")
    torch.cuda.synchronize()
    return inp, q_row, (q_row if fe.shared else q_col), ws


def oracle_queries(fe, inp):
    wq = S.bf16_bits_to_f32(inp["w_q"]).reshape(inp["w_q"].shape)
    return Q.query_front_end(inp["x"], inp["conv_w"], wq, inp["gamma"], inp["beta"], fe.heads,
                             fe.dk, fe.shared, inp["hist"], fe.eps)


def rounded_rows_queries(fe, inp):
    """The oracle's steps with the query linear's documented input rounding (the convolved rows
    to bf16, nearest even) applied to the oracle's own fp64 convolution: [T, A, H, Dk]."""
    A = 1 if fe.shared else 2
    wq = S.bf16_bits_to_f32(inp["w_q"]).reshape(inp["w_q"].shape).astype(np.float64)
    y = Q.causal_conv(inp["x"], inp["conv_w"], inp["hist"]).reshape(fe.T, fe.d_model)
    y16 = S.bf16_bits_to_f32(S.f32_to_bf16_bits(y.astype(np.float32))).reshape(y.shape)
    lin = Q.query_linear(y16.astype(np.float64), wq).reshape(fe.T, A, fe.heads, fe.dk)
    g = np.asarray(inp["gamma"], np.float64).reshape(A, fe.heads, fe.dk)
    b = np.asarray(inp["beta"], np.float64).reshape(A, fe.heads, fe.dk)
    return Q.layer_norm(lin, g, b, fe.eps)


ROUNDED_RTOL = 2e-3   # fp32 accumulation, and a rare bf16 rounding decided the other way


def row_err(got, ref):
    got = np.asarray(got, np.float64).reshape(-1, ref.shape[-1])
    ref = np.asarray(ref, np.float64).reshape(-1, ref.shape[-1])
    return float((np.abs(got - ref).max(axis=1) / np.abs(ref).max(axis=1)).max())


CASES = [
    CF.FrontEnd("small-shared", B=2, L=5, d_model=64, conv_k=4, heads=2, dk=64, shared=True, seed=21),
    CF.FrontEnd("separate-start", B=3, L=7, d_model=96, conv_k=3, heads=1, dk=40, shared=False,
                seed=22, history=False),
    CF.FrontEnd("single-tap", B=4, L=2, d_model=128, conv_k=1, heads=2, dk=128, shared=True, seed=23),
    CF.FE6,
    CF.FrontEnd("prefill-chunk", B=2, L=300, d_model=1024, conv_k=4, heads=2, dk=128, shared=False,
                seed=24),
    # the limits: eight taps, Dk = 1024 (16 values per lane in the LayerNorm, which then adds
    # the query linear's 8 split partials in two batches)
    CF.FrontEnd("limits", B=3, L=9, d_model=2048, conv_k=8, heads=2, dk=1024, shared=False, seed=25),
]


@pytest.mark.parametrize("fe", CASES, ids=[c.name for c in CASES])
def test_query_front_end(fe):
    inp, q_row, q_col, ws = run_query(fe)
    # the convolution: the first T * d bf16 values of the workspace (fp32 sums rounded to bf16,
    # against fp64): within half a bf16 step of the exact value (bf16 carries 8 significant bits:
    # at most 2^-8 relative), plus the fp32 sum's own error
    y16 = ws[: fe.T * fe.d_model * 2].view(torch.int16).cpu().numpy()
    y = S.bf16_bits_to_f32(y16).reshape(fe.B, fe.L, fe.d_model).astype(np.float64)
    y_ref = Q.causal_conv(inp["x"], inp["conv_w"], inp["hist"])
    bound = 2.0 ** -8 * np.abs(y_ref) + 1e-6 * np.abs(y_ref).max()
    conv_err = float(np.abs(y - y_ref).max() / np.abs(y_ref).max())
    assert np.all(np.abs(y - y_ref) <= bound), conv_err
    qr_ref, qc_ref = oracle_queries(fe, inp)
    er, ec = row_err(q_row.cpu().numpy(), qr_ref), row_err(q_col.cpu().numpy(), qc_ref)
    r16 = rounded_rows_queries(fe, inp)
    e16 = max(row_err(q.cpu().numpy(), r16[:, 0 if fe.shared else a]) for a, q in enumerate((q_row, q_col)))
    log(f"[report] {fe.name}: conv err {conv_err:.2e}, q_row err {er:.2e}, q_col err {ec:.2e}, "
        f"against bf16-rounded rows {e16:.2e}")
    assert er <= Q_RTOL and ec <= Q_RTOL and e16 <= ROUNDED_RTOL


def test_query_deterministic():
    fe = CF.FE6
    inp, a, _, _ = run_query(fe)
    _, b, _, _ = run_query(fe, inp)
    assert torch.equal(a, b)


def test_query_graph_replay_stale_workspace():
    """The 1.6B-x12 front-end (convolution, split-K query linear, LayerNorm) captured in a HIP
    graph and replayed over a garbage-filled workspace, with eager work between replays, gives
    the eager queries bit for bit."""
    fe = CF.FE6
    inp = CF.front_end_inputs(fe)
    qd = qdesc(fe)
    st, nws = U.umem_query_workspace_size(qd, fe.B, fe.L)
    U.check(st)
    ws = torch.empty(max(nws, 256), dtype=torch.uint8, device="cuda")
    dev = lambda a: None if a is None else torch.from_numpy(np.ascontiguousarray(a)).cuda()
    x, hist, cw = dev(inp["x"]), dev(inp["hist"]), dev(inp["conv_w"])
    wq = dev(CF.output_major(inp["w_q"]).view(np.int16))
    g_, b_ = dev(inp["gamma"]), dev(inp["beta"])
    q_row = torch.empty((fe.T, fe.heads, fe.dk), dtype=torch.float32, device="cuda")
    q_col = None if fe.shared else torch.empty_like(q_row)

    def step():
        U.check(U.umem_query(qd, fe.B, fe.L, x, hist, cw, wq, g_, b_, q_row, q_col, ws, ws.numel()),
                "umem_query")

    step()
    torch.cuda.synchronize()
    want = q_row.clone()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for rep in range(4):
        q_row.fill_(-1.0)
        ws.fill_(0x3C)
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(q_row, want), rep
        step()
        torch.cuda.synchronize()


@pytest.mark.parametrize("H,n,dk", [(2, 300, 64), (4, 2048, 128), (2, 1792, 448), (1, 5, 1000)])
def test_key_norm(H, n, dk):
    cfg = CF.Layer("keys", T=1, heads=H, dk=dk, n_keys=n, topk=1, topm=1, dv=8, vdtype=CF.F32, seed=40 + dk)
    kr, _ = CF.keys(cfg)
    g, b = CF.key_norm_params(cfg)
    keys = torch.from_numpy(kr).cuda()
    out = torch.empty_like(keys)
    U.check(U.umem_key_norm(H, n, dk, keys, torch.from_numpy(g).cuda(), torch.from_numpy(b).cuda(),
                            1e-5, out))
    torch.cuda.synchronize()
    ref = Q.key_norm(kr, g, b, 1e-5)
    err = row_err(out.cpu().numpy(), ref)
    log(f"[report] key norm H={H} n={n} dk={dk}: err {err:.2e}")
    assert err <= 1e-5
    # in place
    U.check(U.umem_key_norm(H, n, dk, keys, torch.from_numpy(g).cuda(), torch.from_numpy(b).cuda(),
                            1e-5, keys))
    torch.cuda.synchronize()
    assert torch.equal(keys, out)


def test_front_end_feeds_the_layer():
    """Queries from the front-end and LayerNormed keys drive the rank-2 Tucker layer with two
    component cores; the selection and pooling are checked against the oracle on those same
    queries and keys."""
    fe = CF.FrontEnd("e2e", B=4, L=8, d_model=128, conv_k=4, heads=2, dk=64, shared=True, seed=31)
    cfg = CF.Layer("e2e-layer", T=fe.T, heads=2, dk=64, n_keys=96, topk=16, topm=24, dv=512,
                   vdtype=CF.BF16, seed=31, rank=2, grid=CF.GRID_TUCKER, cores=2)
    _, q_row, q_col, _ = run_query(fe)
    dl = SD.make_layer(cfg)
    g, b = CF.key_norm_params(cfg)
    kr = torch.empty_like(dl.k_row)
    kc = torch.empty_like(dl.k_col)
    for src, dst in ((dl.k_row, kr), (dl.k_col, kc)):
        U.check(U.umem_key_norm(cfg.heads, cfg.n_keys, cfg.dk, src, torch.from_numpy(g).cuda(),
                                torch.from_numpy(b).cuda(), 1e-5, dst))
    dl = dataclasses.replace(dl, q_row=q_row[None], q_col=q_col[None], k_row=kr, k_col=kc)
    idx, w, ax = G.score_topk(dl, cfg.T, 0)
    pooled = G.gather(dl, idx, w, cfg.T)
    torch.cuda.synchronize()
    qh, kh = q_row.cpu().numpy(), (kr.cpu().numpy(), kc.cpu().numpy())
    _, rep = P.check_selection(cfg, qh, qh, kh[0], kh[1], CF.core(cfg), G.host(idx), G.host(w),
                               G.host(ax))
    _, err = P.check_pooled(cfg, G.value_rows_fn(cfg), G.host(idx), G.host(w), G.host(pooled))
    log(f"[report] front-end -> layer: {rep}, pooled err {err:.2e}")
