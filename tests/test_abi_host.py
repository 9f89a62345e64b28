"""The C ABI on the host: the library loads, exports exactly what include/umem.h declares, and
rejects bad arguments before it touches the GPU.  No kernel is launched here: every call below
fails validation (or only sizes the workspace)."""
import ctypes
import os
import re

import pytest

import paper_2411_12364_amd as U
from synth import configs as CF

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    text = open(os.path.join(ROOT, "include", "umem.h")).read()
    return set(re.findall(r"UMEM_API\s+[\w\s\*]+?\b(umem_\w+)\s*\(", text))


def test_header_and_binding_agree():
    names = declared_symbols()
    assert names == set(U.EXPORTED)
    lib = ctypes.CDLL(U.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


def test_only_abi_symbols_exported():
    out = os.popen(f"nm -D --defined-only {U.LIB_PATH}").read()
    exported = {l.split()[-1] for l in out.splitlines() if l.split() and l.split()[1] == "T"}
    assert {s for s in exported if not s.startswith("_")} == declared_symbols()


def desc(**kw):
    d = U.umem_desc()
    base = dict(heads=2, dk=128, n_keys=4480, rank=1, topk=32, topm=32, grid=0, weight=0,
                n_values=4480 * 4480, dv=512, vdtype=1, expand=1, dv_virt=0, d_out=0, cores=0)
    base.update(kw)
    for k, v in base.items():
        setattr(d, k, v)
    return d


def test_status_strings():
    for st in (0, -1, -2, -3, -4):
        assert U.umem_status_string(st)
    assert U.umem_status_string(7) == "unknown status"


def test_workspace_size_layout():
    st, n = U.umem_workspace_size(desc(), 32)
    assert st == U.UMEM_OK
    sel = 2 * 32 * 2 * 4480 * 4
    assert n >= sel + 2 * 32 * 2 * 32 * 4 and n % 256 == 0
    st, n0 = U.umem_workspace_size(desc(), 0)
    assert st == U.UMEM_OK and n0 == 0
    # Tucker + IVE + projections need the pooled sums and the intermediate
    c5 = desc(heads=4, n_keys=2048, rank=2, grid=1, topk=64, topm=64, n_values=1 << 20, expand=4,
              dv_virt=512, d_out=2048)
    st, n5 = U.umem_workspace_size(c5, 4096)
    assert st == U.UMEM_OK
    assert n5 >= 2 * 4096 * 4 * 2048 * 4 + 4096 * 4 * 512 * 4 + 4096 * 512 * 4


@pytest.mark.parametrize("kw,want", [
    (dict(heads=0), U.UMEM_ERR_INVALID_ARG),
    (dict(topk=4481), U.UMEM_ERR_INVALID_ARG),
    (dict(topm=32 * 32 + 1), U.UMEM_ERR_INVALID_ARG),
    (dict(rank=2), U.UMEM_ERR_INVALID_ARG),                    # additive grid needs rank 1
    (dict(grid=1, rank=3), U.UMEM_ERR_INVALID_ARG),            # dk % rank != 0
    (dict(expand=2, n_values=4480 * 2240, dv_virt=8), U.UMEM_ERR_INVALID_ARG),   # not a square
    (dict(expand=4, n_values=4480 * 1120), U.UMEM_ERR_INVALID_ARG),              # no D'v
    (dict(n_values=1000), U.UMEM_ERR_INVALID_ARG),             # N_p * E != n^2
    (dict(vdtype=2), U.UMEM_ERR_INVALID_ARG),
    (dict(cores=-1), U.UMEM_ERR_INVALID_ARG),
    (dict(cores=2), U.UMEM_ERR_INVALID_ARG),                               # MCS needs the Tucker grid
    (dict(cores=2, grid=1, rank=2, weight=1), U.UMEM_ERR_INVALID_ARG),     # ... and raw weights
    (dict(cores=3, grid=1, rank=2), U.UMEM_ERR_INVALID_ARG),               # dv % h != 0
    (dict(cores=16, grid=1, rank=2), U.UMEM_ERR_UNSUPPORTED),              # h <= 8
    (dict(cores=8, grid=1, rank=2, dv=32), U.UMEM_ERR_UNSUPPORTED),        # 8-byte slices
    (dict(cores=8, grid=1, rank=2, dv=64), U.UMEM_OK),                     # 16-byte slices
    (dict(cores=2, grid=1, rank=2), U.UMEM_OK),
    (dict(cores=1), U.UMEM_OK),
    (dict(n_keys=20000, n_values=20000 * 20000), U.UMEM_ERR_UNSUPPORTED),
    (dict(topk=111, topm=8), U.UMEM_ERR_UNSUPPORTED),
    (dict(topm=300, topk=32), U.UMEM_ERR_UNSUPPORTED),
    (dict(grid=1, rank=8), U.UMEM_ERR_UNSUPPORTED),
    (dict(dv=100), U.UMEM_ERR_UNSUPPORTED),                    # 200-byte rows
    (dict(d_out=100), U.UMEM_ERR_UNSUPPORTED),                 # weight rows of 16-byte pieces
    (dict(dv=4, vdtype=0, d_out=64), U.UMEM_ERR_UNSUPPORTED),  # output linear alone: K = dv, 8 | K
    (dict(dv=8, vdtype=0, d_out=64), U.UMEM_OK),
    (dict(expand=4, n_values=4480 * 1120, dv_virt=260), U.UMEM_ERR_UNSUPPORTED),
    (dict(heads=64, topm=64), U.UMEM_ERR_UNSUPPORTED),         # bag 4096
])
def test_descriptor_validation(kw, want):
    st, n = U.umem_workspace_size(desc(**kw), 8)
    assert st == want and (n == 0) == (st != U.UMEM_OK)


def test_entry_points_reject_before_launch():
    d = desc()
    fake = 1 << 20          # an aligned non-null address; never dereferenced (validation fails)
    assert U.umem_score_topk(d, 8, None, fake, fake, fake, None, fake, fake, None, fake, 1 << 30, 0) == U.UMEM_ERR_INVALID_ARG
    assert U.umem_score_topk(d, 8, fake + 4, fake, fake, fake, None, fake, fake, None, fake, 1 << 30, 0) == U.UMEM_ERR_INVALID_ARG
    assert U.umem_score_topk(d, 8, fake, fake, fake, fake, None, fake, fake, None, fake, 16, 0) == U.UMEM_ERR_WORKSPACE
    assert U.umem_score_topk(d, 8, fake, fake, fake, fake, None, fake, fake, None, fake + 64, 1 << 30, 0) == U.UMEM_ERR_WORKSPACE
    assert U.umem_score_topk(d, -1, fake, fake, fake, fake, None, fake, fake, None, fake, 1 << 30, 0) == U.UMEM_ERR_INVALID_ARG
    assert U.umem_score_topk(d, (1 << 20) + 1, fake, fake, fake, fake, None, fake, fake, None, fake, 1 << 40, 0) == U.UMEM_ERR_UNSUPPORTED
    tucker = desc(grid=1, rank=2)
    assert U.umem_axis_scores(tucker, 8, fake, fake, fake, fake, None, fake, fake, 1 << 20, 0) == U.UMEM_ERR_INVALID_ARG
    assert U.umem_axis_scores(tucker, 8, fake, fake, fake, fake, fake, fake, None, 0, 0) == U.UMEM_ERR_WORKSPACE
    # more than 64 tokens: the fp16 planes of the scoring and their rows' exponents need their
    # scratch after the factors
    planes = 2 * 2 * (100 + 4480) * 2 * 128 * 2 + 2 * (100 + 4480) * 2 * 4
    st, nfull = U.umem_workspace_size(tucker, 100)
    assert st == U.UMEM_OK and nfull >= 2048 + planes
    assert U.umem_axis_scores(tucker, 100, fake, fake, fake, fake, fake, fake, fake, 2048, 0) == U.UMEM_ERR_WORKSPACE
    assert U.umem_axis_scores(tucker, 100, fake, fake, fake, fake, fake, fake, fake, 2048 + planes - 1, 0) == U.UMEM_ERR_WORKSPACE
    additive = desc()
    assert U.umem_axis_scores(additive, 100, fake, fake, fake, fake, None, fake, None, 0, 0) == U.UMEM_ERR_WORKSPACE
    assert U.umem_select(d, 8, None, None, None, None, None, None, fake, fake, None, None, None, 0) == U.UMEM_ERR_INVALID_ARG
    # select with pooling: values and pooled together, aligned, and only where the layer allows
    assert U.umem_select(d, 8, fake, None, None, None, None, None, fake, fake, None, None, fake, 0) == U.UMEM_ERR_INVALID_ARG
    assert U.umem_select(d, 8, fake, None, None, None, None, None, fake, fake, None, fake, fake + 4, 0) == U.UMEM_ERR_INVALID_ARG
    assert U.umem_select(desc(heads=3), 8, fake, None, None, None, None, None, fake, fake, None, fake, fake, 0) == U.UMEM_ERR_UNSUPPORTED
    assert U.umem_select(desc(topm=65, topk=16), 8, fake, None, None, None, None, None, fake, fake, None, fake, fake, 0) == U.UMEM_ERR_UNSUPPORTED
    # gather: bad sizes, misaligned values, bag beyond the limit, unsupported row
    assert U.umem_gather_sum(100, 512, 1, fake, 4, 0, fake, fake, None, 1, 1, fake, 0) == U.UMEM_ERR_INVALID_ARG
    assert U.umem_gather_sum(100, 512, 1, fake + 8, 4, 64, fake, fake, None, 1, 1, fake, 0) == U.UMEM_ERR_INVALID_ARG
    assert U.umem_gather_sum(100, 512, 1, fake, 4, 4096, fake, fake, None, 1, 1, fake, 0) == U.UMEM_ERR_UNSUPPORTED
    assert U.umem_gather_sum(100, 100, 1, fake, 4, 64, fake, fake, None, 1, 1, fake, 0) == U.UMEM_ERR_UNSUPPORTED
    assert U.umem_gather_sum(100, 512, 3, fake, 4, 64, fake, fake, None, 1, 1, fake, 0) == U.UMEM_ERR_INVALID_ARG
    # multi-core weights: dv % h, 16-byte slices, h <= 8
    assert U.umem_gather_sum(100, 512, 1, fake, 4, 64, fake, fake, None, 1, 3, fake, 0) == U.UMEM_ERR_INVALID_ARG
    assert U.umem_gather_sum(100, 8, 1, fake, 4, 64, fake, fake, None, 1, 2, fake, 0) == U.UMEM_ERR_UNSUPPORTED
    assert U.umem_gather_sum(100, 512, 1, fake, 4, 64, fake, fake, None, 1, 16, fake, 0) == U.UMEM_ERR_UNSUPPORTED
    assert U.umem_gather_sum(100, 512, 1, fake, 4, 64, fake, fake, None, 1, -1, fake, 0) == U.UMEM_ERR_INVALID_ARG
    # projection: missing weights / workspace
    assert U.umem_project(8, 4, 512, 512, 2048, fake, fake, None, fake, fake, 1 << 20, 0) == U.UMEM_ERR_INVALID_ARG
    assert U.umem_project(8, 4, 512, 512, 2048, fake, fake, fake, fake, fake, 64, 0) == U.UMEM_ERR_WORKSPACE
    # workspace of the projection: the intermediate plus split-K partials where K is long
    st, n = U.umem_project_workspace_size(8, 4, 512, 512, 2048)
    assert st == U.UMEM_OK and n >= 8 * 512 * 4
    st, n1 = U.umem_project_workspace_size(512, 4, 4096, 1024, 2048)
    assert st == U.UMEM_OK and n1 >= 512 * 1024 * 4 * 2       # K = 16384 over 64 tiles: split
    st, n2 = U.umem_project_workspace_size(1 << 16, 4, 512, 512, 2048)
    assert st == U.UMEM_OK and n2 == ((1 << 16) * 512 * 4 + 255) // 256 * 256   # many tiles: none
    assert U.umem_project_workspace_size(0, 4, 512, 512, 2048) == (U.UMEM_OK, 0)
    assert U.umem_project_workspace_size(8, 4, 512, 516, 2048)[0] == U.UMEM_ERR_UNSUPPORTED
    assert U.umem_project_workspace_size(8, 2, 512, 0, 2048)[0] == U.UMEM_ERR_INVALID_ARG
    assert U.umem_project(8, 4, 512, 512, 2048, fake, fake, fake, fake, fake, n - 16, 0) == U.UMEM_ERR_WORKSPACE
    # the GEMMs read 16-byte pieces of pooled rows and weight rows
    assert U.umem_project(8, 4, 512, 516, 2048, fake, fake, fake, fake, fake, 1 << 20, 0) == U.UMEM_ERR_UNSUPPORTED
    assert U.umem_project(8, 4, 512, 512, 2044, fake, fake, fake, fake, fake, 1 << 20, 0) == U.UMEM_ERR_UNSUPPORTED
    assert U.umem_project(8, 1, 6, 0, 64, fake, None, fake, fake, None, 0, 0) == U.UMEM_ERR_UNSUPPORTED
    assert U.umem_project(8, 3, 4, 8, 64, fake, fake, fake, fake, fake, 1 << 20, 0) == U.UMEM_ERR_UNSUPPORTED  # K = 12
    # weights within the loads' 32-bit byte range: [8192, 4 * 65536] bf16 is 4 GiB
    assert U.umem_project_workspace_size(8, 4, 65536, 8192, 0)[0] == U.UMEM_ERR_UNSUPPORTED
    assert U.umem_project(8, 4, 512, 512, 2048, fake, fake + 8, fake, fake, fake, 1 << 20, 0) == U.UMEM_ERR_UNSUPPORTED
    assert U.umem_project(8, 4, 512, 512, 2048, fake + 4, fake, fake, fake, fake, 1 << 20, 0) == U.UMEM_ERR_UNSUPPORTED
    # forward: perm required iff expand > 1, projection weights iff D'v / d_out
    ive = desc(heads=4, n_keys=2048, rank=2, grid=1, topk=64, topm=64, n_values=1 << 20, expand=4,
               dv_virt=512, d_out=2048)
    big = 1 << 36
    assert U.umem_forward(ive, 8, fake, fake, fake, fake, fake, fake, None, fake, fake, fake, None, None, fake, big, 0) == U.UMEM_ERR_INVALID_ARG
    assert U.umem_forward(ive, 8, fake, fake, fake, fake, fake, fake, fake, None, fake, fake, None, None, fake, big, 0) == U.UMEM_ERR_INVALID_ARG
    assert U.umem_forward(d, 8, fake, fake, fake, fake, None, fake, fake, None, None, fake, None, None, fake, big, 0) == U.UMEM_ERR_INVALID_ARG


def test_zero_tokens_is_a_noop():
    d = desc()
    assert U.umem_score_topk(d, 0, None, None, None, None, None, None, None, None, None, 0, 0) == U.UMEM_OK
    assert U.umem_forward(d, 0, None, None, None, None, None, None, None, None, None, None, None, None, None, 0, 0) == U.UMEM_OK
    assert U.umem_gather_sum(100, 512, 1, None, 0, 64, None, None, None, 1, 1, None, 0) == U.UMEM_OK


def test_one_hip_runtime_in_process():
    """The binding loads torch's HIP runtime before libumem.so, so the process maps a single
    libamdhip64 (two copies would not share devices, streams or memory)."""
    with open("/proc/self/maps") as f:
        paths = {line.split()[-1] for line in f if "libamdhip64" in line}
    assert len({os.path.realpath(p) for p in paths}) == 1, paths


def qdesc(**kw):
    d = U.umem_query_desc()
    base = dict(d_model=2048, conv_k=4, heads=2, dk=448, shared=1, eps=1e-5)
    base.update(kw)
    for k, v in base.items():
        setattr(d, k, v)
    return d


@pytest.mark.parametrize("kw,want", [
    (dict(), U.UMEM_OK),
    (dict(d_model=0), U.UMEM_ERR_INVALID_ARG),
    (dict(conv_k=0), U.UMEM_ERR_INVALID_ARG),
    (dict(shared=2), U.UMEM_ERR_INVALID_ARG),
    (dict(eps=-1.0), U.UMEM_ERR_INVALID_ARG),
    (dict(eps=float("nan")), U.UMEM_ERR_INVALID_ARG),
    (dict(d_model=2046), U.UMEM_ERR_UNSUPPORTED),          # 16-byte pieces of a hidden row
    (dict(d_model=2052), U.UMEM_ERR_UNSUPPORTED),          # 16-byte pieces of a weight row (bf16)
    (dict(d_model=1 << 20, heads=8, dk=256, shared=0), U.UMEM_ERR_UNSUPPORTED),   # a 8 GiB weight
    (dict(d_model=1 << 21, heads=1, dk=4, shared=0), U.UMEM_ERR_UNSUPPORTED),     # K beyond 2^20
    (dict(conv_k=9), U.UMEM_ERR_UNSUPPORTED),
    (dict(dk=1028), U.UMEM_ERR_UNSUPPORTED),
    (dict(heads=1, dk=4), U.UMEM_ERR_UNSUPPORTED),         # 4 query outputs: not whole 16-byte pieces
    (dict(heads=1, dk=4, shared=0), U.UMEM_OK),
])
def test_query_desc_validation(kw, want):
    st, n = U.umem_query_workspace_size(qdesc(**kw), 512, 1)
    assert st == want and (n == 0) == (st != U.UMEM_OK)


def test_query_workspace_and_entry_validation():
    qd = qdesc()
    st, n = U.umem_query_workspace_size(qd, 512, 1)
    assert st == U.UMEM_OK and n >= 512 * 2048 * 4 + 512 * 2 * 448 * 4
    assert U.umem_query_workspace_size(qd, 0, 5) == (U.UMEM_OK, 0)
    assert U.umem_query_workspace_size(qd, -1, 5)[0] == U.UMEM_ERR_INVALID_ARG
    assert U.umem_query_workspace_size(qd, 1 << 20, 2)[0] == U.UMEM_ERR_UNSUPPORTED
    fake = 1 << 20
    args = [fake, fake, fake, fake, fake, fake, fake, None]    # x, hist, conv_w, w_q, gamma, beta, q_row, q_col
    bad = list(args)
    bad[0] = None
    assert U.umem_query(qd, 512, 1, *bad, fake, n, 0) == U.UMEM_ERR_INVALID_ARG
    bad = list(args)
    bad[7] = fake                                              # q_col with a shared query
    assert U.umem_query(qd, 512, 1, *bad, fake, n, 0) == U.UMEM_ERR_INVALID_ARG
    bad = list(args)
    bad[3] = fake + 8                                          # w_q not 16-byte aligned
    assert U.umem_query(qd, 512, 1, *bad, fake, n, 0) == U.UMEM_ERR_INVALID_ARG
    assert U.umem_query(qd, 512, 1, *args, fake, n - 16, 0) == U.UMEM_ERR_WORKSPACE
    assert U.umem_query(qd, 0, 1, None, None, None, None, None, None, None, None, None, 0, 0) == U.UMEM_OK
    assert U.umem_key_norm(2, 0, 448, fake, fake, fake, 1e-5, fake, 0) == U.UMEM_ERR_INVALID_ARG
    assert U.umem_key_norm(2, 16, 1100, fake, fake, fake, 1e-5, fake, 0) == U.UMEM_ERR_UNSUPPORTED
    assert U.umem_key_norm(2, 16, 448, fake + 2, fake, fake, 1e-5, fake, 0) == U.UMEM_ERR_INVALID_ARG
    assert U.umem_key_norm(2, 16, 448, fake, fake, fake, -1.0, fake, 0) == U.UMEM_ERR_INVALID_ARG


def test_backward_validation():
    fake = 1 << 20
    st, n = U.umem_gather_backward_workspace_size(4096, 256, 512)
    assert st == U.UMEM_OK and n >= 4096 * 256 * 16
    assert U.umem_gather_backward_workspace_size(0, 64, 512) == (U.UMEM_OK, 0)
    assert U.umem_gather_backward_workspace_size(1 << 16, 128, 512)[0] == U.UMEM_ERR_UNSUPPORTED
    g = [100, 512, 1, fake, 4, 64, fake, fake, None, 1, 1]           # as umem_gather_sum
    assert U.umem_gather_backward(*g, None, fake, fake, fake, n, 0) == U.UMEM_ERR_INVALID_ARG   # d_pooled
    assert U.umem_gather_backward(*g, fake, fake, None, fake, n, 0) == U.UMEM_ERR_INVALID_ARG   # dw
    assert U.umem_gather_backward(*g, fake + 4, fake, fake, fake, n, 0) == U.UMEM_ERR_INVALID_ARG
    assert U.umem_gather_backward(*g, fake, fake, fake, fake, 16, 0) == U.UMEM_ERR_WORKSPACE
    g4 = list(g)
    g4[9] = 4                                                          # expand without perm
    assert U.umem_gather_backward(*g4, fake, fake, fake, fake, n, 0) == U.UMEM_ERR_INVALID_ARG
    # the compact form: d_pooled, rows, d_rows, n_rows, dw, ws, ws_bytes, stream
    R = U.umem_gather_backward_rows
    assert R(*g, None, fake, fake, fake, fake, fake, n, 0) == U.UMEM_ERR_INVALID_ARG     # d_pooled
    assert R(*g, fake, None, fake, fake, fake, fake, n, 0) == U.UMEM_ERR_INVALID_ARG     # rows
    assert R(*g, fake, fake, None, fake, fake, fake, n, 0) == U.UMEM_ERR_INVALID_ARG     # d_rows
    assert R(*g, fake, fake, fake, None, fake, fake, n, 0) == U.UMEM_ERR_INVALID_ARG     # n_rows
    assert R(*g, fake, fake, fake + 4, fake, fake, fake, n, 0) == U.UMEM_ERR_INVALID_ARG  # d_rows aligned
    assert R(*g, fake, fake + 2, fake, fake, fake, fake, n, 0) == U.UMEM_ERR_INVALID_ARG  # rows aligned
    assert R(*g, fake, fake, fake, fake, fake, fake, 16, 0) == U.UMEM_ERR_WORKSPACE
    assert R(*g4, fake, fake, fake, fake, fake, fake, n, 0) == U.UMEM_ERR_INVALID_ARG
    g0 = list(g)
    g0[4] = 0                                                          # T == 0: nothing to do
    assert R(*g0, None, None, None, None, None, None, 0, 0) == U.UMEM_OK
    d = desc(grid=1, rank=2)
    st, ns = U.umem_score_backward_workspace_size(d, 32)
    assert st == U.UMEM_OK and ns > 0
    a = [d, 32, fake, fake, fake, fake, fake, fake, fake, fake]        # ... core, idx, w, dw
    assert U.umem_score_backward(*a, fake, fake, fake, fake, None, fake, ns, 0) == U.UMEM_ERR_INVALID_ARG  # dcore
    assert U.umem_score_backward(*a, fake, fake, fake + 4, fake, fake, fake, ns, 0) == U.UMEM_ERR_INVALID_ARG
    assert U.umem_score_backward(*a, fake, fake, fake, fake, fake, fake, 64, 0) == U.UMEM_ERR_WORKSPACE
    da = desc()
    a = [da, 32, fake, fake, fake, fake, None, fake, None, fake]
    assert U.umem_score_backward(*a, fake, fake, fake, fake, fake, fake, ns, 0) == U.UMEM_ERR_INVALID_ARG  # dcore, additive
    ds = desc(weight=1)
    a = [ds, 32, fake, fake, fake, fake, None, fake, None, fake]        # SoftMax needs w
    assert U.umem_score_backward(*a, fake, fake, fake, fake, None, fake, ns, 0) == U.UMEM_ERR_INVALID_ARG
    assert U.umem_score_backward_workspace_size(desc(heads=64, topm=32), 1 << 11)[0] == U.UMEM_ERR_UNSUPPORTED


def _split_ways(rows, N, K):
    """The projection GEMM's split of K, as its header states it: doubled while the launch has
    fewer than 512 work items and each split keeps at least 4 K-steps of 64."""
    tiles = -(-rows // 128) * -(-N // 128)
    S = 1
    while tiles * S < 512 and K // (2 * S) >= 4 * 64:
        S *= 2
    return S


def _partials_needed(M, N, K):
    """Bytes of split-K partials the largest launch of one GEMM writes.  A's bytes must stay in a
    32-bit buffer range, so A is launched in bands of the largest multiple of 128 rows below
    2 GiB; each band splits K for its own tile count."""
    band = max(128, ((2 ** 31 - 1) // (K * 4)) // 128 * 128)
    shapes = [M] if M <= band else [band, M - (M - 1) // band * band]
    need = 0
    for rows in shapes:
        S = _split_ways(rows, N, K)
        if S > 1:
            need = max(need, S * rows * N * 4)
    return need


@pytest.mark.parametrize("T,E,dv,dvv,dout", [
    (2048, 1, 1 << 18, 0, 128),      # two bands of 1920 and 128 rows: 64-way split of the first
    (1921, 1, 1 << 18, 0, 128),
    (400, 1, 1 << 20, 0, 8),         # bands of 384 and 16 rows
    (16300, 16, 2048, 256, 0),       # the IVE projector alone at E = 16, 16.3K tokens
    (512, 4, 4096, 1024, 2048),      # no band: the whole matrix in one launch
])
def test_project_workspace_covers_every_band(T, E, dv, dvv, dout):
    """The split-K scratch covers the largest band: a band of fewer rows than the whole matrix
    has fewer tiles and may split K more ways."""
    st, n = U.umem_project_workspace_size(T, E, dv, dvv, dout)
    assert st == U.UMEM_OK
    if dvv == 0:
        need = _partials_needed(T, dout, dv)
    else:
        tmp = -(-(T * dvv * 4) // 256) * 256 if dout else 0
        need = tmp + max(_partials_needed(T, dvv, E * dv), _partials_needed(T, dout, dvv) if dout else 0)
    assert n >= need, (n, need)


def test_random_layers_are_accepted():
    """Every seeded random layer of tests/test_gpu_random_layers.py passes the descriptor checks
    (so its GPU case tests the kernels, not a refusal)."""
    from tests.gpu_util import desc_for
    from tests.test_gpu_random_layers import N_CASES, random_layer
    for i in range(N_CASES):
        cfg = random_layer(i)
        st, nbytes = U.umem_workspace_size(desc_for(cfg), cfg.T)
        assert st == U.UMEM_OK, (i, cfg)


def test_random_front_ends_are_accepted():
    from tests.test_gpu_random_layers import N_FRONT_ENDS, random_front_end
    for i in range(N_FRONT_ENDS):
        fe = random_front_end(i)
        d = U.umem_query_desc()
        d.d_model, d.conv_k, d.heads, d.dk = fe.d_model, fe.conv_k, fe.heads, fe.dk
        d.shared, d.eps = int(fe.shared), fe.eps
        st, nbytes = U.umem_query_workspace_size(d, fe.B, fe.L)
        assert st == U.UMEM_OK, (i, fe)
