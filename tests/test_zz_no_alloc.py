"""umem_forward_noalloc, the forward for callers that cannot allocate: its workspace is the
library's static per-GPU array.  On the GPU it must give umem_forward's results bit for bit (the
same kernels in the same order), on consecutive calls whose second one is smaller and finds the
first one's contents in the array, without changing the GPU's free memory; on the host it
rejects a call whose scratch would not fit before touching the GPU."""
from __future__ import annotations

import dataclasses
import sys

import numpy as np
import pytest

import paper_2411_12364_amd as U
from synth import configs as CF

torch = pytest.importorskip("torch")


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _desc(cfg):
    d = U.umem_desc()
    d.heads, d.dk, d.n_keys, d.rank = cfg.heads, cfg.dk, cfg.n_keys, cfg.rank
    d.topk, d.topm, d.grid, d.weight = cfg.topk, cfg.topm, cfg.grid, cfg.weight
    d.n_values, d.dv, d.vdtype, d.expand = cfg.n_values, cfg.dv, cfg.vdtype, cfg.expand
    d.dv_virt, d.d_out, d.cores = cfg.dv_virt, cfg.d_out, cfg.cores
    return d


# ---------------------------------------------------------------- host: limits, before the GPU

def test_static_scratch_limit_on_the_host():
    """The largest decode-20M batch whose workspace fits the static array, and the first that
    does not: the latter is refused (nothing reaches the GPU; the pointers are never read)."""
    d = _desc(CF.C3)
    fits = [T for T in (778, 779, 780) if U.umem_workspace_size(d, T)[1] <= U.UMEM_STATIC_SCRATCH_BYTES]
    assert fits == [778, 779]
    fake = 1 << 20
    args = [fake] * 4 + [None, fake, None, None, None, fake, None, None, 0]
    assert U.umem_forward_noalloc(d, 780, *args) == U.UMEM_ERR_SCRATCH_LIMIT
    assert U.umem_status_string(U.UMEM_ERR_SCRATCH_LIMIT) != "unknown status"
    assert U.umem_forward_noalloc(d, 0, *([None] * 12), 0) == U.UMEM_OK
    bad = _desc(dataclasses.replace(CF.C3, topk=0))
    assert U.umem_forward_noalloc(bad, 8, *args) == U.UMEM_ERR_INVALID_ARG


# ---------------------------------------------------------------- GPU: against umem_forward

def _small(name, **kw):
    base = dict(T=8, heads=1, dk=64, n_keys=64, topk=8, topm=8, dv=256, vdtype=CF.F32, seed=11)
    base.update(kw)
    return CF.Layer(name, **base)


CASES = [
    # two heads, 1 KiB rows: the selection pools the rows (the scoring clears the output)
    (_small("noalloc-pooled", T=40, heads=2, dk=128, n_keys=150, topk=16, topm=24, dv=512,
            vdtype=CF.BF16), (40, 9)),
    # rank-2 Tucker + IVE + projection: fp16-plane scoring at 130 tokens, the expanded gather,
    # both GEMMs (the scratch holds the planes, the pooled rows and the intermediate)
    (_small("noalloc-projected", T=130, heads=2, dk=64, n_keys=96, topk=16, topm=24, dv=512,
            vdtype=CF.BF16, rank=2, grid=CF.GRID_TUCKER, expand=4, dv_virt=64, d_out=128), (130, 20)),
    # the 20.07M-slot decode layer
    (CF.C3, (32, 4)),
]


@pytest.mark.gpu
@pytest.mark.parametrize("cfg,sizes", CASES, ids=[c[0].name for c in CASES])
def test_noalloc_matches_forward(cfg, sizes):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from synth import device as SD
    log(f"[case] noalloc {cfg.name} T={sizes}")
    dl = SD.make_layer(cfg, batches=2)
    d = _desc(cfg)
    width = cfg.d_out if cfg.d_out else (cfg.dv_virt if cfg.dv_virt else cfg.dv)
    wshape = lambda T: (T, cfg.heads, cfg.topm) + ((cfg.cores,) if cfg.cores > 1 else ())
    for call, T in enumerate(sizes):
        b = call % 2
        st, nws = U.umem_workspace_size(d, T)
        U.check(st)
        assert nws <= U.UMEM_STATIC_SCRATCH_BYTES
        ws = torch.empty(max(nws, 256), dtype=torch.uint8, device="cuda")
        ref = [torch.empty((T, width), dtype=torch.float32, device="cuda"),
               torch.empty((T, cfg.heads, cfg.topm), dtype=torch.int32, device="cuda"),
               torch.empty(wshape(T), dtype=torch.float32, device="cuda")]
        got = [torch.full_like(ref[0], -7.0), torch.full_like(ref[1], -7), torch.full_like(ref[2], -7.0)]
        q_row, q_col = dl.q_row[b, :T].contiguous(), dl.q_col[b, :T].contiguous()
        U.check(U.umem_forward(d, T, q_row, q_col, dl.k_row, dl.k_col, dl.core, dl.values, dl.perm,
                               dl.w_proj, dl.w_out, ref[0], ref[1], ref[2], ws, ws.numel()),
                "umem_forward")
        torch.cuda.synchronize()
        free0 = torch.cuda.mem_get_info()[0]
        U.check(U.umem_forward_noalloc(d, T, q_row, q_col, dl.k_row, dl.k_col, dl.core, dl.values,
                                       dl.perm, dl.w_proj, dl.w_out, got[0], got[1], got[2]),
                "umem_forward_noalloc")
        torch.cuda.synchronize()
        free1 = torch.cuda.mem_get_info()[0]
        for a, x in zip(ref, got):
            assert torch.equal(a, x), (cfg.name, T)
        if call > 0:                      # the array was created with the first call's module load
            assert free1 == free0, (free0, free1)
        log(f"[report] noalloc {cfg.name} T={T}: identical to umem_forward; free memory "
            f"{free0} -> {free1}")
        del ws
