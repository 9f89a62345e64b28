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


@pytest.mark.gpu
@pytest.mark.parametrize("i", range(N_CASES))
def test_random_layer(i):
    from tests.test_gpu_parity import run_and_check
    cfg = random_layer(i)
    run_and_check(cfg, tokens=None if cfg.T <= 64 else np.arange(0, cfg.T, 5))
