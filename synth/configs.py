"""Workload shapes and the seeded recipe for every input tensor of the memory layer.

Shapes follow the paper's scale (Sec. 1 and Table 5: about 20M slots; Trick 6 of Sec. 3.2: value
dim half the model width; Fig. 1: decode with one token per sequence).  Every tensor is drawn
with :mod:`synth` from (seed, tensor_id), i.i.d. with mean 0 and std 1/sqrt(dim) (dim = the
contraction length it enters), except the Tucker core, which has std 1.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np

import synth as S

GRID_ADD = 0
GRID_TUCKER = 1
W_RAW = 0
W_SOFTMAX = 1
F32 = 0
BF16 = 1


@dataclasses.dataclass(frozen=True)
class Layer:
    name: str
    T: int            # tokens in one batch
    heads: int        # H key sets sharing one value table
    dk: int           # query / key dim per axis per head
    n_keys: int       # keys per axis, n; logical slots N = n * n
    topk: int         # per-axis top-k
    topm: int         # global top-m per head
    dv: int           # physical value dim
    vdtype: int       # F32 or BF16 value table
    seed: int
    rank: int = 1                 # Tucker rank r (1 with GRID_ADD)
    grid: int = GRID_ADD
    weight: int = W_RAW
    expand: int = 1               # IVE expansion E (a perfect square)
    dv_virt: int = 0              # D'v of the IVE projectors (0: no projection)
    d_out: int = 0                # output linear width (0: none)
    queries: str = "gauss"        # "gauss" or "clusters"
    n_clusters: int = 8
    cluster_spread: float = 0.1
    cores: int = 1                # multi-core scoring h (component cores per head; Tucker only)

    @property
    def n_slots(self) -> int:
        return self.n_keys * self.n_keys

    @property
    def n_values(self) -> int:
        """Physical rows N_p = N / E."""
        assert self.n_slots % self.expand == 0
        return self.n_slots // self.expand

    @property
    def bag(self) -> int:
        return self.heads * self.topm

    @property
    def vbytes(self) -> int:
        return 4 if self.vdtype == F32 else 2

    def with_tokens(self, T: int) -> "Layer":
        return dataclasses.replace(self, T=T, name=f"{self.name}-T{T}")


C1 = Layer("tiny-pkm-4096", T=8, heads=1, dk=64, n_keys=64, topk=8, topm=8, dv=256, vdtype=F32, seed=0)
C2 = Layer("prefill-1M", T=2048, heads=2, dk=128, n_keys=1024, topk=32, topm=32, dv=1024,
           vdtype=BF16, seed=1)
C3 = Layer("decode-20M", T=32, heads=2, dk=128, n_keys=4480, topk=32, topm=32, dv=512,
           vdtype=BF16, seed=2)
C4_BATCHES = (1, 4, 16, 64, 256, 1024)
C5 = Layer("tucker-ive-4M", T=4096, heads=4, dk=128, n_keys=2048, topk=64, topm=64, dv=512,
           vdtype=BF16, seed=3, rank=2, grid=GRID_TUCKER, expand=4, dv_virt=512, d_out=2048,
           queries="clusters")

# One memory layer of the paper's UltraMem-1.6B-x12 model (its model table: Kdim 448, Knum 1792,
# top-m 42 x 2 heads; common configuration r = 2, h = 2, E = 4) at the decode batch of 512 tokens
# the paper times inference with.  Knum^2 counts the virtual slots, so N_p = 1792^2 / 4 physical
# rows; Dv = 4096 puts the six layers' tables at the model's ~19.7 B sparse parameters, and
# D'v = 1024 is half the 2048 hidden width (the halved value dimension), projected back to 2048.
C6 = Layer("ultramem-1.6B-x12", T=512, heads=2, dk=448, n_keys=1792, topk=42, topm=42, dv=4096,
           vdtype=BF16, seed=6, rank=2, grid=GRID_TUCKER, expand=4, dv_virt=1024, d_out=2048,
           cores=2)

CONFIGS = {c.name: c for c in (C1, C2, C3, C5, C6)}


@dataclasses.dataclass(frozen=True)
class FrontEnd:
    """The query front-end of a layer: B sequences of L tokens of d_model-wide hidden states."""
    name: str
    B: int
    L: int
    d_model: int
    conv_k: int        # causal depthwise convolution taps
    heads: int
    dk: int
    shared: bool       # one query for both key sets
    seed: int
    history: bool = True   # hidden states before each sequence's first token (else a start)
    eps: float = 1e-5

    @property
    def T(self) -> int:
        return self.B * self.L

    @property
    def n_queries(self) -> int:
        return (1 if self.shared else 2) * self.heads * self.dk


# The front-end of the UltraMem-1.6B-x12 layer above at its 512-token decode batch: one new token
# per sequence, the three before it as the convolution's history; hidden width 2048; K_c = 4.
FE6 = FrontEnd("ultramem-1.6B-x12-query", B=512, L=1, d_model=2048, conv_k=4, heads=2, dk=448,
               shared=True, seed=6)


def front_end_inputs(fe: FrontEnd) -> dict:
    """x fp32 [B, L, d]; hist fp32 [B, K_c - 1, d] or None; conv_w fp32 [K_c, d];
    w_q bf16 bits [d, A H Dk]; gamma, beta fp32 [A, H, Dk] (A = 1 shared, else 2)."""
    A = 1 if fe.shared else 2
    x = S.tensor_f32(fe.seed, S.TID_HIDDEN, (fe.B, fe.L, fe.d_model), 1.0)
    hist = (S.tensor_f32(fe.seed, S.TID_HIST, (fe.B, fe.conv_k - 1, fe.d_model), 1.0)
            if fe.history and fe.conv_k > 1 else None)
    conv_w = S.tensor_f32(fe.seed, S.TID_CONV_W, (fe.conv_k, fe.d_model), 1.0 / math.sqrt(fe.conv_k))
    wq = S.tensor_f32(fe.seed, S.TID_W_Q, (fe.d_model, fe.n_queries), 1.0 / math.sqrt(fe.d_model))
    gamma = (np.float32(1.0) + S.tensor_f32(fe.seed, S.TID_Q_GAMMA, (A, fe.heads, fe.dk), 0.1)).astype(np.float32)
    beta = S.tensor_f32(fe.seed, S.TID_Q_BETA, (A, fe.heads, fe.dk), 0.05)
    return dict(x=x, hist=hist, conv_w=conv_w, w_q=S.f32_to_bf16_bits(wq).reshape(wq.shape),
                gamma=gamma, beta=beta)


def key_norm_params(cfg: Layer):
    """gamma, beta fp32 [H, Dk] of the key LayerNorm (the appendix initialises gamma to
    1/sqrt(Dk); a spread around that)."""
    g = S.tensor_f32(cfg.seed, S.TID_K_GAMMA, (cfg.heads, cfg.dk), 0.1 / math.sqrt(cfg.dk))
    b = S.tensor_f32(cfg.seed, S.TID_K_BETA, (cfg.heads, cfg.dk), 0.01 / math.sqrt(cfg.dk))
    return (np.float32(1.0 / math.sqrt(cfg.dk)) + g).astype(np.float32), b


def _tid(base: int, batch: int) -> int:
    return base + (batch << 8)


def queries(cfg: Layer, batch: int = 0, tokens: Optional[np.ndarray] = None):
    """q_row, q_col as fp32 [T, H, Dk] for query batch ``batch`` (rows ``tokens`` only if given).

    "gauss": i.i.d. draws of std 1/sqrt(Dk).  "clusters": token t belongs to cluster
    z_t = draw(t) mod n_clusters; q = centre[z_t] + spread * eps with centres and eps both of
    std 1/sqrt(Dk) (a mixture of Gaussian-like clusters).
    """
    width = cfg.heads * cfg.dk
    std = 1.0 / math.sqrt(cfg.dk)
    t_idx = np.arange(cfg.T) if tokens is None else np.asarray(tokens)
    out = []
    for base, cbase, ebase in ((S.TID_Q_ROW, S.TID_CENTRES_ROW, S.TID_EPS_ROW),
                               (S.TID_Q_COL, S.TID_CENTRES_COL, S.TID_EPS_COL)):
        if cfg.queries == "gauss":
            q = S.rows_f32(cfg.seed, _tid(base, batch), t_idx, width, std)
        else:
            z = S.uniform_int(cfg.seed, _tid(S.TID_CLUSTER, batch), cfg.T, cfg.n_clusters)[t_idx]
            centres = S.rows_f32(cfg.seed, cbase, np.arange(cfg.n_clusters), width, std)
            eps = S.rows_f32(cfg.seed, _tid(ebase, batch), t_idx, width, std)
            q = centres[z] + np.float32(cfg.cluster_spread) * eps
        out.append(np.ascontiguousarray(q.reshape(len(t_idx), cfg.heads, cfg.dk), dtype=np.float32))
    return out[0], out[1]


def keys(cfg: Layer):
    """K_row, K_col as fp32 [H, n, Dk]; with rank r the Dk axis holds r contiguous slices."""
    std = 1.0 / math.sqrt(cfg.dk)
    shape = (cfg.heads, cfg.n_keys, cfg.dk)
    return (S.tensor_f32(cfg.seed, S.TID_K_ROW, shape, std),
            S.tensor_f32(cfg.seed, S.TID_K_COL, shape, std))


def core(cfg: Layer) -> Optional[np.ndarray]:
    """Tucker cores C_h as fp32 [H, r, r] (std 1), or None for the additive grid; with
    multi-core scoring the component cores [H, h, r, r] (each std 1; their sum is the core)."""
    if cfg.grid != GRID_TUCKER:
        return None
    if cfg.cores > 1:
        return S.tensor_f32(cfg.seed, S.TID_CORE, (cfg.heads, cfg.cores, cfg.rank, cfg.rank), 1.0)
    return S.tensor_f32(cfg.seed, S.TID_CORE, (cfg.heads, cfg.rank, cfg.rank), 1.0)


def perm(cfg: Layer) -> Optional[np.ndarray]:
    """The virtual-slot shuffle of implicit value expansion, int32 [E * N_p], or None."""
    if cfg.expand == 1:
        return None
    return S.permutation(cfg.seed, S.TID_PERM, cfg.n_slots)


def value_std(cfg: Layer) -> float:
    return 1.0 / math.sqrt(cfg.dv)


def value_key(cfg: Layer) -> int:
    return S.stream_key(cfg.seed, S.TID_VALUES)


def value_rows_f32(cfg: Layer, rows: np.ndarray) -> np.ndarray:
    """Rows of the value table as stored (bf16 tables widened exactly), fp32 [len(rows), Dv]."""
    x = S.rows_f32(cfg.seed, S.TID_VALUES, rows, cfg.dv, value_std(cfg))
    if cfg.vdtype == BF16:
        x = S.bf16_bits_to_f32(S.f32_to_bf16_bits(x)).reshape(x.shape)
    return x


def value_table_host(cfg: Layer) -> np.ndarray:
    """The whole value table in its storage type (fp32, or bf16 bits as uint16).  Small only."""
    x = S.tensor_f32(cfg.seed, S.TID_VALUES, (cfg.n_values, cfg.dv), value_std(cfg))
    return x if cfg.vdtype == F32 else S.f32_to_bf16_bits(x).reshape(x.shape)


def output_major(w: np.ndarray) -> np.ndarray:
    """A weight drawn as [..., in, out] (the paper's W in x W) in the output-major layout of a linear
    layer's weight, [out, in] with the leading axes folded into in: the layout the GPU takes."""
    return np.ascontiguousarray(w.reshape(-1, w.shape[-1]).T)


def projections(cfg: Layer):
    """IVE projectors W_p as bf16 bits [E, Dv, D'v] and output linear bf16 bits [D'v, d_out]; a
    layer with the output linear alone (D'v = 0) has no W_p and W_out [Dv, d_out]."""
    if cfg.dv_virt == 0:
        if cfg.d_out == 0:
            return None, None
        wo = S.tensor_f32(cfg.seed, S.TID_W_OUT, (cfg.dv, cfg.d_out), 1.0 / math.sqrt(cfg.dv))
        return None, S.f32_to_bf16_bits(wo).reshape(wo.shape)
    wp = S.tensor_f32(cfg.seed, S.TID_W_PROJ, (cfg.expand, cfg.dv, cfg.dv_virt), 1.0 / math.sqrt(cfg.dv))
    wp = S.f32_to_bf16_bits(wp).reshape(wp.shape)
    if cfg.d_out == 0:       # the projectors alone
        return wp, None
    wo = S.tensor_f32(cfg.seed, S.TID_W_OUT, (cfg.dv_virt, cfg.d_out), 1.0 / math.sqrt(cfg.dv_virt))
    return wp, S.f32_to_bf16_bits(wo).reshape(wo.shape)
