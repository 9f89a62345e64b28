"""Helpers for the GPU tests: descriptors and calls through the C ABI on torch tensors."""
from __future__ import annotations

import numpy as np
import torch

import paper_2411_12364_amd as U
from synth import configs as CF


def desc_for(cfg: CF.Layer) -> U.umem_desc:
    d = U.umem_desc()
    d.heads, d.dk, d.n_keys, d.rank = cfg.heads, cfg.dk, cfg.n_keys, cfg.rank
    d.topk, d.topm, d.grid, d.weight = cfg.topk, cfg.topm, cfg.grid, cfg.weight
    d.n_values, d.dv, d.vdtype, d.expand = cfg.n_values, cfg.dv, cfg.vdtype, cfg.expand
    d.dv_virt, d.d_out, d.cores = cfg.dv_virt, cfg.d_out, cfg.cores
    return d


def weights_shape(cfg: CF.Layer, T: int):
    """[T, H, m], or [T, H, m, h] with multi-core scoring."""
    return (T, cfg.heads, cfg.topm) + ((cfg.cores,) if cfg.cores > 1 else ())


def workspace(desc, T) -> torch.Tensor:
    st, nbytes = U.umem_workspace_size(desc, T)
    U.check(st, "umem_workspace_size")
    return torch.empty(max(nbytes, 256), dtype=torch.uint8, device="cuda")


def score_topk(dl, T, batch=0, with_axis=True):
    cfg = dl.cfg
    desc = desc_for(cfg)
    idx = torch.empty((T, cfg.heads, cfg.topm), dtype=torch.int32, device="cuda")
    w = torch.empty(weights_shape(cfg, T), dtype=torch.float32, device="cuda")
    ax = torch.empty((2, T, cfg.heads, cfg.topk), dtype=torch.int32, device="cuda") if with_axis else None
    ws = workspace(desc, T)
    U.check(U.umem_score_topk(desc, T, dl.q_row[batch, :T], dl.q_col[batch, :T], dl.k_row, dl.k_col,
                              dl.core, idx, w, ax, ws, ws.numel()), "umem_score_topk")
    return idx, w, ax


def gather(dl, idx, w, T):
    cfg = dl.cfg
    out = torch.empty((T, cfg.expand, cfg.dv), dtype=torch.float32, device="cuda")
    U.check(U.umem_gather_sum(cfg.n_values, cfg.dv, cfg.vdtype, dl.values, T, cfg.bag, idx, w,
                              dl.perm, cfg.expand, cfg.cores, out), "umem_gather_sum")
    return out


def forward(dl, T, batch=0):
    cfg = dl.cfg
    desc = desc_for(cfg)
    width = cfg.d_out if cfg.d_out else (cfg.dv_virt if cfg.dv_virt else cfg.dv)
    out = torch.empty((T, width), dtype=torch.float32, device="cuda")
    idx = torch.empty((T, cfg.heads, cfg.topm), dtype=torch.int32, device="cuda")
    w = torch.empty(weights_shape(cfg, T), dtype=torch.float32, device="cuda")
    ws = workspace(desc, T)
    U.check(U.umem_forward(desc, T, dl.q_row[batch, :T], dl.q_col[batch, :T], dl.k_row, dl.k_col,
                           dl.core, dl.values, dl.perm, dl.w_proj, dl.w_out, out, idx, w, ws,
                           ws.numel()), "umem_forward")
    return out, idx, w


def host(x):
    return None if x is None else x.detach().cpu().numpy()


def value_rows_fn(cfg):
    """Rows of the value table as the oracle sees them, regenerated on the host."""
    return lambda rows: CF.value_rows_f32(cfg, np.asarray(rows))
