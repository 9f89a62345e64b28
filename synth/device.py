"""GPU copies of the seeded inputs (torch tensors), for the GPU tests and the benchmark.

Small tensors are drawn on the host with :mod:`synth` and uploaded; value tables are drawn on
the device by ``libumem_synth.so``, which computes the same bits (a GPU test checks sampled rows
against the host draw).
"""
from __future__ import annotations

import ctypes
import dataclasses
import math
import os
from typing import Optional

import numpy as np
import torch

import synth as S
from synth import configs as CF

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libumem_synth.so")
_lib = None


def _synth_lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise ImportError(f"{_LIB_PATH} is not built; run __graft_entry__.build() first")
        _lib = ctypes.CDLL(_LIB_PATH)
        _lib.synth_fill_normal.argtypes = [ctypes.c_uint64, ctypes.c_float, ctypes.c_uint64,
                                           ctypes.c_int64, ctypes.c_int, ctypes.c_void_p,
                                           ctypes.c_void_p]
        _lib.synth_fill_normal.restype = ctypes.c_int
    return _lib


def fill_normal_(t: torch.Tensor, seed: int, tensor_id: int, std: float, start: int = 0,
                 chunk: int = 1 << 28) -> torch.Tensor:
    """Fill a contiguous fp32 or bf16 GPU tensor with elements [start, start + numel) of the
    stream (seed, tensor_id)."""
    assert t.is_cuda and t.is_contiguous() and t.dtype in (torch.float32, torch.bfloat16)
    lib = _synth_lib()
    key = S.stream_key(seed, tensor_id)
    scale = float(S.normal_scale_f32(std))
    bf16 = int(t.dtype == torch.bfloat16)
    esize = t.element_size()
    stream = torch.cuda.current_stream().cuda_stream
    n = t.numel()
    for off in range(0, n, chunk):
        cnt = min(chunk, n - off)
        st = lib.synth_fill_normal(key, scale, start + off, cnt, bf16, t.data_ptr() + off * esize, stream)
        if st != 0:
            what = f"HIP error {-st - 1000}" if st <= -1000 else "invalid arguments"
            raise RuntimeError(f"synth_fill_normal failed: {what} (status {st})")
    return t


def _cuda(a: np.ndarray) -> torch.Tensor:
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


@dataclasses.dataclass
class DeviceLayer:
    cfg: CF.Layer
    q_row: torch.Tensor          # [R, T, H, Dk] fp32, R query batches
    q_col: torch.Tensor
    k_row: torch.Tensor          # [H, n, Dk] fp32
    k_col: torch.Tensor
    core: Optional[torch.Tensor]     # [H, r, r] fp32
    values: torch.Tensor             # [N_p, Dv] fp32 or bf16
    perm: Optional[torch.Tensor]     # [E * N_p] int32
    w_proj: Optional[torch.Tensor]   # [D'v, E * Dv] bf16 bits (int16), output-major
    w_out: Optional[torch.Tensor]    # [d_out, D'v] bf16 bits (int16), output-major

    @property
    def batches(self) -> int:
        return self.q_row.shape[0]


def make_layer(cfg: CF.Layer, batches: int = 1, values: Optional[torch.Tensor] = None) -> DeviceLayer:
    """All inputs of ``cfg`` on the GPU, with ``batches`` distinct query batches.  ``values`` may
    pass in an already drawn table of the same seed and shape."""
    qs = [CF.queries(cfg, batch=b) for b in range(batches)]
    q_row = _cuda(np.stack([q[0] for q in qs]))
    q_col = _cuda(np.stack([q[1] for q in qs]))
    kr, kc = CF.keys(cfg)
    core = CF.core(cfg)
    perm = CF.perm(cfg)
    wp, wo = CF.projections(cfg)
    vdt = torch.float32 if cfg.vdtype == CF.F32 else torch.bfloat16
    if values is None:
        values = torch.empty((cfg.n_values, cfg.dv), dtype=vdt, device="cuda")
        fill_normal_(values, cfg.seed, S.TID_VALUES, CF.value_std(cfg))
    assert values.shape == (cfg.n_values, cfg.dv) and values.dtype == vdt
    return DeviceLayer(cfg, q_row, q_col, _cuda(kr), _cuda(kc),
                       None if core is None else _cuda(core), values,
                       None if perm is None else _cuda(perm),
                       None if wp is None else _cuda(CF.output_major(wp)),
                       None if wo is None else _cuda(CF.output_major(wo)))


def value_bytes(cfg: CF.Layer) -> int:
    return cfg.n_values * cfg.dv * cfg.vbytes
