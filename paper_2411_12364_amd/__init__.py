"""UltraMem memory-layer forward on AMD Instinct MI355X (gfx950).

A thin ctypes binding of ``libumem.so``, whose C ABI is declared in ``include/umem.h``.  Every
function here has the C function's name and arguments and only marshals them: device arrays may
be passed as torch tensors (contiguous, on the GPU) or as raw integer addresses, ``None`` is a
NULL pointer, and ``stream=None`` means torch's current stream.  Each returns the C status code;
:func:`check` turns a non-zero status into :class:`UmemError`.  All computation happens in the
library's HIP kernels; there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

# torch first: its HIP runtime (libamdhip64.so, SONAME libamdhip64.so.7) must be the one in the
# process before libumem.so is loaded, so that libumem.so binds to it.  Loaded the other way
# round, torch would bring in a second copy of the runtime, and the two would not share
# devices, streams or allocations.
import torch  # noqa: F401

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libumem.so")

UMEM_OK = 0
UMEM_ERR_INVALID_ARG = -1
UMEM_ERR_UNSUPPORTED = -2
UMEM_ERR_WORKSPACE = -3
UMEM_ERR_HIP = -4
UMEM_ERR_SCRATCH_LIMIT = -5
UMEM_STATIC_SCRATCH_BYTES = 64 << 20
UMEM_F32, UMEM_BF16 = 0, 1
UMEM_GRID_ADD, UMEM_GRID_TUCKER = 0, 1
UMEM_W_RAW, UMEM_W_SOFTMAX = 0, 1

EXPORTED = ("umem_workspace_size", "umem_axis_scores", "umem_select", "umem_score_topk",
            "umem_gather_sum", "umem_project_workspace_size", "umem_project", "umem_forward",
            "umem_forward_noalloc",
            "umem_query_workspace_size", "umem_query", "umem_key_norm",
            "umem_gather_backward_workspace_size", "umem_gather_backward", "umem_gather_backward_rows",
            "umem_score_backward_workspace_size", "umem_score_backward", "umem_status_string")


class umem_desc(ctypes.Structure):
    _fields_ = [
        ("heads", ctypes.c_int32), ("dk", ctypes.c_int32), ("n_keys", ctypes.c_int32),
        ("rank", ctypes.c_int32), ("topk", ctypes.c_int32), ("topm", ctypes.c_int32),
        ("grid", ctypes.c_int32), ("weight", ctypes.c_int32), ("n_values", ctypes.c_int64),
        ("dv", ctypes.c_int32), ("vdtype", ctypes.c_int32), ("expand", ctypes.c_int32),
        ("dv_virt", ctypes.c_int32), ("d_out", ctypes.c_int32), ("cores", ctypes.c_int32),
    ]


class umem_query_desc(ctypes.Structure):
    _fields_ = [
        ("d_model", ctypes.c_int32), ("conv_k", ctypes.c_int32), ("heads", ctypes.c_int32),
        ("dk", ctypes.c_int32), ("shared", ctypes.c_int32), ("eps", ctypes.c_float),
    ]


class UmemError(RuntimeError):
    def __init__(self, status: int, what: str = ""):
        self.status = status
        super().__init__(f"{what}: {umem_status_string(status)} ({status})")


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() first")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    D = ctypes.POINTER(umem_desc)
    sig = {
        "umem_workspace_size": [D, I32, ctypes.POINTER(SZ)],
        "umem_axis_scores": [D, I32, P, P, P, P, P, P, P, SZ, P],
        "umem_select": [D, I32, P, P, P, P, P, P, P, P, P, P, P, P],
        "umem_score_topk": [D, I32, P, P, P, P, P, P, P, P, P, SZ, P],
        "umem_gather_sum": [I64, I32, I32, P, I32, I32, P, P, P, I32, I32, P, P],
        "umem_project_workspace_size": [I32, I32, I32, I32, I32, ctypes.POINTER(SZ)],
        "umem_project": [I32, I32, I32, I32, I32, P, P, P, P, P, SZ, P],
        "umem_forward": [D, I32, P, P, P, P, P, P, P, P, P, P, P, P, P, SZ, P],
        "umem_forward_noalloc": [D, I32, P, P, P, P, P, P, P, P, P, P, P, P, P],
        "umem_query_workspace_size": [ctypes.POINTER(umem_query_desc), I32, I32, ctypes.POINTER(SZ)],
        "umem_query": [ctypes.POINTER(umem_query_desc), I32, I32, P, P, P, P, P, P, P, P, P, SZ, P],
        "umem_key_norm": [I32, I32, I32, P, P, P, ctypes.c_float, P, P],
        "umem_gather_backward_workspace_size": [I32, I32, I32, ctypes.POINTER(SZ)],
        "umem_gather_backward": [I64, I32, I32, P, I32, I32, P, P, P, I32, I32, P, P, P, P, SZ, P],
        "umem_gather_backward_rows": [I64, I32, I32, P, I32, I32, P, P, P, I32, I32, P, P, P, P, P, P,
                                      SZ, P],
        "umem_score_backward_workspace_size": [D, I32, ctypes.POINTER(SZ)],
        "umem_score_backward": [D, I32, P, P, P, P, P, P, P, P, P, P, P, P, P, P, SZ, P],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    lib.umem_status_string.argtypes = [ctypes.c_int]
    lib.umem_status_string.restype = ctypes.c_char_p
    return lib


_lib = _load()


def _p(x):
    """A device address: None -> NULL, int -> itself, torch tensor -> data_ptr()."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if not x.is_contiguous():
        raise ValueError("tensor arguments must be contiguous")
    if x.device.type != "cuda":
        raise ValueError("tensor arguments must live on the GPU")
    return x.data_ptr()


def _s(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _d(desc):
    return ctypes.byref(desc)


def umem_status_string(status: int) -> str:
    return _lib.umem_status_string(status).decode()


def check(status: int, what: str = "umem") -> None:
    if status != UMEM_OK:
        raise UmemError(status, what)


def umem_workspace_size(desc: umem_desc, T: int):
    """Returns (status, bytes)."""
    out = ctypes.c_size_t(0)
    st = _lib.umem_workspace_size(_d(desc), T, ctypes.byref(out))
    return st, out.value


def umem_axis_scores(desc, T, q_row, q_col, k_row, k_col, core, sel, ws=None, ws_bytes=0,
                     stream=None) -> int:
    return _lib.umem_axis_scores(_d(desc), T, _p(q_row), _p(q_col), _p(k_row), _p(k_col), _p(core),
                                 _p(sel), _p(ws), ws_bytes, _s(stream))


def umem_select(desc, T, sel, q_row, q_col, k_row, k_col, core, idx, w, axis_idx=None,
                values=None, pooled=None, stream=None) -> int:
    return _lib.umem_select(_d(desc), T, _p(sel), _p(q_row), _p(q_col), _p(k_row), _p(k_col),
                            _p(core), _p(idx), _p(w), _p(axis_idx), _p(values), _p(pooled),
                            _s(stream))


def umem_score_topk(desc, T, q_row, q_col, k_row, k_col, core, idx, w, axis_idx, ws, ws_bytes,
                    stream=None) -> int:
    return _lib.umem_score_topk(_d(desc), T, _p(q_row), _p(q_col), _p(k_row), _p(k_col), _p(core),
                                _p(idx), _p(w), _p(axis_idx), _p(ws), ws_bytes, _s(stream))


def umem_gather_sum(n_values, dv, vdtype, values, T, bag, idx, w, perm, expand, cores, out,
                    stream=None) -> int:
    return _lib.umem_gather_sum(n_values, dv, vdtype, _p(values), T, bag, _p(idx), _p(w), _p(perm),
                                expand, cores, _p(out), _s(stream))


def umem_project_workspace_size(T, expand, dv, dv_virt, d_out):
    """Returns (status, bytes)."""
    out = ctypes.c_size_t(0)
    st = _lib.umem_project_workspace_size(T, expand, dv, dv_virt, d_out, ctypes.byref(out))
    return st, out.value


def umem_project(T, expand, dv, dv_virt, d_out, pooled, w_proj, w_out, out, ws, ws_bytes,
                 stream=None) -> int:
    return _lib.umem_project(T, expand, dv, dv_virt, d_out, _p(pooled), _p(w_proj), _p(w_out),
                             _p(out), _p(ws), ws_bytes, _s(stream))


def umem_forward(desc, T, q_row, q_col, k_row, k_col, core, values, perm, w_proj, w_out, out,
                 idx_out, w_out_scores, ws, ws_bytes, stream=None) -> int:
    return _lib.umem_forward(_d(desc), T, _p(q_row), _p(q_col), _p(k_row), _p(k_col), _p(core),
                             _p(values), _p(perm), _p(w_proj), _p(w_out), _p(out), _p(idx_out),
                             _p(w_out_scores), _p(ws), ws_bytes, _s(stream))


def umem_forward_noalloc(desc, T, q_row, q_col, k_row, k_col, core, values, perm, w_proj, w_out,
                         out, idx_out, w_out_scores, stream=None) -> int:
    return _lib.umem_forward_noalloc(_d(desc), T, _p(q_row), _p(q_col), _p(k_row), _p(k_col),
                                     _p(core), _p(values), _p(perm), _p(w_proj), _p(w_out), _p(out),
                                     _p(idx_out), _p(w_out_scores), _s(stream))


def umem_query_workspace_size(qd, B, L):
    """Returns (status, bytes)."""
    out = ctypes.c_size_t(0)
    st = _lib.umem_query_workspace_size(ctypes.byref(qd), B, L, ctypes.byref(out))
    return st, out.value


def umem_query(qd, B, L, x, x_hist, conv_w, w_q, gamma, beta, q_row, q_col, ws, ws_bytes,
               stream=None) -> int:
    return _lib.umem_query(ctypes.byref(qd), B, L, _p(x), _p(x_hist), _p(conv_w), _p(w_q),
                           _p(gamma), _p(beta), _p(q_row), _p(q_col), _p(ws), ws_bytes, _s(stream))


def umem_key_norm(heads, n, dk, keys, gamma, beta, eps, out, stream=None) -> int:
    return _lib.umem_key_norm(heads, n, dk, _p(keys), _p(gamma), _p(beta), eps, _p(out), _s(stream))


def umem_gather_backward_workspace_size(T, bag, dv):
    """Returns (status, bytes)."""
    out = ctypes.c_size_t(0)
    st = _lib.umem_gather_backward_workspace_size(T, bag, dv, ctypes.byref(out))
    return st, out.value


def umem_gather_backward(n_values, dv, vdtype, values, T, bag, idx, w, perm, expand, cores,
                         d_pooled, d_values, dw, ws, ws_bytes, stream=None) -> int:
    return _lib.umem_gather_backward(n_values, dv, vdtype, _p(values), T, bag, _p(idx), _p(w),
                                     _p(perm), expand, cores, _p(d_pooled), _p(d_values), _p(dw),
                                     _p(ws), ws_bytes, _s(stream))


def umem_gather_backward_rows(n_values, dv, vdtype, values, T, bag, idx, w, perm, expand, cores,
                              d_pooled, rows, d_rows, n_rows, dw, ws, ws_bytes, stream=None) -> int:
    return _lib.umem_gather_backward_rows(n_values, dv, vdtype, _p(values), T, bag, _p(idx), _p(w),
                                          _p(perm), expand, cores, _p(d_pooled), _p(rows),
                                          _p(d_rows), _p(n_rows), _p(dw), _p(ws), ws_bytes,
                                          _s(stream))


def umem_score_backward_workspace_size(desc, T):
    """Returns (status, bytes)."""
    out = ctypes.c_size_t(0)
    st = _lib.umem_score_backward_workspace_size(_d(desc), T, ctypes.byref(out))
    return st, out.value


def umem_score_backward(desc, T, q_row, q_col, k_row, k_col, core, idx, w, dw, dq_row, dq_col,
                        dk_row, dk_col, dcore, ws, ws_bytes, stream=None) -> int:
    return _lib.umem_score_backward(_d(desc), T, _p(q_row), _p(q_col), _p(k_row), _p(k_col),
                                    _p(core), _p(idx), _p(w), _p(dw), _p(dq_row), _p(dq_col),
                                    _p(dk_row), _p(dk_col), _p(dcore), _p(ws), ws_bytes, _s(stream))
