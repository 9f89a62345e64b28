"""Seeded synthetic inputs for the UltraMem memory-layer forward.

Every number drawn here is a pure function of (seed, tensor_id, element index), so any slice of
any tensor -- one row of a 20M-row value table, one token's query -- can be regenerated on its
own, on the host or on the device, with identical bits.  This module draws numbers and holds
none of the memory layer's arithmetic; both the CPU oracle and the GPU path take their inputs
from it.

Generator (counter-based, integer-only, so host and device agree bit for bit):

* ``splitmix64`` (S. Vigna's published SplitMix64): output ``e`` (0-based) of the sequence
  with state ``s`` is ``fmix(s + (e + 1) * GAMMA)`` mod 2**64, with the published finaliser
  ``fmix``.
* The state of tensor (seed, tensor_id) is ``fmix(((seed << 32) | tensor_id) + GAMMA)``.
* A "normal" draw is an Irwin-Hall(4) variate: the four 16-bit fields of one 64-bit output are
  summed and centred, ``c = u0 + u1 + u2 + u3 - 131070`` (an exact integer, |c| < 2**18), then
  scaled by the fp32 constant ``sqrt(3) / 65536 * std`` in one correctly rounded fp32 multiply.
  It has mean 0 and variance ``std**2`` (to 1 part in 2**32), is bell shaped and bounded by
  +-3.46 std.  A true Gaussian needs ``log``/``cos``, whose last bits differ between host and
  device libraries; this draw needs none.
* bf16 tensors are the fp32 draw rounded to nearest even.
"""
from __future__ import annotations

import math

import numpy as np

GAMMA = 0x9E3779B97F4A7C15
_M1 = 0xBF58476D1CE4E5B9
_M2 = 0x94D049BB133111EB
_MASK64 = (1 << 64) - 1

# Tensor ids.  A query batch b of a rotating set uses tensor_id = base + (b << 8).
TID_Q_ROW = 1
TID_Q_COL = 2
TID_K_ROW = 3
TID_K_COL = 4
TID_CORE = 5
TID_VALUES = 6
TID_PERM = 7
TID_W_PROJ = 8
TID_W_OUT = 9
TID_CENTRES_ROW = 10
TID_CENTRES_COL = 11
TID_EPS_ROW = 12
TID_EPS_COL = 13
TID_CLUSTER = 14
TID_HIDDEN = 15
TID_HIST = 16
TID_CONV_W = 17
TID_W_Q = 18
TID_Q_GAMMA = 19
TID_Q_BETA = 20
TID_K_GAMMA = 21
TID_K_BETA = 22


def _fmix_int(z: int) -> int:
    z &= _MASK64
    z = ((z ^ (z >> 30)) * _M1) & _MASK64
    z = ((z ^ (z >> 27)) * _M2) & _MASK64
    return z ^ (z >> 31)


def _fmix(z: np.ndarray) -> np.ndarray:
    """SplitMix64 finaliser on a uint64 array (numpy array arithmetic wraps mod 2**64)."""
    z = (z ^ (z >> np.uint64(30))) * np.uint64(_M1)
    z = (z ^ (z >> np.uint64(27))) * np.uint64(_M2)
    return z ^ (z >> np.uint64(31))


def stream_key(seed: int, tensor_id: int) -> int:
    """State of the SplitMix64 stream that tensor (seed, tensor_id) is drawn from."""
    return _fmix_int((((seed & 0xFFFFFFFF) << 32) | (tensor_id & 0xFFFFFFFF)) + GAMMA)


def raw64(key: int, elems: np.ndarray) -> np.ndarray:
    """64-bit outputs number ``elems`` (any integer array) of the stream with state ``key``."""
    e = np.asarray(elems, dtype=np.uint64)
    return _fmix(np.uint64(key) + (e + np.uint64(1)) * np.uint64(GAMMA))


def normal_scale_f32(std: float) -> np.float32:
    """The fp32 multiplier that turns a centred Irwin-Hall(4) integer into a draw of this std."""
    return np.float32(math.sqrt(3.0) / 65536.0 * std)


def irwin_hall_int(z: np.ndarray) -> np.ndarray:
    """Centred sum of the four 16-bit fields of each 64-bit word, as int64."""
    m = np.uint64(0xFFFF)
    s = (z & m) + ((z >> np.uint64(16)) & m) + ((z >> np.uint64(32)) & m) + (z >> np.uint64(48))
    return s.astype(np.int64) - 131070


def normal_f32(key: int, elems: np.ndarray, std: float) -> np.ndarray:
    """fp32 draws (mean 0, standard deviation ``std``) at element indices ``elems``."""
    c = irwin_hall_int(raw64(key, elems))
    return c.astype(np.float32) * normal_scale_f32(std)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16, nearest even; returns the uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = (u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def tensor_f32(seed: int, tensor_id: int, shape, std: float) -> np.ndarray:
    """A whole fp32 tensor, element index = row-major linear index."""
    count = int(np.prod(shape))
    return normal_f32(stream_key(seed, tensor_id), np.arange(count, dtype=np.uint64), std).reshape(shape)


def rows_f32(seed: int, tensor_id: int, rows: np.ndarray, width: int, std: float) -> np.ndarray:
    """Rows ``rows`` of a row-major [*, width] fp32 tensor, regenerated on their own."""
    rows = np.asarray(rows, dtype=np.uint64).reshape(-1)
    elems = rows[:, None] * np.uint64(width) + np.arange(width, dtype=np.uint64)[None, :]
    return normal_f32(stream_key(seed, tensor_id), elems.reshape(-1), std).reshape(len(rows), width)


def rows_bf16_bits(seed: int, tensor_id: int, rows: np.ndarray, width: int, std: float) -> np.ndarray:
    return f32_to_bf16_bits(rows_f32(seed, tensor_id, rows, width, std)).reshape(-1, width)


def permutation(seed: int, tensor_id: int, size: int) -> np.ndarray:
    """A uniform random permutation of [0, size): the order that sorts one 64-bit draw per slot
    (equal draws, which have probability ~size**2 / 2**65, keep index order)."""
    z = raw64(stream_key(seed, tensor_id), np.arange(size, dtype=np.uint64))
    return np.argsort(z, kind="stable").astype(np.int32)


def uniform_int(seed: int, tensor_id: int, count: int, modulus: int) -> np.ndarray:
    """``count`` draws in [0, modulus) (64-bit output mod modulus)."""
    z = raw64(stream_key(seed, tensor_id), np.arange(count, dtype=np.uint64))
    return (z % np.uint64(modulus)).astype(np.int64)
