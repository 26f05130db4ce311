"""Oracle: symmetric INT8 checkpoint codec (test infrastructure only).

App. E.1, Eq. 10: for a state S in R^{L x H x dv x dk}, one scale per (l, h, k)
shared over dv:
    a_{l,h,k} = max_v |S_{l,h,v,k}|,   s_{l,h,k} = max(a, 1e-8) / 127,
    q = clip(round(S / s), -127, 127)   stored as int8, s stored in FP32,
and a hit dequantises once as S^ = q s.  The maximum, the division and the rounding
are FP32 (the paper says so), so this module computes in float32.

With the state stored transposed ([dk, dv], rows = key channels), the (l, h, k)
group is exactly one dv-row: one scale per row.  Reading where the paper is silent:
round() is round-half-to-even (the FP32 default).
"""

from __future__ import annotations

import numpy as np

F32 = np.float32


def quantize_rows(rows: np.ndarray):
    """rows [..., dv] float32 -> (q int8 [..., dv], s float32 [...])."""
    x = np.asarray(rows, dtype=F32)
    a = np.max(np.abs(x), axis=-1)
    s = np.maximum(a, F32(1e-8)) / F32(127.0)
    q = np.clip(np.rint(x / s[..., None]), F32(-127.0), F32(127.0)).astype(np.int8)
    return q, s.astype(F32)


def dequantize_rows(q: np.ndarray, s: np.ndarray) -> np.ndarray:
    """S^ = q s in FP32."""
    return (np.asarray(q, dtype=F32) * np.asarray(s, dtype=F32)[..., None]).astype(F32)


def pack_q8(states: np.ndarray, src_slot, unit_row: np.ndarray):
    """Pack then quantise: states [n_pool, rows, dv] f32 -> q [n, R, dv] int8, s [n, R] f32."""
    rows = np.stack([np.asarray(states[i], dtype=F32)[unit_row] for i in src_slot])
    return quantize_rows(rows)


def restore_q8(q: np.ndarray, s: np.ndarray, unit_row: np.ndarray, n_dense_rows: int) -> np.ndarray:
    """Dequantise into fresh dense states [n, rows, dv]; omitted rows are +0.0."""
    n, R, dv = q.shape
    out = np.zeros((n, n_dense_rows, dv), dtype=F32)
    out[:, unit_row, :] = dequantize_rows(q, s)
    return out
