"""Python binding of the DASC C ABI (argument marshalling only).

Each function has the name of the C entry point it calls and does nothing but
turn Python/NumPy/torch arguments into pointers and sizes: every step of the
path runs in libdasc.so.  torch tensors supply device memory and the current
HIP stream; host arrays for the planner are NumPy.

Errors from the library raise DascError carrying the status code.
"""

from __future__ import annotations

import ctypes as C
from dataclasses import dataclass

import numpy as np

from . import _lib
from ._lib import LIB

ARCH = {"kda": _lib.DASC_ARCH_KDA, "gdn": _lib.DASC_ARCH_GDN}
KEEP = {"threshold": _lib.DASC_KEEP_THRESHOLD, "topk_head": _lib.DASC_KEEP_TOPK_PER_HEAD,
        "topk_layer": _lib.DASC_KEEP_TOPK_PER_LAYER}
INIT = {"restored": _lib.DASC_INIT_RESTORED, "zero": _lib.DASC_INIT_ZERO}


class DascError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__(f"{where}: {LIB.dasc_strerror(code).decode()} (status {code})")


def _check(code: int, where: str) -> None:
    if code != _lib.DASC_OK:
        raise DascError(code, where)


@dataclass(frozen=True)
class Shape:
    arch: str
    n_layers: int
    n_heads: int
    n_qk_heads: int
    dk: int
    dv: int

    def c(self) -> _lib.Shape:
        return _lib.Shape(ARCH[self.arch], self.n_layers, self.n_heads, self.n_qk_heads,
                          self.dk, self.dv)

    @property
    def rows(self) -> int:
        return self.n_layers * self.n_heads * self.dk

    @property
    def units(self) -> int:
        return self.rows if self.arch == "kda" else self.n_layers * self.n_heads


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


# ---- plan (host) ---------------------------------------------------------------

def dasc_static_log_decay(a_log, dt_bias=None, a: float = -0.3) -> np.ndarray:
    a_log = np.ascontiguousarray(a_log, dtype=np.float64)
    out = np.empty_like(a_log)
    dt = None if dt_bias is None else np.ascontiguousarray(
        np.broadcast_to(dt_bias, a_log.shape), dtype=np.float64)
    _check(LIB.dasc_static_log_decay(_ptr(a_log), None if dt is None else _ptr(dt), a,
                                     a_log.size, _ptr(out)), "dasc_static_log_decay")
    return out


def dasc_plan(shape: Shape, g_static, keep_mode: str = "threshold", keep_k: int = 0,
              w_max: int = 16, n_ranks: int = 1, eps: float = 1e-3, conv_bytes: int = 0) -> dict:
    """Host planner; returns a dict of NumPy arrays and scalars (see dasc.h)."""
    g = np.ascontiguousarray(g_static, dtype=np.float64)
    desc = _lib.PlanDesc(shape.c(), KEEP[keep_mode], keep_k, w_max, n_ranks, eps, conv_bytes)
    L, H, nu, rows, T = shape.n_layers, shape.n_heads, shape.units, shape.rows, n_ranks
    arr = {
        "keep": np.zeros(nu, np.uint8), "horizon": np.zeros(nu, np.float64),
        "unit_count": np.zeros(L * H, np.int32), "off": np.zeros(L * H + 1, np.int32),
        "layer_off": np.zeros(L + 1, np.int32), "layer_off_rows": np.zeros(L + 1, np.int32),
        "unit_row": np.zeros(rows, np.int32),
        "inv_row": np.zeros(rows, np.int32), "w_units": np.zeros(nu, np.int32),
        "rank_begin": np.zeros(T + 1, np.int32), "send": np.zeros(T * T, np.int64),
    }
    out = _lib.PlanOut()
    for name, a in arr.items():
        setattr(out, name, a.ctypes.data_as(type(getattr(out, name))))
    if g.size != nu:
        raise ValueError(f"g_static has {g.size} entries, shape needs {nu}")
    _check(LIB.dasc_plan(C.byref(desc), _ptr(g), C.byref(out)), "dasc_plan")
    res = {k: getattr(out, k) for k, _ in _lib.PlanOut._fields_ if k not in arr}
    unit_shape = (L, H, shape.dk) if shape.arch == "kda" else (L, H)
    res.update({
        "keep": arr["keep"].astype(bool).reshape(unit_shape),
        "horizon": arr["horizon"].reshape(unit_shape),
        "unit_count": arr["unit_count"].reshape(L, H),
        "off": arr["off"], "layer_off": arr["layer_off"], "layer_off_rows": arr["layer_off_rows"],
        "unit_row": arr["unit_row"][: res["n_rows"]].copy(),
        "inv_row": arr["inv_row"], "w_units": arr["w_units"].reshape(unit_shape),
        "rank_begin": arr["rank_begin"], "send": arr["send"].reshape(T, T),
    })
    return res


def dasc_matched_slots(budget_bytes: int, slot_bytes: int) -> int:
    out = C.c_int64()
    _check(LIB.dasc_matched_slots(budget_bytes, slot_bytes, C.byref(out)), "dasc_matched_slots")
    return out.value


def dasc_tp_permutation(shape: Shape, unit_count: np.ndarray, n_ranks: int) -> dict:
    """Stage-1 head-bundle permutation across TP ranks (host).  unit_count is the plan's
    [L, H] retained units.  Returns head_perm [L, H], rank_rows [T] and
    rank_rows_identity [T]."""
    uc = np.ascontiguousarray(unit_count, dtype=np.int32).reshape(-1)
    if uc.size != shape.n_layers * shape.n_heads:
        raise ValueError(f"unit_count has {uc.size} entries, shape needs "
                         f"{shape.n_layers * shape.n_heads}")
    perm = np.zeros(uc.size, np.int32)
    rows = np.zeros(max(n_ranks, 1), np.int64)
    ident = np.zeros(max(n_ranks, 1), np.int64)
    _check(LIB.dasc_tp_permutation(C.byref(shape.c()), _ptr(uc), n_ranks, _ptr(perm),
                                   _ptr(rows), _ptr(ident)), "dasc_tp_permutation")
    return {"head_perm": perm.reshape(shape.n_layers, shape.n_heads), "rank_rows": rows,
            "rank_rows_identity": ident}


# ---- device calls (torch tensors) ----------------------------------------------------

def _dev(t, dtype, name):
    import torch

    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _need(t, n: int, name: str) -> None:
    # The C ABI takes raw pointers; make sure the kernels stay inside each buffer.
    if t.numel() < n:
        raise ValueError(f"{name} has {t.numel()} elements, the call addresses {n}")


def _stream(stream):
    import torch

    s = torch.cuda.current_stream() if stream is None else stream
    return C.c_void_p(s.cuda_stream)


def dasc_pack(shape: Shape, states, src_slot, unit_row, ckpt, dst_slot, n_ranks: int = 1,
              slice_rows: int | None = None, stream=None) -> None:
    """states [n_pool, L, H, dk, dv] f32 -> ckpt [T, n_slots, C_rows, dv] (or [n_slots, R, dv])."""
    import torch

    n_rows = unit_row.numel()
    slice_rows = n_rows if slice_rows is None else slice_rows
    n_slots = ckpt.shape[1] if ckpt.dim() == 4 else ckpt.shape[0]
    _need(states, states.shape[0] * shape.rows * shape.dv, "states")
    _need(ckpt, n_ranks * n_slots * slice_rows * shape.dv, "ckpt")
    _need(dst_slot, src_slot.numel(), "dst_slot")
    _check(LIB.dasc_pack(
        C.byref(shape.c()), _dev(states, torch.float32, "states"), states.shape[0],
        _dev(src_slot, torch.int32, "src_slot"), _dev(unit_row, torch.int32, "unit_row"), n_rows,
        _dev(ckpt, torch.float32, "ckpt"), n_slots, _dev(dst_slot, torch.int32, "dst_slot"),
        n_ranks, slice_rows, src_slot.numel(), _stream(stream)), "dasc_pack")


def dasc_restore(shape: Shape, ckpt, src_slot, inv_row, states, dst_slot, n_rows: int,
                 n_ranks: int = 1, slice_rows: int | None = None, stream=None) -> None:
    import torch

    slice_rows = n_rows if slice_rows is None else slice_rows
    n_slots = ckpt.shape[1] if ckpt.dim() == 4 else ckpt.shape[0]
    _need(states, states.shape[0] * shape.rows * shape.dv, "states")
    _need(ckpt, n_ranks * n_slots * slice_rows * shape.dv, "ckpt")
    _need(inv_row, shape.rows, "inv_row")
    _need(dst_slot, src_slot.numel(), "dst_slot")
    _check(LIB.dasc_restore(
        C.byref(shape.c()), _dev(ckpt, torch.float32, "ckpt"), n_slots,
        _dev(src_slot, torch.int32, "src_slot"), n_ranks, slice_rows, n_rows,
        _dev(inv_row, torch.int32, "inv_row"), _dev(states, torch.float32, "states"),
        states.shape[0], _dev(dst_slot, torch.int32, "dst_slot"), src_slot.numel(),
        _stream(stream)), "dasc_restore")


def dasc_pack_padded(shape: Shape, states, src_slot, unit_row, layer_off_rows, ckpt, dst_slot,
                     stream=None) -> None:
    """App. B Scheme 1 pack; ckpt is [L, n_slots, r_max_rows, dv] float32, with
    layer_off_rows and r_max_rows from dasc_plan (the device copy of its layer_off_rows,
    and ckpt's third dimension)."""
    import torch

    L, n_slots, r_max = ckpt.shape[0], ckpt.shape[1], ckpt.shape[2]
    if L != shape.n_layers or ckpt.dim() != 4:
        raise ValueError("padded ckpt must be [L, n_slots, r_max_rows, dv]")
    _need(states, states.shape[0] * shape.rows * shape.dv, "states")
    _need(layer_off_rows, L + 1, "layer_off_rows")
    _need(dst_slot, src_slot.numel(), "dst_slot")
    _check(LIB.dasc_pack_padded(
        C.byref(shape.c()), _dev(states, torch.float32, "states"), states.shape[0],
        _dev(src_slot, torch.int32, "src_slot"), _dev(unit_row, torch.int32, "unit_row"),
        unit_row.numel(), _dev(layer_off_rows, torch.int32, "layer_off_rows"), r_max,
        _dev(ckpt, torch.float32, "ckpt"), n_slots, _dev(dst_slot, torch.int32, "dst_slot"),
        src_slot.numel(), _stream(stream)), "dasc_pack_padded")


def dasc_restore_padded(shape: Shape, ckpt, src_slot, layer_off_rows, inv_row, states, dst_slot,
                        n_rows: int, stream=None) -> None:
    """App. B Scheme 1 restore from ckpt [L, n_slots, r_max_rows, dv]."""
    import torch

    L, n_slots, r_max = ckpt.shape[0], ckpt.shape[1], ckpt.shape[2]
    if L != shape.n_layers or ckpt.dim() != 4:
        raise ValueError("padded ckpt must be [L, n_slots, r_max_rows, dv]")
    _need(states, states.shape[0] * shape.rows * shape.dv, "states")
    _need(layer_off_rows, L + 1, "layer_off_rows")
    _need(inv_row, shape.rows, "inv_row")
    _need(dst_slot, src_slot.numel(), "dst_slot")
    _check(LIB.dasc_restore_padded(
        C.byref(shape.c()), _dev(ckpt, torch.float32, "ckpt"), n_slots,
        _dev(src_slot, torch.int32, "src_slot"), _dev(layer_off_rows, torch.int32, "layer_off_rows"),
        r_max, n_rows, _dev(inv_row, torch.int32, "inv_row"), _dev(states, torch.float32, "states"),
        states.shape[0], _dev(dst_slot, torch.int32, "dst_slot"), src_slot.numel(),
        _stream(stream)), "dasc_restore_padded")


def dasc_pack_q8(shape: Shape, states, src_slot, unit_row, q, scale, dst_slot, stream=None) -> None:
    """INT8 pack: q [n_slots, R, dv] int8, scale [n_slots, R] float32 (see dasc.h)."""
    import torch

    n_rows = unit_row.numel()
    n_slots = q.shape[0]
    _need(states, states.shape[0] * shape.rows * shape.dv, "states")
    _need(q, n_slots * n_rows * shape.dv, "q")
    _need(scale, n_slots * n_rows, "scale")
    _need(dst_slot, src_slot.numel(), "dst_slot")
    _check(LIB.dasc_pack_q8(
        C.byref(shape.c()), _dev(states, torch.float32, "states"), states.shape[0],
        _dev(src_slot, torch.int32, "src_slot"), _dev(unit_row, torch.int32, "unit_row"), n_rows,
        _dev(q, torch.int8, "q"), _dev(scale, torch.float32, "scale"), n_slots,
        _dev(dst_slot, torch.int32, "dst_slot"), src_slot.numel(), _stream(stream)), "dasc_pack_q8")


def dasc_restore_q8(shape: Shape, q, scale, src_slot, inv_row, states, dst_slot, n_rows: int,
                    stream=None) -> None:
    import torch

    n_slots = q.shape[0]
    _need(states, states.shape[0] * shape.rows * shape.dv, "states")
    _need(q, n_slots * n_rows * shape.dv, "q")
    _need(scale, n_slots * n_rows, "scale")
    _need(inv_row, shape.rows, "inv_row")
    _need(dst_slot, src_slot.numel(), "dst_slot")
    _check(LIB.dasc_restore_q8(
        C.byref(shape.c()), _dev(q, torch.int8, "q"), _dev(scale, torch.float32, "scale"), n_slots,
        _dev(src_slot, torch.int32, "src_slot"), n_rows, _dev(inv_row, torch.int32, "inv_row"),
        _dev(states, torch.float32, "states"), states.shape[0],
        _dev(dst_slot, torch.int32, "dst_slot"), src_slot.numel(), _stream(stream)), "dasc_restore_q8")


def dasc_refresh_workspace_bytes(shape: Shape, n_req: int, W: int) -> int:
    out = C.c_size_t()
    _check(LIB.dasc_refresh_workspace_bytes(C.byref(shape.c()), n_req, W, C.byref(out)),
           "dasc_refresh_workspace_bytes")
    return out.value


def _workspace(shape: Shape, n_req: int, W: int, workspace, device, stream):
    """(tensor, pointer, bytes) of the refresh workspace: the caller's uint8 device tensor,
    or one drawn from torch's allocator when none is given and the call needs it.  A drawn
    one is allocated on the launch stream itself, so that torch's allocator orders its
    reuse after this call's kernels and the block is never one that work still queued on
    another stream is using.  The caller keeps the returned tensor alive until the launch
    has been enqueued."""
    import torch

    if workspace is None:
        need = dasc_refresh_workspace_bytes(shape, n_req, W)
        if need == 0:
            return None, None, 0
        if stream is None:
            workspace = torch.empty(need, dtype=torch.uint8, device=device)
        else:
            with torch.cuda.stream(stream):
                workspace = torch.empty(need, dtype=torch.uint8, device=device)
    return workspace, _dev(workspace, torch.uint8, "workspace"), workspace.numel()


REFRESH_KERNEL = {"auto": _lib.DASC_REFRESH_KERNEL_AUTO, "column": _lib.DASC_REFRESH_KERNEL_COLUMN,
                  "channel_wy": _lib.DASC_REFRESH_KERNEL_CHANNEL_WY}


def _refresh_args(shape: Shape, inv_row, states, slot, k, v, g, beta, W: int):
    import torch

    n_req, H, dk, dv = slot.numel(), shape.n_heads, shape.dk, shape.dv
    _need(states, states.shape[0] * shape.rows * dv, "states")
    _need(inv_row, shape.rows, "inv_row")
    _need(k, n_req * shape.n_qk_heads * W * dk, "k")
    _need(v, n_req * H * W * dv, "v")
    _need(g, n_req * H * W * (dk if shape.arch == "kda" else 1), "g")
    _need(beta, n_req * H * W, "beta")
    return (_dev(inv_row, torch.int32, "inv_row"), _dev(states, torch.float32, "states"),
            states.shape[0], _dev(slot, torch.int32, "slot"), _dev(k, torch.bfloat16, "k"),
            _dev(v, torch.bfloat16, "v"), _dev(g, torch.float32, "g"),
            _dev(beta, torch.float32, "beta"), n_req)


def dasc_refresh(shape: Shape, layer: int, inv_row, states, slot, k, v, g, beta, W: int,
                 init_mode: str = "restored", workspace=None, stream=None) -> None:
    """Refresh one layer's omitted units for every request in `slot`.

    k [n_req, Hqk, W, dk] and v [n_req, H, W, dv] are bfloat16 device tensors; g is
    [n_req, H, W, dk] (KDA) or [n_req, H, W] (GDN) and beta [n_req, H, W], float32.
    """
    a = _refresh_args(shape, inv_row, states, slot, k, v, g, beta, W)
    ws, ws_ptr, ws_bytes = _workspace(shape, a[-1], W, workspace, states.device, stream)
    _check(LIB.dasc_refresh(C.byref(shape.c()), layer, *a, W,
                            INIT[init_mode], ws_ptr, ws_bytes, _stream(stream)), "dasc_refresh")
    del ws


def dasc_refresh_noalloc(shape: Shape, layer: int, inv_row, states, slot, k, v, g, beta, W: int,
                         init_mode: str = "restored", stream=None) -> None:
    """dasc_refresh without a workspace: the library's static device scratch stands in for
    it (dasc.h), so neither this call nor the library allocates device memory."""
    a = _refresh_args(shape, inv_row, states, slot, k, v, g, beta, W)
    _check(LIB.dasc_refresh_noalloc(C.byref(shape.c()), layer, *a, W, INIT[init_mode],
                                    _stream(stream)), "dasc_refresh_noalloc")


def dasc_refresh_select(shape: Shape, layer: int, inv_row, states, slot, k, v, g, beta, W: int,
                        kernel: str, init_mode: str = "restored", workspace=None,
                        stream=None) -> None:
    """dasc_refresh on a named kernel ("auto", "column" or "channel_wy"), for tests and
    comparisons (dasc_testing.h)."""
    a = _refresh_args(shape, inv_row, states, slot, k, v, g, beta, W)
    if kernel == "auto":
        ws, ws_ptr, ws_bytes = _workspace(shape, a[-1], W, workspace, states.device, stream)
    else:
        ws, ws_ptr, ws_bytes = None, None, 0
    _check(LIB.dasc_refresh_select(C.byref(shape.c()), layer, *a, W,
                                   INIT[init_mode], ws_ptr, ws_bytes, REFRESH_KERNEL[kernel],
                                   _stream(stream)), "dasc_refresh_select")
    del ws


def dasc_restore_refresh(shape: Shape, layer: int, ckpt, src_slot, inv_row, states, dst_slot,
                         k, v, g, beta, W: int, n_rows: int, n_ranks: int = 1,
                         slice_rows: int | None = None, init_mode: str = "restored",
                         workspace=None, stream=None) -> None:
    """Restore one layer of each request's state from its checkpoint and refresh its
    omitted units in one launch (dk = dv = 128).  Arguments as dasc_restore and
    dasc_refresh; request i reads checkpoint src_slot[i] and writes pool slot dst_slot[i].
    """
    import torch

    n_req, H, dk, dv = src_slot.numel(), shape.n_heads, shape.dk, shape.dv
    slice_rows = n_rows if slice_rows is None else slice_rows
    n_slots = ckpt.shape[1] if ckpt.dim() == 4 else ckpt.shape[0]
    _need(ckpt, n_ranks * n_slots * slice_rows * dv, "ckpt")
    _need(states, states.shape[0] * shape.rows * dv, "states")
    _need(inv_row, shape.rows, "inv_row")
    _need(dst_slot, n_req, "dst_slot")
    _need(k, n_req * shape.n_qk_heads * W * dk, "k")
    _need(v, n_req * H * W * dv, "v")
    _need(g, n_req * H * W * (dk if shape.arch == "kda" else 1), "g")
    _need(beta, n_req * H * W, "beta")
    ws, ws_ptr, ws_bytes = _workspace(shape, n_req, W, workspace, states.device, stream)
    _check(LIB.dasc_restore_refresh(
        C.byref(shape.c()), layer, _dev(ckpt, torch.float32, "ckpt"), n_slots,
        _dev(src_slot, torch.int32, "src_slot"), n_ranks, slice_rows, n_rows,
        _dev(inv_row, torch.int32, "inv_row"), _dev(states, torch.float32, "states"),
        states.shape[0], _dev(dst_slot, torch.int32, "dst_slot"),
        _dev(k, torch.bfloat16, "k"), _dev(v, torch.bfloat16, "v"),
        _dev(g, torch.float32, "g"), _dev(beta, torch.float32, "beta"),
        n_req, W, INIT[init_mode], ws_ptr, ws_bytes, _stream(stream)), "dasc_restore_refresh")
    del ws
