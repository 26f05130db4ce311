"""Oracle: ragged pack (Store) and zero-fill restore (Load, no refresh).

Test infrastructure only.  Both operations are pure bit moves, so they are
written on raw 32-bit words: no floating-point value is ever interpreted, and
-0.0, NaN payloads, infinities and subnormals must survive unchanged.

  Sec. 4.1 / App. B "Scheme 2": the retained units of every layer are flat-packed
      one after another, so a checkpoint holds sum_l r_l units; here a unit is one
      dv-row (KDA) or dk consecutive dv-rows (GDN) of the [dk, dv] state.
  Sec. 4.2: on a hit the retained units are loaded exactly and omitted units are
      left at zero (+0.0, all bits clear).
  Sec. 4.3: with T ranks the packed units are cut into T slices of C units each
      (the last one may be shorter); slice r of checkpoint i lives at
      ckpt[r, i, 0 : len_r].

  App. B "Scheme 1" (padded, the comparison layout): every layer reserves the largest
      retained count R_max = max_l r_l; only the first r_l entries of layer l are
      valid, the rest is padding (left as it was).

Layouts
  states : [n_pool, L * H * dk, dv] words (a pool of active states)
  ckpt   : [T, n_slots, C_rows, dv] words (T = 1 gives [1, n_slots, R, dv])
  padded : [L, n_slots, R_max * rows_per_unit, dv] words
"""

from __future__ import annotations

import numpy as np


def as_words(a: np.ndarray) -> np.ndarray:
    """View an fp32 array as uint32 words (no copy, no value interpretation)."""
    return np.ascontiguousarray(a).view(np.uint32)


def pack(states: np.ndarray, src_slot, unit_row: np.ndarray, ckpt: np.ndarray, dst_slot,
         slice_rows: int | None = None) -> np.ndarray:
    """ckpt[:, dst_slot[i]] <- rows unit_row of states[src_slot[i]]; returns a new ckpt.

    states [n_pool, rows, dv] uint32; ckpt [T, n_slots, C_rows, dv] uint32.
    Rows of ckpt that no packed unit maps to are left as they were.
    """
    out = ckpt.copy()
    T = out.shape[0]
    R = unit_row.shape[0]
    C = R if slice_rows is None else slice_rows
    if T * C < R:
        raise ValueError("slices do not cover the packed rows")
    j = np.arange(R)
    for i in range(len(src_slot)):
        out[j // C, dst_slot[i], j % C, :] = states[src_slot[i]][unit_row, :]
    return out


def restore(ckpt: np.ndarray, src_slot, unit_row: np.ndarray, states: np.ndarray, dst_slot,
            slice_rows: int | None = None) -> np.ndarray:
    """states[dst_slot[i]] <- zeros, then packed rows back at unit_row; returns a new pool."""
    out = states.copy()
    R = unit_row.shape[0]
    C = R if slice_rows is None else slice_rows
    j = np.arange(R)
    for i in range(len(src_slot)):
        dense = np.zeros(out.shape[1:], dtype=out.dtype)
        dense[unit_row, :] = ckpt[j // C, src_slot[i], j % C, :]
        out[dst_slot[i]] = dense
    return out


def concat_slices(ckpt: np.ndarray, slot: int, n_rows: int, slice_rows: int) -> np.ndarray:
    """Re-join the T slices of one checkpoint into the flat [R, dv] layout."""
    T = ckpt.shape[0]
    parts = []
    for r in range(T):
        lo, hi = r * slice_rows, min((r + 1) * slice_rows, n_rows)
        if hi > lo:
            parts.append(ckpt[r, slot, : hi - lo])
    return np.concatenate(parts, axis=0) if parts else ckpt[0, slot, :0]


def pack_padded(states: np.ndarray, src_slot, unit_row: np.ndarray, layer_off: np.ndarray,
                rows_per_unit: int, ckpt: np.ndarray, dst_slot) -> np.ndarray:
    """App. B Scheme 1: entry e < r_l of layer l of checkpoint dst_slot[i] holds the
    e-th retained row of layer l of states[src_slot[i]]; padding entries are left as
    they were.  layer_off [L+1] are the per-layer offsets o_l in units; ckpt is
    [L, n_slots, R_max_rows, dv].  Returns a new ckpt."""
    out = ckpt.copy()
    L = layer_off.shape[0] - 1
    for i in range(len(src_slot)):
        for l in range(L):
            lo, hi = int(layer_off[l]) * rows_per_unit, int(layer_off[l + 1]) * rows_per_unit
            if hi - lo > out.shape[2]:
                raise ValueError("layer holds more rows than the padded width")
            out[l, dst_slot[i], : hi - lo] = states[src_slot[i]][unit_row[lo:hi]]
    return out


def restore_padded(ckpt: np.ndarray, src_slot, unit_row: np.ndarray, layer_off: np.ndarray,
                   rows_per_unit: int, states: np.ndarray, dst_slot) -> np.ndarray:
    """Load from the padded layout: the valid entries of every layer back at their
    dense rows, every other row +0.0.  Returns a new pool."""
    out = states.copy()
    L = layer_off.shape[0] - 1
    for i in range(len(src_slot)):
        dense = np.zeros(out.shape[1:], dtype=out.dtype)
        for l in range(L):
            lo, hi = int(layer_off[l]) * rows_per_unit, int(layer_off[l + 1]) * rows_per_unit
            dense[unit_row[lo:hi]] = ckpt[l, src_slot[i], : hi - lo]
        out[dst_slot[i]] = dense
    return out
