"""Oracle: the static selection plan (test infrastructure only).

Follows, in order:
  Sec. 3.3, Eq. 2   static log-decay g = -exp(A_log) * softplus(a + dt_bias), a = -0.3
  Sec. 3.3, Eq. 3   static retention horizon H_s = ln(eps) / g, eps = 1e-3
  Sec. 4.1          a unit is global (kept) iff H_s(u) > W_max; KDA unit = one
                    (head, key-channel) row, GDN unit = one whole head
  App. B, Scheme 2  ragged layout: layer l owns [o_l, o_{l+1}), o_0 = 0, o_{l+1} = o_l + r_l
  Sec. 4.2, Eq. 7   W_u = clamp(next_pow2(H_s(u)), 4, W_max), W_replay = max over omitted u
  Sec. 4.3          per-rank slot width C = ceil(sum_r U_r / T)
  Sec. 4.3 stage 1  load-time head-bundle permutation across TP ranks (tp_permutation)
  Sec. 4.1, Eq. 6   C_temp^rag, C_ckpt^rag; padded C_temp^pad and layout gain R_max / r_bar
  App. C.1, Eq. 8   matched-HBM slot count N = floor(B / b_bottleneck) - 1

Readings where the paper is silent (each also listed in the design notes):
  * state orientation [dk, dv]: a KDA unit is one dv-contiguous row of S^T;
  * top-k modes (keep k per head / per layer) rank by H_s descending, ties to the
    lower dense unit index; they stand in for "threshold chosen to keep x%";
  * kept units are laid out in (layer, head, channel) order, refining the
    per-layer offsets o_l to per-(layer, head) row offsets;
  * next_pow2(x) is the smallest power of two >= x; the clamp's upper end is W_max;
  * owner (compute) rank of head h under TP degree T is floor(h * T / H); storage
    rank of packed unit p is floor(p / C);
  * the per-rank bottleneck in Eq. 6 / Eq. 8 is the balanced slot width C units;
  * stage-1 permutation (no algorithm given): a bundle is one query/key head with the
    H/Hqk value heads that share it; longest-processing-time placement, bundles by
    retained rows descending (ties: lower layer, then lower bundle) onto the least
    loaded rank (ties: lower rank) that still has room for it in that layer (every
    rank holds Hqk/T bundles of every layer); the identity is kept whenever it is no
    worse, so the worst rank never grows.

All arithmetic is binary64; transcendental calls go through Python's ``math``
module (the platform libm) one element at a time.
"""

from __future__ import annotations

import math

import numpy as np

KEEP_MODES = ("threshold", "topk_head", "topk_layer")


def softplus(x: float) -> float:
    """softplus(x) = ln(1 + e^x), evaluated as max(x, 0) + ln(1 + e^{-|x|})."""
    return max(x, 0.0) + math.log1p(math.exp(-abs(x)))


def static_log_decay(a_log: np.ndarray, dt_bias: np.ndarray | float = 0.0, a: float = -0.3) -> np.ndarray:
    """Eq. 2 with the input-dependent logit fixed at a (Sec. 3.3)."""
    a_log = np.asarray(a_log, dtype=np.float64)
    dt = np.broadcast_to(np.asarray(dt_bias, dtype=np.float64), a_log.shape)
    out = np.empty(a_log.shape, dtype=np.float64)
    fa, fd, fo = a_log.reshape(-1), dt.reshape(-1), out.reshape(-1)
    for i in range(fa.size):
        fo[i] = -math.exp(float(fa[i])) * softplus(a + float(fd[i]))
    return out


def horizon(g: np.ndarray, eps: float = 1e-3) -> np.ndarray:
    """Eq. 3: H_s = ln(eps) / g (tokens for the decay factor to fall to eps)."""
    g = np.asarray(g, dtype=np.float64)
    if not np.all(np.isfinite(g)) or np.any(g >= 0):
        raise ValueError("static log-decay must be finite and negative")
    if not (0.0 < eps < 1.0):
        raise ValueError("eps must lie in (0, 1)")
    return math.log(eps) / g


def next_pow2(x: float) -> int:
    """Smallest power of two that is >= x (x > 0)."""
    p = 1
    while p < x:
        p *= 2
    return p


def replay_window(h: float, w_max: int) -> int:
    """Eq. 7 for one unit: clamp(next_pow2(H_s), 4, W_max)."""
    if h >= w_max:  # next_pow2(h) >= h >= W_max, so the clamp returns W_max
        return int(w_max)
    return int(min(max(next_pow2(h), 4), w_max))


def _rank_desc(values: list[float]) -> list[int]:
    # descending H_s, ties to the lower index
    return sorted(range(len(values)), key=lambda i: (-values[i], i))


def select(H: np.ndarray, arch: str, mode: str, w_max: int, keep_k: int = 0) -> np.ndarray:
    """Keep mask over units.  H is [L, H, dk] (KDA) or [L, H] (GDN)."""
    if mode == "threshold":
        return H > float(w_max)                     # Sec. 4.1: strictly greater
    keep = np.zeros(H.shape, dtype=bool)
    if mode == "topk_head":
        if arch != "kda":
            raise ValueError("per-head top-k needs channel units")
        L, Hh, dk = H.shape
        if not 0 <= keep_k <= dk:
            raise ValueError("keep_k out of range")
        for l in range(L):
            for h in range(Hh):
                for c in _rank_desc([float(x) for x in H[l, h]])[:keep_k]:
                    keep[l, h, c] = True
        return keep
    if mode == "topk_layer":
        L = H.shape[0]
        per_layer = H.reshape(L, -1)
        if not 0 <= keep_k <= per_layer.shape[1]:
            raise ValueError("keep_k out of range")
        flat = keep.reshape(L, -1)
        for l in range(L):
            for u in _rank_desc([float(x) for x in per_layer[l]])[:keep_k]:
                flat[l, u] = True
        return keep
    raise ValueError(f"unknown keep mode {mode!r}")


def build_plan(g: np.ndarray, arch: str, n_layers: int, n_heads: int, dk: int, dv: int,
               w_max: int, mode: str = "threshold", keep_k: int = 0, eps: float = 1e-3,
               n_ranks: int = 1, conv_bytes: int = 0) -> dict:
    """The whole offline plan from per-unit static log-decay g.

    g: [L, H, dk] for KDA, [L, H] for GDN.  Returns a dict of numpy arrays/scalars:
      keep[L,H(,dk)] bool, horizon, unit_count[L,H] (units kept per head),
      off[L*H+1] (row offsets of each (l,h) block in the packed buffer),
      layer_off[L+1] (App. B o_l, in units), layer_off_rows[L+1] (the same in rows),
      r_max_rows (rows each layer reserves in the padded layout of App. B Scheme 1),
      unit_row[R] (dense row of packed row j),
      inv_row[L*H*dk] (packed row of dense row, -1 if omitted), n_rows R,
      n_units, rows_per_unit, w_units (Eq. 7 per unit, 0 for kept units), w_replay,
      slice_units C, slice_rows, rank_begin[T+1] (rows), send[T,T] (units),
      c_temp_rag, c_temp_pad, layout_gain, c_ckpt, slot_bytes_rank, dense_slot_bytes_rank.
    """
    L, Hh = n_layers, n_heads
    exp_shape = (L, Hh, dk) if arch == "kda" else (L, Hh)
    g = np.asarray(g, dtype=np.float64)
    if g.shape != exp_shape:
        raise ValueError(f"g has shape {g.shape}, expected {exp_shape}")
    if n_ranks < 1:
        raise ValueError("n_ranks must be >= 1")
    Hs = horizon(g, eps)
    keep = select(Hs, arch, mode, w_max, keep_k)

    rows_per_unit = 1 if arch == "kda" else dk
    unit_bytes = rows_per_unit * dv * 4                      # FP32 temporal state
    n_dense_rows = L * Hh * dk

    # kept units per (l, h) and row offsets in (l, h, c) order
    if arch == "kda":
        unit_count = keep.sum(axis=2).astype(np.int64)
        rows_lh = unit_count.copy()
    else:
        unit_count = keep.astype(np.int64)
        rows_lh = unit_count * dk
    off = np.zeros(L * Hh + 1, dtype=np.int64)
    acc = 0
    for i, r in enumerate(rows_lh.reshape(-1)):
        off[i] = acc
        acc += int(r)
    off[-1] = acc
    n_rows = acc

    unit_row = np.empty(n_rows, dtype=np.int64)
    inv_row = np.full(n_dense_rows, -1, dtype=np.int64)
    j = 0
    for l in range(L):
        for h in range(Hh):
            for c in range(dk):
                kept = keep[l, h, c] if arch == "kda" else keep[l, h]
                if kept:
                    dense = (l * Hh + h) * dk + c
                    unit_row[j] = dense
                    inv_row[dense] = j
                    j += 1
    assert j == n_rows

    # App. B: per-layer offsets in units
    r_layer = unit_count.sum(axis=1)
    layer_off = np.zeros(L + 1, dtype=np.int64)
    for l in range(L):
        layer_off[l + 1] = layer_off[l] + int(r_layer[l])
    n_units = int(layer_off[-1])

    # Eq. 7 over omitted units
    w_units = np.zeros(Hs.shape, dtype=np.int64)
    w_replay = 0
    for idx in np.ndindex(Hs.shape):
        if not keep[idx]:
            w = replay_window(float(Hs[idx]), w_max)
            w_units[idx] = w
            w_replay = max(w_replay, w)

    # Sec. 4.3: balanced slot width and the owner -> storage send matrix
    T = n_ranks
    C = -(-n_units // T)
    rank_begin = np.array([min(r * C, n_units) * rows_per_unit for r in range(T + 1)], dtype=np.int64)
    send = np.zeros((T, T), dtype=np.int64)
    p = 0
    for l in range(L):
        for h in range(Hh):
            owner = (h * T) // Hh
            for _ in range(int(unit_count[l, h])):
                send[owner, p // C] += 1
                p += 1

    # Eq. 6 and the padded layout (Sec. 4.1 / App. B)
    n_l = Hh * dk if arch == "kda" else Hh
    sum_n = L * n_l
    r_max = int(r_layer.max()) if L else 0
    r_bar = n_units / L
    inf = float("inf")
    c_temp_rag = sum_n / n_units if n_units else inf
    c_temp_pad = sum_n / (L * r_max) if r_max else inf
    layout_gain = r_max / r_bar if n_units else float("nan")
    dense_rank = -(-sum_n // T) * unit_bytes                 # dense per-rank temporal bytes
    rag_rank = C * unit_bytes
    c_ckpt = (dense_rank + conv_bytes) / (rag_rank + conv_bytes) if (rag_rank + conv_bytes) else inf

    # App. B Scheme 1: every layer reserves the largest layer's retained rows
    layer_off_rows = layer_off * rows_per_unit
    r_max_rows = r_max * rows_per_unit

    return {
        "arch": arch, "g": g, "horizon": Hs, "keep": keep, "unit_count": unit_count,
        "off": off, "layer_off": layer_off, "layer_off_rows": layer_off_rows,
        "r_max_rows": r_max_rows, "unit_row": unit_row, "inv_row": inv_row,
        "n_rows": n_rows, "n_units": n_units, "rows_per_unit": rows_per_unit,
        "w_units": w_units, "w_replay": w_replay,
        "slice_units": C, "slice_rows": C * rows_per_unit, "rank_begin": rank_begin, "send": send,
        "c_temp_rag": c_temp_rag, "c_temp_pad": c_temp_pad, "layout_gain": layout_gain,
        "c_ckpt": c_ckpt, "slot_bytes_rank": rag_rank + conv_bytes,
        "dense_slot_bytes_rank": dense_rank + conv_bytes,
    }


def matched_slots(budget_bytes: int, bottleneck_slot_bytes: int) -> int:
    """Eq. 8: N = floor(B / b_bottleneck) - 1 (slot 0 is reserved by the allocator)."""
    if bottleneck_slot_bytes <= 0:
        raise ValueError("slot bytes must be positive")
    return budget_bytes // bottleneck_slot_bytes - 1


def tp_permutation(unit_count: np.ndarray, arch: str, n_qk_heads: int, n_ranks: int,
                   dk: int) -> dict:
    """Sec. 4.3, stage 1: a model-load-time reindexing of linear-attention head bundles
    across the T tensor-parallel ranks, chosen so that the most loaded rank holds as few
    retained rows as possible (the number of resident checkpoints is limited by it).

    unit_count: [L, H] retained units per (layer, head) (KDA: rows; GDN: 0 or 1 heads).
    Rank r computes bundle positions [r * Hqk/T, (r + 1) * Hqk/T) of every layer.
    Returns head_perm [L, H] (head_perm[l, p] = original head now at position p; the
    heads of a bundle stay consecutive and in order), rank_rows [T] after the
    permutation and rank_rows_identity [T] before it.
    """
    L, H = unit_count.shape
    B, T = n_qk_heads, n_ranks
    if H % B != 0 or B % T != 0:
        raise ValueError("heads must split into bundles, bundles evenly over ranks")
    g, cap = H // B, B // T
    rows_per_unit = 1 if arch == "kda" else dk
    load = [[sum(int(unit_count[l, b * g + i]) for i in range(g)) * rows_per_unit
             for b in range(B)] for l in range(L)]

    ident = [0] * T
    for l in range(L):
        for b in range(B):
            ident[b // cap] += load[l][b]

    order = sorted(((l, b) for l in range(L) for b in range(B)),
                   key=lambda lb: (-load[lb[0]][lb[1]], lb[0], lb[1]))
    U = [0] * T
    used = [[0] * T for _ in range(L)]
    owner = [[0] * B for _ in range(L)]
    for l, b in order:
        best = -1
        for r in range(T):
            if used[l][r] < cap and (best < 0 or U[r] < U[best]):
                best = r
        owner[l][b] = best
        used[l][best] += 1
        U[best] += load[l][b]

    if max(U) >= max(ident):          # no better than the identity: keep it
        owner = [[b // cap for b in range(B)] for _ in range(L)]
        U = list(ident)
    perm = np.zeros((L, H), dtype=np.int64)
    for l in range(L):
        pos = 0
        for r in range(T):
            for b in range(B):          # a rank's bundles in their original order
                if owner[l][b] == r:
                    for i in range(g):
                        perm[l, pos] = b * g + i
                        pos += 1
    return {"head_perm": perm, "rank_rows": np.array(U, dtype=np.int64),
            "rank_rows_identity": np.array(ident, dtype=np.int64)}
