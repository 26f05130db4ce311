"""Oracle: the gated delta rule and the bounded-suffix refresh (test infrastructure).

Sec. 3.1, Eq. 1 defines the KDA state update on S in R^{dv x dk}:

    S_t = S_{t-1} Diag(alpha_t) (I - beta_t k_t k_t^T) + beta_t v_t k_t^T,
    alpha_t in (0, 1)^{dk},  alpha_t = exp(g_t)

GDN is the same rule with one scalar gate per head (Sec. 3.1).  This module works
on the transpose S' = S^T in R^{dk x dv} (row c = key channel c), which turns
Eq. 1 into

    S~  = Diag(alpha_t) S'_{t-1}                       (decay first)
    S'_t = S~ + beta_t k_t (v_t - S~^T k_t)^T           (then erase and write)

Three independent forms are given:
  replay_naive       the transposed per-token form above;
  replay_paper_form  Eq. 1 literally, with explicit dk x dk matrices, in the
                     paper's [dv, dk] orientation (small cases only);
  replay_chunked     the chunkwise WY form.  Unrolling the rule over a chunk of
                     tokens 1..C with cumulative log-decay G_t = sum_{s<=t} g_s:
                       A_ts = beta_t sum_c k_tc k_sc exp(G_tc - G_sc)   (s < t)
                       T    = (I + A)^{-1}
                       W~   = T (beta * (k * exp(G)))     U~ = T (beta * v)
                       U    = U~ - W~ S'                  (per-token deltas)
                       S'  <- Diag(exp(G_C)) S' + (k * exp(G_C - G))^T U
                     which equals the per-token form up to rounding.

refresh() is the Sec. 4.2 load policy with refresh: replay the last W tokens
and copy only the omitted (local) units into the active state.  Reading of the
start state (the paper replays from a zero scratch state; the serving contract
here starts from the restored state): both are provided, "restored" by default.
All arithmetic is binary64.
"""

from __future__ import annotations

import numpy as np


def widen_bf16(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> float64 (exact)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _gates(g: np.ndarray, k: np.ndarray) -> np.ndarray:
    """Per-channel log-gates [..., W, dk]; a per-head gate [..., W] is broadcast over dk."""
    g = np.asarray(g, dtype=np.float64)
    if g.ndim == k.ndim - 1:
        return np.broadcast_to(g[..., None], k.shape)
    return g


def replay_naive(S0: np.ndarray, k: np.ndarray, v: np.ndarray, g: np.ndarray, beta: np.ndarray) -> np.ndarray:
    """Per-token recurrence on S' [..., dk, dv] over all W tokens.

    k [..., W, dk], v [..., W, dv], g [..., W, dk] or [..., W], beta [..., W].
    """
    S = np.array(S0, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    beta = np.asarray(beta, dtype=np.float64)
    gg = _gates(g, k)
    for t in range(k.shape[-2]):
        S = np.exp(gg[..., t, :])[..., :, None] * S                 # Diag(alpha_t) S'
        kt = k[..., t, :]
        y = np.einsum("...c,...cj->...j", kt, S)                      # S~^T k_t
        d = beta[..., t, None] * (v[..., t, :] - y)
        S = S + kt[..., :, None] * d[..., None, :]                    # + beta k (v - S~^T k)^T
    return S


def replay_paper_form(Sp0: np.ndarray, k: np.ndarray, v: np.ndarray, g: np.ndarray, beta: np.ndarray) -> np.ndarray:
    """Eq. 1 as printed, on S [..., dv, dk], with explicit matrices (tiny inputs only)."""
    Sp0 = np.asarray(Sp0, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    beta = np.asarray(beta, dtype=np.float64)
    gg = _gates(g, k)
    out = np.empty_like(Sp0)
    dk = k.shape[-1]
    for idx in np.ndindex(Sp0.shape[:-2]):
        S = Sp0[idx].copy()
        for t in range(k.shape[-2]):
            kt, vt, bt = k[idx][t], v[idx][t], beta[idx][t]
            decay = np.diag(np.exp(gg[idx][t]))
            erase = np.eye(dk) - bt * np.outer(kt, kt)
            S = S @ decay @ erase + bt * np.outer(vt, kt)
        out[idx] = S
    return out


def replay_chunked(S0: np.ndarray, k: np.ndarray, v: np.ndarray, g: np.ndarray, beta: np.ndarray,
                   chunk: int = 64) -> np.ndarray:
    """Chunkwise WY form of the same recurrence on S' [..., dk, dv]."""
    S = np.array(S0, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    beta = np.asarray(beta, dtype=np.float64)
    gg = _gates(g, k)
    W = k.shape[-2]
    for s0 in range(0, W, chunk):
        sl = slice(s0, min(s0 + chunk, W))
        K, V, b = k[..., sl, :], v[..., sl, :], beta[..., sl]
        C = K.shape[-2]
        G = np.cumsum(gg[..., sl, :], axis=-2)                         # [..., C, dk]
        lower = np.tril(np.ones((C, C), dtype=bool), -1)               # s < t
        expo = np.where(lower[:, :, None], G[..., :, None, :] - G[..., None, :, :], -np.inf)
        A = b[..., :, None] * np.einsum("...tc,...sc,...tsc->...ts", K, K, np.exp(expo))
        Tm = np.linalg.inv(np.eye(C) + A)
        Wt = Tm @ (b[..., None] * (K * np.exp(G)))
        Ut = Tm @ (b[..., None] * V)
        U = Ut - Wt @ S
        Khat = K * np.exp(G[..., -1:, :] - G)
        S = np.exp(G[..., -1, :])[..., :, None] * S + np.swapaxes(Khat, -1, -2) @ U
    return S


def refresh(states: np.ndarray, inv_row_layer: np.ndarray, k_bits: np.ndarray, v_bits: np.ndarray,
            g: np.ndarray, beta: np.ndarray, n_qk_heads: int, init: str = "restored",
            pairs: list | None = None):
    """Sec. 4.2 refresh of one layer.

    states        [n_req, H, dk, dv] fp32: the restored active states (input)
    inv_row_layer [H * dk]: packed row of each dense row of this layer, < 0 if omitted
    k_bits        [n_req, Hqk, W, dk] bf16 bits; v_bits [n_req, H, W, dv] bf16 bits
    g             [n_req, H, W, dk] (KDA) or [n_req, H, W] (GDN) fp32; beta [n_req, H, W] fp32
    init          "restored" (start from the restored state) or "zero" (the paper's
                  zero-initialised scratch state)
    pairs         optional list of (request, head) to evaluate; default all of them

    Returns (out, omitted): out float64 [len(pairs), dk, dv] where omitted rows hold the
    replayed state and every other row the input value; omitted [H, dk] bool.
    A head is replayed as a whole because its rows are coupled through S~^T k_t;
    a head with nothing omitted is returned unchanged.
    """
    n_req, H, dk, dv = states.shape
    omitted = (np.asarray(inv_row_layer).reshape(H, dk) < 0)
    group = H // n_qk_heads
    if pairs is None:
        pairs = [(n, h) for n in range(n_req) for h in range(H)]
    out = np.stack([np.asarray(states[n, h], dtype=np.float64) for n, h in pairs])
    todo = [i for i, (n, h) in enumerate(pairs) if omitted[h].any()]
    if todo:
        S0 = out[todo] if init == "restored" else np.zeros((len(todo), dk, dv))
        k = np.stack([widen_bf16(k_bits[pairs[i][0], pairs[i][1] // group]) for i in todo])
        v = np.stack([widen_bf16(v_bits[pairs[i]]) for i in todo])
        gg = np.stack([g[pairs[i]] for i in todo])
        bb = np.stack([beta[pairs[i]] for i in todo])
        SW = replay_naive(S0, k, v, gg, bb)
        for b, i in enumerate(todo):
            m = omitted[pairs[i][1]]
            out[i][m] = SW[b][m]
    return out, omitted


def refresh_error(got: np.ndarray, want: np.ndarray, omitted: np.ndarray, pairs: list) -> float:
    """Largest per-(request, head) error over refreshed rows, normalised by that head's
    largest refreshed magnitude: max |got - want| / max |want|.

    got, want: [len(pairs), dk, dv]; omitted: [H, dk]."""
    worst = 0.0
    for i, (_, h) in enumerate(pairs):
        m = omitted[h]
        if not m.any():
            continue
        ref = np.abs(want[i][m]).max()
        err = np.abs(np.asarray(got[i], dtype=np.float64)[m] - want[i][m]).max()
        worst = max(worst, err / ref if ref > 0 else err)
    return worst


def refresh_error_elementwise(got: np.ndarray, want: np.ndarray, omitted: np.ndarray,
                              pairs: list, floor: float = 1e-3) -> float:
    """Largest element-wise relative error over refreshed rows, with an absolute floor:
    max |got - want| / max(|want|, floor * max |want|), the floor taken per (request,
    head) so that entries near zero do not divide by ~0.

    got, want: [len(pairs), dk, dv]; omitted: [H, dk]."""
    worst = 0.0
    for i, (_, h) in enumerate(pairs):
        m = omitted[h]
        if not m.any():
            continue
        w = want[i][m]
        den = np.maximum(np.abs(w), floor * np.abs(w).max())
        den = np.where(den > 0, den, 1.0)
        err = np.abs(np.asarray(got[i], dtype=np.float64)[m] - w) / den
        worst = max(worst, float(err.max()))
    return worst
