"""Seeded synthetic inputs shaped like the paper's two models.

The paper evaluates Kimi-Linear-48B-A3B (20 KDA layers, 32 heads, dk = dv = 128)
and Qwen3-Next-80B-A3B (36 GDN layers, 16 q/k heads shared by 32 value heads,
dk = dv = 128) with an FP32 temporal state and BF16 model execution (Sec. 5.1,
Sec. 4.1).  No weights or datasets are available, so every tensor here is drawn
from a seeded generator with the shapes of those models:

* per-unit decay rates lambda (the role of exp(A_log) in Eq. 2, with dt_bias = 0),
  log-uniform over a stated range;
* checkpoint states ~ N(0, std) in fp32;
* suffix-replay inputs: keys L2-normalised N(0, 1) rounded to bf16, values
  N(0, 1) rounded to bf16, per-token log-gates g = -lambda * softplus(z) with
  z ~ N(0, 1) (the token-dependent gate logit of Eq. 2), and update strengths
  beta = sigmoid(N(0, 1)), both fp32.

Every random draw comes from ``numpy.random.SeedSequence(seed).spawn`` streams,
one stream per tensor kind, so the same seed always yields the same bits.  The
only arithmetic here is input shaping (normalisation, rounding to bf16, the
synthetic gate recipe); nothing of the checkpoint method itself lives here.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

# One spawned stream per tensor kind; fixed indices keep draws independent.
_S_LAMBDA, _S_STATE, _S_KEY, _S_VALUE, _S_GATE, _S_BETA, _S_PLANT = range(7)
_N_STREAMS = 8


def streams(seed: int, n: int = _N_STREAMS) -> list[np.random.Generator]:
    """Independent generators spawned from one root seed."""
    return [np.random.default_rng(s) for s in np.random.SeedSequence(seed).spawn(n)]


def _stream(seed: int, idx: int, salt: int = 0) -> np.random.Generator:
    # salt separates e.g. layers or windows that draw the same tensor kind
    root = np.random.SeedSequence([seed, idx, salt])
    return np.random.default_rng(root)


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (nearest, ties to even); returns the uint16 bit pattern."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def f32_from_bf16_bits(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


@dataclass(frozen=True)
class Workload:
    """One synthetic configuration: shape, selection rule and batch sizes."""

    name: str
    arch: str                 # "kda" (channel units) or "gdn" (head units)
    n_layers: int
    n_heads: int              # state (value) heads per layer
    n_qk_heads: int           # key heads; value head j reads key head j // (H / Hqk)
    dk: int
    dv: int
    keep_mode: str            # "threshold" | "topk_head" | "topk_layer"
    keep_k: int               # units kept per head/layer in the top-k modes
    w_max: int                # W_max of Sec. 4.1 / Eq. 7
    lam_range: tuple          # log-uniform range of lambda
    n_ckpt: int               # checkpoints packed and restored per step
    state_std: float
    n_ranks: int = 1          # TP degree T for the per-rank slice table
    n_req: int = 0            # requests refreshed per step
    windows: tuple = ()       # suffix lengths W
    refresh_layers: tuple = (0,)
    planted: bool = False     # kept counts planted per head (full-model KDA set)
    eps: float = 1e-3         # epsilon of Eq. 3
    seed: int = 0
    notes: str = field(default="", compare=False)

    @property
    def units_per_layer(self) -> int:
        return self.n_heads * self.dk if self.arch == "kda" else self.n_heads

    @property
    def rows_per_state(self) -> int:
        return self.n_layers * self.n_heads * self.dk


WORKLOADS: dict[str, Workload] = {
    w.name: w
    for w in [
        Workload(
            name="tiny_kda", arch="kda", n_layers=1, n_heads=2, n_qk_heads=2, dk=16, dv=16,
            keep_mode="topk_head", keep_k=8, w_max=32, lam_range=(1e-3, 1.0),
            n_ckpt=4, state_std=0.1, n_req=4, windows=(32,),
            notes="1 layer, 2 heads, 16x16; keep 8 of 16 channels per head; refresh W=32",
        ),
        Workload(
            name="kimi_layer", arch="kda", n_layers=1, n_heads=32, n_qk_heads=32, dk=128, dv=128,
            keep_mode="topk_layer", keep_k=1556, w_max=1024, lam_range=(1e-4, 1.0),
            n_ckpt=64, state_std=0.05, n_req=16, windows=(256, 1024, 2048),
            notes="Kimi-Linear-shaped KDA layer, 32 heads 128x128, keep 38% of rows "
                  "(1556 of 4096), 64 checkpoints; refresh 16 requests",
        ),
        Workload(
            name="kimi_model", arch="kda", n_layers=24, n_heads=32, n_qk_heads=32, dk=128, dv=128,
            keep_mode="threshold", keep_k=0, w_max=1024, lam_range=(1e-4, 1.0),
            n_ckpt=256, state_std=0.05, n_ranks=8, planted=True,
            notes="24 KDA layers x 32 heads 128x128, 256 checkpoints, heavy-tailed kept "
                  "counts (30% of heads keep <= 16 rows), T = 8 rank slices",
        ),
        Workload(
            name="qwen_gdn", arch="gdn", n_layers=36, n_heads=32, n_qk_heads=16, dk=128, dv=128,
            keep_mode="topk_layer", keep_k=12, w_max=1024, lam_range=(1e-4, 1.0),
            n_ckpt=128, state_std=0.05, n_req=8, windows=(1024,),
            refresh_layers=tuple(range(36)),
            notes="Qwen3-Next-shaped GDN: 36 layers, 16 q/k heads, 32 v-heads, keep 12 "
                  "v-heads per layer, 128 checkpoints; refresh 8 requests x 36 layers",
        ),
    ]
}


def log_lambda(wl: Workload) -> np.ndarray:
    """ln(lambda) per unit: [L, H, dk] for KDA, [L, H] for GDN (float64).

    lambda stands for exp(A_log) of Eq. 2; with dt_bias = 0 this array *is* A_log.
    """
    rng = _stream(wl.seed, _S_LAMBDA)
    lo, hi = math.log(wl.lam_range[0]), math.log(wl.lam_range[1])
    if wl.arch == "gdn":
        return rng.uniform(lo, hi, size=(wl.n_layers, wl.n_heads))
    if not wl.planted:
        return rng.uniform(lo, hi, size=(wl.n_layers, wl.n_heads, wl.dk))
    return _planted_log_lambda(wl)


def planted_counts(wl: Workload) -> np.ndarray:
    """Kept rows per (layer, head) for the heavy-tailed full-model set.

    30% of heads (rounded: 230 of 768) draw a count uniformly from 0..16, the rest
    from 17..dk; one small head is forced to 0 and one large head to dk.
    """
    rng = _stream(wl.seed, _S_PLANT)
    n = wl.n_layers * wl.n_heads
    n_small = int(round(0.3 * n))
    order = rng.permutation(n)
    small, big = order[:n_small], order[n_small:]
    r = np.empty(n, dtype=np.int64)
    r[small] = rng.integers(0, 17, size=small.size)
    r[big] = rng.integers(17, wl.dk + 1, size=big.size)
    r[small[0]] = 0
    r[big[0]] = wl.dk
    return r.reshape(wl.n_layers, wl.n_heads)


def _planted_log_lambda(wl: Workload) -> np.ndarray:
    # Kept channels get lambda in [1e-4, 1e-3], omitted ones lambda in [1.5e-2, 1]:
    # with a = -0.3 and eps = 1e-3 their horizons fall above ~12,460 and below ~831
    # tokens, so the single threshold W_max = 1024 reproduces the planted counts.
    counts = planted_counts(wl)
    rng = _stream(wl.seed, _S_LAMBDA, 1)
    out = np.empty((wl.n_layers, wl.n_heads, wl.dk))
    for l in range(wl.n_layers):
        for h in range(wl.n_heads):
            keep = np.zeros(wl.dk, dtype=bool)
            keep[rng.choice(wl.dk, size=counts[l, h], replace=False)] = True
            out[l, h] = np.where(
                keep,
                rng.uniform(math.log(1e-4), math.log(1e-3), size=wl.dk),
                rng.uniform(math.log(1.5e-2), 0.0, size=wl.dk),
            )
    return out


def states_host(wl: Workload, n: int, salt: int = 0, std: float | None = None) -> np.ndarray:
    """n states [n, L, H, dk, dv] fp32 ~ N(0, std) on the host."""
    rng = _stream(wl.seed, _S_STATE, salt)
    std = wl.state_std if std is None else std
    shape = (n, wl.n_layers, wl.n_heads, wl.dk, wl.dv)
    return (rng.standard_normal(size=shape, dtype=np.float32) * np.float32(std))


def states_device(wl: Workload, n: int, device, salt: int = 0, std: float | None = None):
    """n states drawn directly in device memory (for multi-GB pools).

    Uses torch's seeded device generator; the host copy of any slot is obtained by
    copying it back, so both sides still read the same bits.
    """
    import torch

    std = wl.state_std if std is None else std
    gen = torch.Generator(device=device)
    gen.manual_seed(wl.seed * 1_000_003 + 7919 * salt + 17)
    shape = (n, wl.n_layers, wl.n_heads, wl.dk, wl.dv)
    out = torch.empty(shape, dtype=torch.float32, device=device)
    # fill slot by slot to bound the temporary
    for i in range(n):
        out[i].normal_(0.0, std, generator=gen)
    return out


def refresh_inputs(wl: Workload, W: int, lam_layer: np.ndarray, n_req: int | None = None,
                   salt: int = 0) -> dict:
    """Suffix-replay inputs for one layer.

    lam_layer: ln(lambda) of this layer, [H, dk] (KDA) or [H] (GDN).
    Returns host arrays:
      k    uint16 (bf16 bits) [n_req, Hqk, W, dk], L2-normalised over dk before rounding
      v    uint16 (bf16 bits) [n_req, H,   W, dv]
      g    float32 [n_req, H, W, dk] (KDA) or [n_req, H, W] (GDN), g = -lambda*softplus(z)
      beta float32 [n_req, H, W], sigmoid(N(0,1))
    """
    n_req = wl.n_req if n_req is None else n_req
    H, Hqk, dk, dv = wl.n_heads, wl.n_qk_heads, wl.dk, wl.dv
    rk = _stream(wl.seed, _S_KEY, salt)
    rv = _stream(wl.seed, _S_VALUE, salt)
    rg = _stream(wl.seed, _S_GATE, salt)
    rb = _stream(wl.seed, _S_BETA, salt)

    k = rk.standard_normal(size=(n_req, Hqk, W, dk), dtype=np.float32)
    k /= np.sqrt(np.sum(k * k, axis=-1, keepdims=True, dtype=np.float32))
    v = rv.standard_normal(size=(n_req, H, W, dv), dtype=np.float32)

    lam = np.exp(np.asarray(lam_layer, dtype=np.float64))
    if wl.arch == "kda":
        z = rg.standard_normal(size=(n_req, H, W, dk), dtype=np.float32)
        lam_b = lam.astype(np.float32)[None, :, None, :]
    else:
        z = rg.standard_normal(size=(n_req, H, W), dtype=np.float32)
        lam_b = lam.astype(np.float32)[None, :, None]
    sp = np.logaddexp(np.float32(0.0), z)  # softplus of the synthetic gate logit
    g = (-lam_b * sp).astype(np.float32)
    zb = rb.standard_normal(size=(n_req, H, W), dtype=np.float32)
    beta = (1.0 / (1.0 + np.exp(-zb))).astype(np.float32)
    return {
        "k": bf16_bits_from_f32(k),
        "v": bf16_bits_from_f32(v),
        "g": np.ascontiguousarray(g),
        "beta": np.ascontiguousarray(beta),
    }


def refresh_inputs_device(wl: Workload, W: int, lam_layer: np.ndarray, device,
                          n_req: int | None = None, salt: int = 0) -> dict:
    """refresh_inputs' recipe drawn directly in device memory with torch's seeded
    generator, for benchmark inputs too large to draw on the host quickly.  Same shapes,
    dtypes and distributions (keys L2-normalised in fp32 then rounded to bf16 by
    round-to-nearest-even, values rounded the same way, g = -lambda * softplus(z),
    beta = sigmoid(N(0, 1))); not the same bits as the host recipe.  Returns device
    tensors: k, v bfloat16; g, beta float32."""
    import torch

    n_req = wl.n_req if n_req is None else n_req
    H, Hqk, dk, dv = wl.n_heads, wl.n_qk_heads, wl.dk, wl.dv
    gen = torch.Generator(device=device)
    gen.manual_seed(wl.seed * 1_000_003 + 104_729 * (salt + 1) + 31 * W)
    k = torch.randn((n_req, Hqk, W, dk), generator=gen, device=device)
    k = (k / torch.sqrt((k * k).sum(dim=-1, keepdim=True))).to(torch.bfloat16)
    v = torch.randn((n_req, H, W, dv), generator=gen, device=device).to(torch.bfloat16)
    lam = torch.exp(torch.as_tensor(np.asarray(lam_layer, dtype=np.float64))).to(torch.float32)
    if wl.arch == "kda":
        z = torch.randn((n_req, H, W, dk), generator=gen, device=device)
        lam_b = lam.to(device)[None, :, None, :]
    else:
        z = torch.randn((n_req, H, W), generator=gen, device=device)
        lam_b = lam.to(device)[None, :, None]
    g = (-lam_b * torch.nn.functional.softplus(z)).contiguous()
    beta = torch.sigmoid(torch.randn((n_req, H, W), generator=gen, device=device)).contiguous()
    return {"k": k.contiguous(), "v": v.contiguous(), "g": g, "beta": beta}
