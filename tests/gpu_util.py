"""Helpers for the GPU parity tests (uploads, plans, progress lines)."""

from __future__ import annotations

import functools
import sys

import numpy as np

import paper_2608_30386_amd as D
from oracle import plan as OP
from workloads import Workload, log_lambda


def announce(msg: str) -> None:
    """Name the case about to touch the GPU (flushed, so it survives a crash)."""
    sys.stdout.write(f"[gpu] {msg}\n")
    sys.stdout.flush()


def shape_of(wl: Workload) -> D.Shape:
    return D.Shape(wl.arch, wl.n_layers, wl.n_heads, wl.n_qk_heads, wl.dk, wl.dv)


def plans(wl: Workload):
    """Library plan and oracle plan for a workload; their tables must agree."""
    a_log = log_lambda(wl)
    lib = D.dasc_plan(shape_of(wl), D.dasc_static_log_decay(a_log), wl.keep_mode, wl.keep_k,
                      wl.w_max, wl.n_ranks, wl.eps)
    orc = OP.build_plan(OP.static_log_decay(a_log), wl.arch, wl.n_layers, wl.n_heads, wl.dk,
                        wl.dv, wl.w_max, wl.keep_mode, wl.keep_k, wl.eps, wl.n_ranks)
    np.testing.assert_array_equal(lib["unit_row"], orc["unit_row"])
    np.testing.assert_array_equal(lib["inv_row"], orc["inv_row"])
    return lib, orc


def dev(a: np.ndarray):
    import torch

    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def dev_i32(a) -> "torch.Tensor":
    return dev(np.asarray(a, dtype=np.int32))


def dev_bf16(bits: np.ndarray):
    import torch

    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def host_words(t) -> np.ndarray:
    """Device fp32 tensor -> host uint32 words (bit-exact)."""
    return t.cpu().numpy().view(np.uint32)


def restored_states(wl: Workload, plan, n_req: int, salt: int = 0) -> np.ndarray:
    """Restored active states [n_req, L, H, dk, dv] fp32: states_host packed and restored
    on the host by the oracle (retained rows kept, omitted rows +0.0)."""
    from oracle import pack as OK
    from workloads import states_host

    st = states_host(wl, n_req, salt=salt)
    words = st.reshape(n_req, -1, wl.dv).view(np.uint32)
    R = int(plan["n_rows"])
    ck = OK.pack(words, list(range(n_req)), plan["unit_row"],
                 np.zeros((1, n_req, R, wl.dv), np.uint32), list(range(n_req)))
    back = OK.restore(ck, list(range(n_req)), plan["unit_row"], np.zeros_like(words),
                      list(range(n_req)))
    full = back.view(np.float32).reshape(n_req, wl.n_layers, wl.n_heads, wl.dk, wl.dv)
    return np.ascontiguousarray(full)


@functools.lru_cache(maxsize=2)
def kimi_layer_oracle(W: int):
    """The serving-shape KDA layer (16 requests x 32 heads, 128 x 128) at window W: the
    plan, the restored pool, the suffix inputs and the fp64 oracle refresh of EVERY
    refreshed (request, head).  Computed once per window and shared by the refresh and
    fused-load tests (request i restores from source state i in both)."""
    from oracle import recurrence as OR
    from workloads import WORKLOADS, refresh_inputs

    wl = WORKLOADS["kimi_layer"]
    lib, _ = plans(wl)
    pool = restored_states(wl, lib, wl.n_req)
    inp = refresh_inputs(wl, W, log_lambda(wl)[0])
    om = (lib["inv_row"] < 0).reshape(wl.n_heads, wl.dk)
    pairs = [(n, h) for n in range(wl.n_req) for h in range(wl.n_heads) if om[h].any()]
    announce(f"fp64 oracle: {len(pairs)} (request, head) pairs at W={W}")
    want, om2 = OR.refresh(pool[:, 0], lib["inv_row"], inp["k"], inp["v"], inp["g"], inp["beta"],
                           wl.n_qk_heads, "restored", pairs=pairs)
    return wl, lib, pool, inp, pairs, want, om2
