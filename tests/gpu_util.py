"""Helpers for the GPU parity tests (uploads, plans, progress lines)."""

from __future__ import annotations

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
