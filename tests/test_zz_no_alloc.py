"""dasc_refresh_noalloc: the refresh with the library's static device scratch in place of
a workspace, called through the C ABI, against dasc_refresh with a caller workspace on
the same inputs.  The kernels are the same, so the results must agree bit for bit; two
calls in a row (the second smaller) check that the shared scratch carries nothing from
one call into the next.  The GDN shape is the one that uses the scratch (its per-chunk
factor records); a KDA shape, which needs none, goes through the same entry."""

import math

import numpy as np
import pytest

import paper_2608_30386_amd as D
from tests.gpu_util import announce, dev, dev_bf16, dev_i32, plans, shape_of
from tests.test_gpu_refresh import _inputs_128, check
from workloads import WORKLOADS, log_lambda, refresh_inputs

pytestmark = pytest.mark.gpu


def _pair(sh, layer, inv, pool, slots, inp, W):
    """(noalloc result, dasc_refresh result) on fresh copies of the pool."""
    import torch

    outs = []
    for noalloc in (True, False):
        states = dev(pool)
        args = (sh, layer, dev_i32(inv), states, dev_i32(slots), dev_bf16(inp["k"]),
                dev_bf16(inp["v"]), dev(inp["g"]), dev(inp["beta"]), W)
        announce(f"{'noalloc' if noalloc else 'workspace'} refresh {sh} layer={layer} "
                 f"n_req={len(slots)} W={W}")
        if noalloc:
            D.dasc_refresh_noalloc(*args)
        else:
            ws = torch.empty(D.dasc_refresh_workspace_bytes(sh, len(slots), W), dtype=torch.uint8,
                             device="cuda")
            D.dasc_refresh(*args, workspace=ws)
        torch.cuda.synchronize()
        outs.append(states.cpu().numpy())
    return outs


def test_noalloc_gdn_two_calls_second_smaller():
    wl = WORKLOADS["qwen_gdn"]
    lib, _ = plans(wl)
    sh = shape_of(wl)
    layer = 3
    rng = np.random.default_rng(3)
    for n_req, W in ((8, 1024), (3, 200)):      # 32 MiB of factor records, then 2.5 MiB
        pool = (0.05 * rng.standard_normal((n_req + 1, wl.n_layers, 32, 128, 128))).astype(np.float32)
        pool.reshape(n_req + 1, -1, 128)[:, lib["inv_row"] < 0] = 0.0
        slots = list(range(1, n_req + 1))
        inp = refresh_inputs(wl, W, log_lambda(wl)[layer], n_req=n_req, salt=100 + W)
        a, b = _pair(sh, layer, lib["inv_row"], pool, slots, inp, W)
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), "noalloc differs"
        lo = layer * 32 * 128
        om = (lib["inv_row"][lo:lo + 32 * 128] < 0).reshape(32, 128)
        pairs = [(n, h) for n in range(n_req) for h in range(32) if om[h].any()][:: max(1, n_req // 2)]
        err = check(sh, pool, a, layer, lib["inv_row"], inp, pairs, slots=slots)
        announce(f"noalloc gdn n_req={n_req} W={W}: bit-equal to dasc_refresh, err {err:.2e}")


def test_noalloc_kda_matches():
    L, H, Hqk, n_req, W = 1, 4, 2, 3, 100
    sh = D.Shape("kda", L, H, Hqk, 128, 128)
    rng = np.random.default_rng(5)
    g_static = D.dasc_static_log_decay(rng.uniform(math.log(1e-4), 0, size=(L, H, 128)))
    inv = D.dasc_plan(sh, g_static, "threshold", 0, 64)["inv_row"]
    pool = (0.05 * rng.standard_normal((3, L, H, 128, 128))).astype(np.float32)
    pool.reshape(3, -1, 128)[:, inv < 0] = 0.0
    inp = _inputs_128("kda", n_req, H, Hqk, W, seed=9)
    a, b = _pair(sh, 0, inv, pool, [2, 0, 1], inp, W)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    check(sh, pool, a, 0, inv, inp, [(n, h) for n in range(n_req) for h in range(H)],
          slots=[2, 0, 1])
