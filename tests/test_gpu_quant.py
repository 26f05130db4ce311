"""GPU parity of the INT8 checkpoint codec (dasc_pack_q8 / dasc_restore_q8): bit-exact
codes, scales and dequantised states against the FP32 oracle of Eq. 10."""

import math

import numpy as np
import pytest

import paper_2608_30386_amd as D
from oracle import quant as OQ
from tests.gpu_util import announce, dev, dev_i32, plans, shape_of
from workloads import WORKLOADS, states_host

pytestmark = pytest.mark.gpu


def _roundtrip(sh, plan, states_np, src, dst, n_slots):
    import torch

    n_pool, rows, dv = states_np.shape[0], sh.rows, sh.dv
    R = int(plan["n_rows"])
    st = dev(states_np.reshape(n_pool, sh.n_layers, sh.n_heads, sh.dk, dv))
    q = torch.full((n_slots, R, dv), 77, dtype=torch.int8, device="cuda")
    s = torch.full((n_slots, R), -1.0, dtype=torch.float32, device="cuda")
    announce(f"pack_q8 {sh} R={R} n={len(src)}")
    D.dasc_pack_q8(sh, st, dev_i32(src), dev_i32(plan["unit_row"]), q, s, dev_i32(dst))
    torch.cuda.synchronize()
    wq, ws = OQ.pack_q8(states_np.reshape(n_pool, rows, dv), src, plan["unit_row"])
    gq, gs = q.cpu().numpy(), s.cpu().numpy()
    for i, d in enumerate(dst):
        assert np.array_equal(gq[d], wq[i]), "codes differ from the oracle"
        assert np.array_equal(gs[d].view(np.uint32), ws[i].view(np.uint32)), "scales differ"
    for d in set(range(n_slots)) - set(dst):        # untouched slots keep their bytes
        assert np.all(gq[d] == 77) and np.all(gs[d] == -1.0)

    out = torch.full((n_pool, sh.n_layers, sh.n_heads, sh.dk, dv), 5.0, device="cuda")
    back = list(range(len(dst)))
    announce(f"restore_q8 {sh} R={R} n={len(dst)}")
    D.dasc_restore_q8(sh, q, s, dev_i32(dst), dev_i32(plan["inv_row"]), out, dev_i32(back), n_rows=R)
    torch.cuda.synchronize()
    want = OQ.restore_q8(wq, ws, plan["unit_row"], rows)
    got = out.cpu().numpy().reshape(n_pool, rows, dv)
    for i, b in enumerate(back):
        assert np.array_equal(got[b].view(np.uint32), want[i].view(np.uint32)), "restore differs"


def test_kimi_layer_q8_full_size():
    wl = WORKLOADS["kimi_layer"]
    lib, _ = plans(wl)
    st = states_host(wl, wl.n_ckpt)
    n = wl.n_ckpt
    _roundtrip(shape_of(wl), lib, st, src=list(range(n)), dst=list(range(n))[::-1], n_slots=n)


@pytest.mark.parametrize("dv,dk", [(4, 8), (8, 4), (16, 16), (64, 32), (256, 8), (1024, 4)])
def test_q8_row_widths_and_zero_rows(dv, dk):
    rng = np.random.default_rng(dv)
    L, H = 2, 3
    sh = D.Shape("kda", L, H, H, dk, dv)
    g = D.dasc_static_log_decay(rng.uniform(math.log(1e-4), 0, size=(L, H, dk)))
    plan = D.dasc_plan(sh, g, "threshold", 0, 64)
    st = (rng.standard_normal((3, L, H, dk, dv)) * rng.uniform(1e-3, 5, size=(3, L, H, dk, 1))).astype(np.float32)
    st.reshape(3, -1, dv)[:, plan["unit_row"][:3]] = 0.0     # some all-zero kept rows
    _roundtrip(sh, plan, st, src=[2, 0, 1], dst=[1, 0, 3], n_slots=4)


def test_q8_error_bound_gdn():
    wl = WORKLOADS["qwen_gdn"]
    lib, _ = plans(wl)
    sh = shape_of(wl)
    st = states_host(wl, 2)
    _roundtrip(sh, lib, st, src=[0, 1], dst=[1, 0], n_slots=2)
