"""The checkpoint path captured into a HIP graph (as the bench times it) gives, on every
replay, exactly what plain launches give: pack, restore and refresh of a KDA layer,
replayed three times with the outputs scrambled and other eager work in between."""

import numpy as np
import pytest

import paper_2608_30386_amd as D
from tests.gpu_util import announce, dev, dev_bf16, dev_i32, plans, shape_of
from workloads import WORKLOADS, log_lambda, refresh_inputs, states_host

pytestmark = pytest.mark.gpu


def test_graph_replays_match_plain_launches():
    import torch

    wl = WORKLOADS["kimi_layer"]
    lib, _ = plans(wl)
    sh = shape_of(wl)
    n_ckpt, n_req, W, R = 8, 4, 256, int(lib["n_rows"])
    st = dev(states_host(wl, n_ckpt))
    inp = refresh_inputs(wl, W, log_lambda(wl)[0], n_req=n_req)
    k, v = dev_bf16(inp["k"]), dev_bf16(inp["v"])
    g, beta = dev(inp["g"]), dev(inp["beta"])
    unit_row, inv_row = dev_i32(lib["unit_row"]), dev_i32(lib["inv_row"])
    ids, req = dev_i32(np.arange(n_ckpt)), dev_i32(np.arange(n_req))

    def make_step(ckpt, active):
        def step():
            D.dasc_pack(sh, st, ids, unit_row, ckpt, ids)
            D.dasc_restore(sh, ckpt, ids, inv_row, active, ids, n_rows=R)
            D.dasc_refresh(sh, 0, inv_row, active, req, k, v, g, beta, W)
        return step

    announce(f"plain launches: pack/restore {n_ckpt} ckpts, refresh {n_req} req W={W}")
    ck_ref = torch.empty((n_ckpt, R, sh.dv), device="cuda")
    act_ref = torch.empty_like(st)
    make_step(ck_ref, act_ref)()
    torch.cuda.synchronize()
    ck_want = ck_ref.cpu().numpy().view(np.uint32)
    act_want = act_ref.cpu().numpy().view(np.uint32)

    ckpt = torch.empty_like(ck_ref)
    active = torch.empty_like(act_ref)
    step = make_step(ckpt, active)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    announce("capture")
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()

    scratch = torch.empty_like(ck_ref)
    for rep in range(3):
        ckpt.fill_(float("nan"))
        active.fill_(-1.0)
        D.dasc_pack(sh, st, ids.flip(0), unit_row, scratch, ids)   # other eager work
        torch.cuda.synchronize()
        announce(f"replay {rep}")
        graph.replay()
        torch.cuda.synchronize()
        assert np.array_equal(ckpt.cpu().numpy().view(np.uint32), ck_want), f"replay {rep}: ckpt"
        assert np.array_equal(active.cpu().numpy().view(np.uint32), act_want), f"replay {rep}: states"
    announce("graph replays bit-identical to plain launches")
