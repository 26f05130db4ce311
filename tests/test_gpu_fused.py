"""GPU parity of dasc_restore_refresh: one launch that restores a layer from its packed
checkpoint and refreshes the omitted units (KDA rows on the channel-wise kernel, GDN heads
on the scalar-gate kernel).  Checked against the oracle's restore
followed by its refresh (refreshed rows within 2e-3, every other row of the layer
bit-exact), bit for bit against the library's own dasc_restore + dasc_refresh, and for
rows it must not touch (other layers, other pool slots)."""

import math

import numpy as np
import pytest

import paper_2608_30386_amd as D
from oracle import pack as OK
from oracle import recurrence as OR
from tests.gpu_util import announce, dev, dev_bf16, dev_i32, kimi_layer_oracle, plans, shape_of
from tests.test_gpu_refresh import _inputs_128, sample_pairs
from workloads import WORKLOADS, log_lambda, refresh_inputs, states_host

pytestmark = pytest.mark.gpu

TOL = 2e-3
SENTINEL = 0x7FC0DEAD        # a quiet-NaN pattern no kernel writes


def oracle_ckpt(states, unit_row, n_slots, ck_slots, n_ranks, slice_rows):
    """Pack every state i into checkpoint slot ck_slots[i] (oracle, uint32 words)."""
    n, dv = states.shape[0], states.shape[-1]
    words = states.reshape(n, -1, dv).view(np.uint32)
    ck = np.zeros((n_ranks, n_slots, slice_rows, dv), np.uint32)
    return OK.pack(words, list(range(n)), unit_row, ck, list(ck_slots), slice_rows)


def oracle_restored(ck, ck_slots, unit_row, rows, dv, slice_rows):
    """Restored state of each request i (checkpoint ck_slots[i]), uint32 [n, rows, dv]."""
    out = np.zeros((len(ck_slots), rows, dv), np.uint32)
    return OK.restore(ck, list(ck_slots), unit_row, out, list(range(len(ck_slots))), slice_rows)


def run_fused(sh, layer, ck, ck_slots, inv_row, pool, dst, inp, W, n_rows, n_ranks, slice_rows,
              init="restored"):
    import torch

    states = dev(pool)
    announce(f"restore_refresh {sh} layer={layer} n_req={len(dst)} W={W} T={n_ranks} init={init}")
    D.dasc_restore_refresh(sh, layer, dev(ck.view(np.float32)), dev_i32(ck_slots), dev_i32(inv_row),
                           states, dev_i32(dst), dev_bf16(inp["k"]), dev_bf16(inp["v"]),
                           dev(inp["g"]), dev(inp["beta"]), W, n_rows=n_rows, n_ranks=n_ranks,
                           slice_rows=slice_rows, init_mode=init)
    torch.cuda.synchronize()
    return states.cpu().numpy()


def run_unfused(sh, layer, ck, ck_slots, inv_row, pool, dst, inp, W, n_rows, n_ranks, slice_rows,
                init="restored"):
    import torch

    states = dev(pool)
    announce(f"restore + refresh {sh} layer={layer} n_req={len(dst)} W={W}")
    D.dasc_restore(sh, dev(ck.view(np.float32)), dev_i32(ck_slots), dev_i32(inv_row), states,
                   dev_i32(dst), n_rows=n_rows, n_ranks=n_ranks, slice_rows=slice_rows)
    D.dasc_refresh(sh, layer, dev_i32(inv_row), states, dev_i32(dst), dev_bf16(inp["k"]),
                   dev_bf16(inp["v"]), dev(inp["g"]), dev(inp["beta"]), W, init)
    torch.cuda.synchronize()
    return states.cpu().numpy()


def check_fused(sh, layer, got, restored, inv_row, dst, inp, pairs, init, n_pool, oracle=None,
                report=None):
    """Refreshed rows vs the oracle on `pairs` (computed here, or given as `oracle` =
    (want, omitted)); the layer's other rows are the restored rows bit for bit; other
    layers and other pool slots keep the sentinel."""
    H, dk, dv = sh.n_heads, sh.dk, sh.dv
    n_req = len(dst)
    lo, hi = layer * H * dk, (layer + 1) * H * dk
    inv_layer = inv_row[lo:hi]
    if oracle is None:
        layer_in = restored.view(np.float32)[:, lo:hi].reshape(n_req, H, dk, dv)
        want, om = OR.refresh(layer_in, inv_layer, inp["k"], inp["v"], inp["g"], inp["beta"],
                              sh.n_qk_heads, init, pairs=pairs)
    else:
        want, om = oracle
    g4 = got.reshape(n_pool, -1, dk, dv)
    g_pairs = np.stack([g4[dst[n], layer * H + h] for n, h in pairs])
    err = OR.refresh_error(g_pairs, want, om, pairs)
    if report is not None:
        report["elementwise"] = OR.refresh_error_elementwise(g_pairs, want, om, pairs)
    assert err <= TOL, f"refresh error {err:.3e} > {TOL}"
    words = got.reshape(n_pool, -1, dv).view(np.uint32)
    keep = ~om.reshape(-1)                              # rows of the layer not refreshed
    for n in range(n_req):
        assert np.array_equal(words[dst[n], lo:hi][keep], restored[n, lo:hi][keep]), \
            "a row that is not refreshed differs from the restored row"
        assert np.all(words[dst[n], :lo] == SENTINEL) and np.all(words[dst[n], hi:] == SENTINEL), \
            "a row of another layer was written"
    for s in set(range(n_pool)) - set(dst):
        assert np.all(words[s] == SENTINEL), "a pool slot outside dst_slot was written"
    return err


def sentinel_pool(n_pool, sh):
    return np.full((n_pool, sh.n_layers, sh.n_heads, sh.dk, sh.dv), SENTINEL,
                   np.uint32).view(np.float32)


@pytest.mark.parametrize("W", [1024, 1000])
def test_kimi_layer_fused(W):
    wl = WORKLOADS["kimi_layer"]
    lib, _ = plans(wl)
    sh = shape_of(wl)
    n_req, R = wl.n_req, int(lib["n_rows"])
    st = states_host(wl, n_req)
    ck_slots = list(range(n_req))[::-1]                 # request i reads checkpoint 15 - i
    ck = oracle_ckpt(st, lib["unit_row"], n_req, ck_slots, 1, R)
    restored = oracle_restored(ck, ck_slots, lib["unit_row"], sh.rows, sh.dv, R)
    n_pool = n_req + 2
    dst = [(5 * i + 1) % n_pool for i in range(n_req)]   # distinct: gcd(5, 18) = 1
    pool = sentinel_pool(n_pool, sh)
    om = (lib["inv_row"] < 0).reshape(wl.n_heads, wl.dk)
    rep, oracle = {}, None
    if W == 1024:
        # the serving shape's oracle over every refreshed head (request i restores from
        # source state i here as in the refresh test, with the same suffix inputs)
        _, _, pool_o, inp, pairs, want, om_o = kimi_layer_oracle(W)
        np.testing.assert_array_equal(pool_o.reshape(n_req, -1, wl.dv).view(np.uint32), restored)
        oracle = (want, om_o)
    else:
        inp = refresh_inputs(wl, W, log_lambda(wl)[0])
        pairs = sample_pairs(n_req, wl.n_heads, om, 8, seed=W)
    got = run_fused(sh, 0, ck, ck_slots, lib["inv_row"], pool, dst, inp, W, R, 1, R)
    err = check_fused(sh, 0, got, restored, lib["inv_row"], dst, inp, pairs, "restored", n_pool,
                      oracle=oracle, report=rep)
    ref = run_unfused(sh, 0, ck, ck_slots, lib["inv_row"], pool, dst, inp, W, R, 1, R)
    g, r = got.reshape(n_pool, -1).view(np.uint32), ref.reshape(n_pool, -1).view(np.uint32)
    assert np.array_equal(g[dst], r[dst]), "fused differs from restore + refresh"
    announce(f"kimi_layer fused W={W}: {len(pairs)} heads vs oracle, max per-head rel err "
             f"{err:.2e}, element-wise {rep['elementwise']:.2e}; bit-equal to unfused")


@pytest.mark.parametrize("arch,init", [("kda", "restored"), ("kda", "zero"), ("gdn", "restored"),
                                       ("gdn", "zero")])
def test_sliced_checkpoint_multilayer(arch, init):
    rng = np.random.default_rng(11)
    L, H, Hqk, W, n_req, T = 3, 4, 2, 100, 3, 3
    sh = D.Shape(arch, L, H, Hqk, 128, 128)
    unit_shape = (L, H, 128) if arch == "kda" else (L, H)   # KDA: rows; GDN: heads
    g_static = D.dasc_static_log_decay(rng.uniform(math.log(1e-4), 0, size=unit_shape))
    g_static[1, 0] = math.log(1e-3) / 2.0          # layer 1, head 0: every row omitted
    g_static[1, 1] = math.log(1e-3) / 1e4          # layer 1, head 1: every row kept
    plan = D.dasc_plan(sh, g_static, "threshold", 0, 64, T)
    R, C = int(plan["n_rows"]), int(plan["slice_rows"])
    st = (0.05 * rng.standard_normal((n_req, L, H, 128, 128))).astype(np.float32)
    n_slots = 5
    ck_slots = [4, 0, 2]
    ck = oracle_ckpt(st, plan["unit_row"], n_slots, ck_slots, T, C)
    restored = oracle_restored(ck, ck_slots, plan["unit_row"], sh.rows, 128, C)
    n_pool = 6
    dst = [5, 1, 3]
    pool = sentinel_pool(n_pool, sh)
    inp = _inputs_128(arch, n_req, H, Hqk, W, seed=5)
    got = run_fused(sh, 1, ck, ck_slots, plan["inv_row"], pool, dst, inp, W, R, T, C, init)
    pairs = [(n, h) for n in range(n_req) for h in range(H)]
    err = check_fused(sh, 1, got, restored, plan["inv_row"], dst, inp, pairs, init, n_pool)
    ref = run_unfused(sh, 1, ck, ck_slots, plan["inv_row"], pool, dst, inp, W, R, T, C, init)
    lo, hi = H * 128, 2 * H * 128
    g = got.reshape(n_pool, -1, 128).view(np.uint32)[:, lo:hi]
    r = ref.reshape(n_pool, -1, 128).view(np.uint32)[:, lo:hi]
    assert np.array_equal(g[dst], r[dst]), "fused differs from restore + refresh"
    announce(f"sliced T={T} {arch} fused init={init} max rel err {err:.2e}")


def test_qwen_gdn_fused_one_layer():
    wl = WORKLOADS["qwen_gdn"]
    lib, _ = plans(wl)
    sh = shape_of(wl)
    n_req, R, layer = 4, int(lib["n_rows"]), 7
    st = states_host(wl, n_req)
    ck_slots = [1, 3, 0, 2]
    ck = oracle_ckpt(st, lib["unit_row"], n_req, ck_slots, 1, R)
    restored = oracle_restored(ck, ck_slots, lib["unit_row"], sh.rows, sh.dv, R)
    n_pool = 5
    dst = [4, 0, 2, 1]
    pool = sentinel_pool(n_pool, sh)
    inp = refresh_inputs(wl, 1024, log_lambda(wl)[layer], n_req=n_req, salt=layer)
    got = run_fused(sh, layer, ck, ck_slots, lib["inv_row"], pool, dst, inp, 1024, R, 1, R)
    lo = layer * sh.n_heads * sh.dk
    om = (lib["inv_row"][lo:lo + sh.n_heads * sh.dk] < 0).reshape(sh.n_heads, sh.dk)
    pairs = [(n, h) for n in range(n_req) for h in range(sh.n_heads) if om[h].any()]   # all 80
    err = check_fused(sh, layer, got, restored, lib["inv_row"], dst, inp, pairs, "restored", n_pool)
    ref = run_unfused(sh, layer, ck, ck_slots, lib["inv_row"], pool, dst, inp, 1024, R, 1, R)
    hi = lo + sh.n_heads * sh.dk
    g_ = got.reshape(n_pool, -1, sh.dv).view(np.uint32)[:, lo:hi]
    r_ = ref.reshape(n_pool, -1, sh.dv).view(np.uint32)[:, lo:hi]
    assert np.array_equal(g_[dst], r_[dst]), "fused differs from restore + refresh"
    announce(f"qwen_gdn fused layer={layer}: all {len(pairs)} heads, max rel err {err:.2e}, "
             "bit-equal to unfused")
