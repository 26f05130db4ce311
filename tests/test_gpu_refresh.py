"""GPU parity of dasc_refresh against the fp64 oracle.

Bar: refreshed rows within 2e-3 of the oracle, measured per (request, head) as
max |got - want| / max |want| over the refreshed rows; every other row of the
active state bit-identical to its input.
"""

import math

import numpy as np
import pytest

import paper_2608_30386_amd as D
from paper_2608_30386_amd._lib import DASC_MAX_WINDOW
from oracle import pack as OK
from oracle import recurrence as OR
from tests.gpu_util import (announce, dev, dev_bf16, dev_i32, host_words, kimi_layer_oracle, plans,
                            restored_states, shape_of)
from workloads import WORKLOADS, bf16_bits_from_f32, log_lambda, refresh_inputs, states_host

pytestmark = pytest.mark.gpu

TOL = 2e-3


def run_refresh(sh, pool, layer, inv_row, inp, W, init="restored", slots=None, kernel=None):
    """dasc_refresh (or, with `kernel`, dasc_refresh_select on that kernel) on a copy of
    the pool; returns the pool after the call."""
    import torch

    n_req = inp["k"].shape[0]
    states = dev(pool)
    slots = list(range(n_req)) if slots is None else slots
    announce(f"refresh {sh} layer={layer} n_req={n_req} W={W} init={init} kernel={kernel}")
    args = (sh, layer, dev_i32(inv_row), states, dev_i32(slots), dev_bf16(inp["k"]),
            dev_bf16(inp["v"]), dev(inp["g"]), dev(inp["beta"]), W)
    if kernel is None:
        D.dasc_refresh(*args, init)
    else:
        D.dasc_refresh_select(*args, kernel, init)
    torch.cuda.synchronize()
    return states.cpu().numpy()


def check(sh, pool, got_pool, layer, inv_row, inp, pairs, init="restored", slots=None,
          oracle=None, report=None):
    """Refreshed rows vs the oracle on `pairs` (computed here, or given as `oracle` =
    (want, omitted)); all other rows bit-identical.  Returns the per-head max-normalised
    error; `report`, a dict, also receives the element-wise error (floor 1e-3 max|y|)."""
    n_req = inp["k"].shape[0]
    slots = list(range(n_req)) if slots is None else slots
    H, dk = sh.n_heads, sh.dk
    inv_layer = inv_row[layer * H * dk:(layer + 1) * H * dk]
    if oracle is None:
        layer_in = np.stack([pool[slots[n], layer] for n in range(n_req)])
        want, om = OR.refresh(layer_in, inv_layer, inp["k"], inp["v"], inp["g"], inp["beta"],
                              sh.n_qk_heads, init, pairs=pairs)
    else:
        want, om = oracle
    got = np.stack([got_pool[slots[n], layer, h] for n, h in pairs])
    err = OR.refresh_error(got, want, om, pairs)
    if report is not None:
        report["per_head"] = err
        report["elementwise"] = OR.refresh_error_elementwise(got, want, om, pairs)
        report["pairs"] = len(pairs)
    assert err <= TOL, f"refresh error {err:.3e} > {TOL}"
    # every row that is not refreshed keeps its bits, in every slot and layer
    mask = np.zeros(pool.shape[:4], dtype=bool)
    for n in range(n_req):
        mask[slots[n], layer] = om
    a = pool.view(np.uint32)[~mask]
    b = got_pool.view(np.uint32)[~mask]
    assert np.array_equal(a, b), "a row that is not omitted changed"
    return err


def sample_pairs(n_req, H, omitted, k, seed=0):
    rng = np.random.default_rng(seed)
    cand = [(n, h) for n in range(n_req) for h in range(H) if omitted[h].any()]
    idx = rng.choice(len(cand), size=min(k, len(cand)), replace=False)
    return [cand[i] for i in sorted(idx)]


@pytest.mark.parametrize("init", ["restored", "zero"])
def test_tiny_kda_all_heads(init):
    wl = WORKLOADS["tiny_kda"]
    lib, _ = plans(wl)
    sh = shape_of(wl)
    pool = restored_states(wl, lib, wl.n_req)
    inp = refresh_inputs(wl, 32, log_lambda(wl)[0])
    got = run_refresh(sh, pool, 0, lib["inv_row"], inp, 32, init)
    pairs = [(n, h) for n in range(wl.n_req) for h in range(wl.n_heads)]
    err = check(sh, pool, got, 0, lib["inv_row"], inp, pairs, init)
    announce(f"tiny_kda init={init} max rel err {err:.2e}")


@pytest.mark.parametrize("W", [256, 1024])
def test_kimi_layer_serving_shape_every_head(W):
    # every refreshed (request, head) of the serving shape (16 x 32 heads) against the fp64
    # oracle, in the launch the bench times
    wl, lib, pool, inp, pairs, want, om = kimi_layer_oracle(W)
    sh = shape_of(wl)
    got = run_refresh(sh, pool, 0, lib["inv_row"], inp, W)
    rep = {}
    err = check(sh, pool, got, 0, lib["inv_row"], inp, pairs, oracle=(want, om), report=rep)
    assert rep["pairs"] == wl.n_req * int(om.any(axis=1).sum())
    announce(f"kimi_layer W={W}: all {rep['pairs']} heads, max per-head rel err {err:.2e}, "
             f"element-wise {rep['elementwise']:.2e}")


def test_kimi_layer_serving_shape_w2048():
    wl = WORKLOADS["kimi_layer"]
    lib, _ = plans(wl)
    sh = shape_of(wl)
    W = 2048
    pool = restored_states(wl, lib, wl.n_req)
    inp = refresh_inputs(wl, W, log_lambda(wl)[0])
    got = run_refresh(sh, pool, 0, lib["inv_row"], inp, W)
    om = (lib["inv_row"] < 0).reshape(wl.n_heads, wl.dk)
    pairs = sample_pairs(wl.n_req, wl.n_heads, om, 64, seed=W)
    rep = {}
    err = check(sh, pool, got, 0, lib["inv_row"], inp, pairs, report=rep)
    announce(f"kimi_layer W={W}: {len(pairs)} sampled heads, max per-head rel err {err:.2e}, "
             f"element-wise {rep['elementwise']:.2e}")


def test_qwen_gdn_full_layers():
    # every omitted v-head of two whole layers (8 requests x 20 heads each) against the
    # fp64 oracle
    wl = WORKLOADS["qwen_gdn"]
    lib, _ = plans(wl)
    sh = shape_of(wl)
    n_req = wl.n_req
    pool = restored_states(wl, lib, n_req)
    lam = log_lambda(wl)
    for layer in (0, 35):
        inp = refresh_inputs(wl, 1024, lam[layer], salt=layer)
        got = run_refresh(sh, pool, layer, lib["inv_row"], inp, 1024)
        om = (lib["inv_row"][layer * 32 * 128:(layer + 1) * 32 * 128] < 0).reshape(32, 128)
        assert om.all(axis=1).sum() == 20                   # 20 of 32 v-heads omitted
        pairs = [(n, h) for n in range(n_req) for h in range(32) if om[h].any()]
        assert len(pairs) == 160
        rep = {}
        err = check(sh, pool, got, layer, lib["inv_row"], inp, pairs, report=rep)
        announce(f"qwen_gdn layer={layer}: all 160 heads, max per-head rel err {err:.2e}, "
                 f"element-wise {rep['elementwise']:.2e}")


@pytest.mark.parametrize("arch,dk,dv,H,Hqk,W", [
    ("kda", 32, 12, 3, 3, 1),
    ("kda", 64, 256, 2, 2, 33),
    ("kda", 128, 20, 2, 1, 100),
    ("gdn", 16, 64, 4, 2, 31),
    ("gdn", 128, 128, 4, 2, 65),
])
def test_ragged_shapes(arch, dk, dv, H, Hqk, W):
    rng = np.random.default_rng(dk * 1000 + dv + W)
    L, n_req = 2, 3
    sh = D.Shape(arch, L, H, Hqk, dk, dv)
    unit_shape = (L, H, dk) if arch == "kda" else (L, H)
    g_static = D.dasc_static_log_decay(rng.uniform(math.log(1e-4), 0, size=unit_shape))
    g_static[1, 0] = math.log(1e-3) / 2.0        # layer 1, head 0: every unit omitted
    g_static[1, 1] = math.log(1e-3) / 1e4        # layer 1, head 1: every unit kept
    plan = D.dasc_plan(sh, g_static, "threshold", 0, 64)
    n_pool = 5
    pool = (0.05 * rng.standard_normal((n_pool, L, H, dk, dv))).astype(np.float32)
    inv = plan["inv_row"]
    pool.reshape(n_pool, -1, dv)[:, inv < 0] = 0.0
    k = rng.standard_normal((n_req, Hqk, W, dk)).astype(np.float32)
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    gshape = (n_req, H, W, dk) if arch == "kda" else (n_req, H, W)
    lam = np.exp(rng.uniform(math.log(1e-3), 0, size=gshape[:2] + (1,) * (len(gshape) - 2)))
    inp = {
        "k": bf16_bits_from_f32(k),
        "v": bf16_bits_from_f32(rng.standard_normal((n_req, H, W, dv)).astype(np.float32)),
        "g": (-lam * np.logaddexp(0, rng.standard_normal(gshape))).astype(np.float32),
        "beta": (1 / (1 + np.exp(-rng.standard_normal((n_req, H, W))))).astype(np.float32),
    }
    slots = [4, 0, 2]
    for init in ("restored", "zero"):
        got = run_refresh(sh, pool, 1, inv, inp, W, init, slots=slots)
        pairs = [(n, h) for n in range(n_req) for h in range(H)]
        check(sh, pool, got, 1, inv, inp, pairs, init, slots=slots)


def _inputs_128(arch, n_req, H, Hqk, W, seed, g_lo=None):
    rng = np.random.default_rng(seed)
    dk = dv = 128
    k = rng.standard_normal((n_req, Hqk, W, dk)).astype(np.float32)
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    gshape = (n_req, H, W, dk) if arch == "kda" else (n_req, H, W)
    lam = np.exp(rng.uniform(math.log(1e-4), 0, size=gshape[:2] + (1,) * (len(gshape) - 2)))
    g = -lam * np.logaddexp(0, rng.standard_normal(gshape))
    if g_lo is not None:        # plant very strong decays on a few tokens
        m = rng.random(gshape) < 0.05
        g = np.where(m, rng.uniform(g_lo, -8.0, size=gshape), g)
    return {
        "k": bf16_bits_from_f32(k),
        "v": bf16_bits_from_f32(rng.standard_normal((n_req, H, W, dv)).astype(np.float32)),
        "g": g.astype(np.float32),
        "beta": (1 / (1 + np.exp(-rng.standard_normal((n_req, H, W))))).astype(np.float32),
    }


@pytest.mark.parametrize("arch,W,g_lo", [
    ("kda", 1, None), ("kda", 31, None), ("kda", 33, None), ("kda", 100, None),
    ("kda", 64, -30.0), ("gdn", 1, None), ("gdn", 31, None), ("gdn", 33, None),
    ("gdn", 47, None), ("gdn", 63, None), ("gdn", 65, None), ("gdn", 96, -30.0),
    ("gdn", 129, None), ("gdn", 200, -30.0),
])
def test_chunked_kernel_ragged_and_strong_decay(arch, W, g_lo):
    # dk = dv = 128 takes the chunked MFMA kernel; ragged last chunks and very strong
    # decays (floored at -10 inside the kernel) must stay within the bar
    L, H, Hqk, n_req = 1, 4, 2, 3
    sh = D.Shape(arch, L, H, Hqk, 128, 128)
    rng = np.random.default_rng(W)
    unit_shape = (L, H, 128) if arch == "kda" else (L, H)
    g_static = D.dasc_static_log_decay(rng.uniform(math.log(1e-4), 0, size=unit_shape))
    g_static[0, 0] = math.log(1e-3) / 2.0
    plan = D.dasc_plan(sh, g_static, "threshold", 0, 64)
    inv = plan["inv_row"]
    pool = (0.05 * rng.standard_normal((4, L, H, 128, 128))).astype(np.float32)
    pool.reshape(4, -1, 128)[:, inv < 0] = 0.0
    inp = _inputs_128(arch, n_req, H, Hqk, W, seed=W, g_lo=g_lo)
    slots = [3, 1, 0]
    for init in ("restored", "zero"):
        got = run_refresh(sh, pool, 0, inv, inp, W, init, slots=slots)
        pairs = [(n, h) for n in range(n_req) for h in range(H)]
        err = check(sh, pool, got, 0, inv, inp, pairs, init, slots=slots)
        announce(f"chunked {arch} W={W} g_lo={g_lo} init={init} max rel err {err:.2e}")


@pytest.mark.parametrize("strong_chunks", [(0, 2, 3), (1, 4)])
def test_kda_fast_and_strong_chunks_interleaved(strong_chunks):
    # Chunks of 32 tokens where some channel decays by more than 2^96 take the
    # strong-decay path, the others the fast path, decided per chunk.  Here one channel of
    # every head decays at every token of the chosen chunks (log-gate -12, floored at -10
    # inside the kernel: 2^-461 over a chunk), so that the window switches paths at chosen
    # chunk boundaries, including the first chunk and the ragged last one (W = 150).
    L, H, Hqk, n_req, W = 1, 4, 2, 3, 150
    sh = D.Shape("kda", L, H, Hqk, 128, 128)
    rng = np.random.default_rng(7)
    g_static = D.dasc_static_log_decay(rng.uniform(math.log(1e-4), 0, size=(L, H, 128)))
    plan = D.dasc_plan(sh, g_static, "threshold", 0, 64)
    inv = plan["inv_row"]
    pool = (0.05 * rng.standard_normal((4, L, H, 128, 128))).astype(np.float32)
    pool.reshape(4, -1, 128)[:, inv < 0] = 0.0
    inp = _inputs_128("kda", n_req, H, Hqk, W, seed=11)
    for c in strong_chunks:
        inp["g"][:, :, 32 * c:32 * (c + 1), 5] = -12.0
    slots = [2, 0, 3]
    for init in ("restored", "zero"):
        got = run_refresh(sh, pool, 0, inv, inp, W, init, slots=slots)
        pairs = [(n, h) for n in range(n_req) for h in range(H)]
        err = check(sh, pool, got, 0, inv, inp, pairs, init, slots=slots)
        announce(f"strong chunks {strong_chunks} init={init} max rel err {err:.2e}")


@pytest.mark.parametrize("kernel", [None, "channel_wy"])
def test_gdn_fast_and_strong_chunks_interleaved(kernel):
    # The same switch with one gate per token (GDN heads): the chosen chunks decay at every
    # token, on the GDN kernel and on the channel-wise kernel with its scalar-gate loads.
    L, H, Hqk, n_req, W = 1, 4, 2, 3, 150
    sh = D.Shape("gdn", L, H, Hqk, 128, 128)
    rng = np.random.default_rng(8)
    g_static = D.dasc_static_log_decay(rng.uniform(math.log(1e-4), 0, size=(L, H)))
    g_static[0, 0] = math.log(1e-3) / 2.0
    plan = D.dasc_plan(sh, g_static, "threshold", 0, 64)
    inv = plan["inv_row"]
    pool = (0.05 * rng.standard_normal((4, L, H, 128, 128))).astype(np.float32)
    pool.reshape(4, -1, 128)[:, inv < 0] = 0.0
    inp = _inputs_128("gdn", n_req, H, Hqk, W, seed=12)
    for c in (0, 2, 3):
        inp["g"][:, 1:, 32 * c:32 * (c + 1)] = -12.0
    slots = [1, 3, 0]
    for init in ("restored", "zero"):
        got = run_refresh(sh, pool, 0, inv, inp, W, init, slots=slots, kernel=kernel)
        pairs = [(n, h) for n in range(n_req) for h in range(H)]
        err = check(sh, pool, got, 0, inv, inp, pairs, init, slots=slots)
        announce(f"gdn strong chunks kernel={kernel} init={init} max rel err {err:.2e}")


def test_chunked_and_column_kernels_agree():
    wl = WORKLOADS["kimi_layer"]
    lib, _ = plans(wl)
    sh = shape_of(wl)
    n_req = 4
    pool = restored_states(wl, lib, n_req)
    inp = refresh_inputs(wl, 160, log_lambda(wl)[0], n_req=n_req)
    a = run_refresh(sh, pool, 0, lib["inv_row"], inp, 160)
    b = run_refresh(sh, pool, 0, lib["inv_row"], inp, 160, kernel="column")
    om = lib["inv_row"] < 0
    diff = np.abs(a.reshape(n_req, -1, 128)[:, om] - b.reshape(n_req, -1, 128)[:, om]).max()
    scale = np.abs(b.reshape(n_req, -1, 128)[:, om]).max()
    announce(f"chunked vs column max diff / max {diff / scale:.2e}")
    assert diff <= 1e-3 * scale
    assert np.array_equal(a.reshape(n_req, -1, 128)[:, ~om], b.reshape(n_req, -1, 128)[:, ~om])


def test_gdn_scalar_gate_kernel_matches_channel_kernel():
    # GDN heads take the scalar-gate kernel; the channel-wise kernel must give the same
    # state to within both kernels' distance from the oracle, and both stay in the bar
    wl = WORKLOADS["qwen_gdn"]
    lib, _ = plans(wl)
    sh = shape_of(wl)
    n_req, layer, W = 3, 5, 333
    pool = restored_states(wl, lib, n_req)
    inp = refresh_inputs(wl, W, log_lambda(wl)[layer], n_req=n_req, salt=layer)
    a = run_refresh(sh, pool, layer, lib["inv_row"], inp, W)
    b = run_refresh(sh, pool, layer, lib["inv_row"], inp, W, kernel="channel_wy")
    lo = layer * sh.n_heads * sh.dk
    om = (lib["inv_row"][lo:lo + sh.n_heads * sh.dk] < 0).reshape(sh.n_heads, sh.dk)
    pairs = sample_pairs(n_req, sh.n_heads, om, 6, seed=1)
    for got in (a, b):
        check(sh, pool, got, layer, lib["inv_row"], inp, pairs)
    diff = np.abs(a[:, layer][:, om] - b[:, layer][:, om]).max()
    scale = np.abs(b[:, layer][:, om]).max()
    announce(f"gdn scalar-gate vs channel kernel max diff / max {diff / scale:.2e}")
    assert diff <= 1e-4 * scale


def test_gdn_workspace_reuse():
    # the per-chunk factors live in a caller-owned workspace; one buffer reused by calls
    # with different windows (the larger first, then a smaller one, which reads only
    # what it wrote) gives the bits of a freshly drawn one
    import torch

    L, H, Hqk, n_req = 1, 4, 2, 3
    sh = D.Shape("gdn", L, H, Hqk, 128, 128)
    rng = np.random.default_rng(11)
    g_static = D.dasc_static_log_decay(rng.uniform(math.log(1e-4), 0, size=(L, H)))
    g_static[0, 0] = math.log(1e-3) / 2.0
    g_static[0, 3] = math.log(1e-3) / 2.0
    inv = D.dasc_plan(sh, g_static, "threshold", 0, 64)["inv_row"]
    pool = (0.05 * rng.standard_normal((3, L, H, 128, 128))).astype(np.float32)
    pool.reshape(3, -1, 128)[:, inv < 0] = 0.0
    ws = torch.full((D.dasc_refresh_workspace_bytes(sh, n_req, 160),), 0x7F, dtype=torch.uint8,
                    device="cuda")
    for W in (160, 40):
        inp = _inputs_128("gdn", n_req, H, Hqk, W, seed=W)
        args = (dev_i32(inv), None, dev_i32([2, 0, 1]), dev_bf16(inp["k"]), dev_bf16(inp["v"]),
                dev(inp["g"]), dev(inp["beta"]), W)
        outs = []
        for workspace in (ws, None):
            states = dev(pool)
            announce(f"gdn workspace reuse W={W} explicit={workspace is not None}")
            D.dasc_refresh(sh, 0, args[0], states, *args[2:], workspace=workspace)
            torch.cuda.synchronize()
            outs.append(states.cpu().numpy())
        assert np.array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32))
        check(sh, pool, outs[0], 0, inv, inp, [(n, h) for n in range(n_req) for h in range(H)],
              slots=[2, 0, 1])


@pytest.mark.parametrize("arch", ["kda", "gdn"])
def test_maximum_window(arch):
    # W = DASC_MAX_WINDOW (2^21 tokens): every token but the last 1024 is an identity step
    # (k = v = 0, g = 0, beta = 0: no decay, no update, exactly), so the result is the
    # oracle's replay of those 1024 tokens from the restored state.  The kernels still walk
    # the whole window: 65,536 chunks, input offsets up to 2^30 bytes, a 512 MiB GDN
    # factor workspace.  GDN: two v-heads on one key head.
    import torch

    W, tail = DASC_MAX_WINDOW, 1024
    L, H, n_req = 1, 2, 1
    Hqk = 2 if arch == "kda" else 1
    sh = D.Shape(arch, L, H, Hqk, 128, 128)
    rng = np.random.default_rng(21)
    unit_shape = (L, H, 128) if arch == "kda" else (L, H)
    g_static = D.dasc_static_log_decay(rng.uniform(math.log(1e-4), 0, size=unit_shape))
    g_static[0, 0] = math.log(1e-3) / 2.0             # head 0 (GDN) / row 0 (KDA) omitted
    if arch == "gdn":
        g_static[0, 1] = math.log(1e-3) / 1000.0      # head 1 kept
    inv = D.dasc_plan(sh, g_static, "threshold", 0, 64)["inv_row"]
    pool = (0.05 * rng.standard_normal((1, L, H, 128, 128))).astype(np.float32)
    pool.reshape(1, -1, 128)[:, inv < 0] = 0.0
    inp = _inputs_128(arch, n_req, H, Hqk, tail, seed=W)

    def whole(x, bits=False):
        shape = list(x.shape)
        shape[2] = W
        t = torch.zeros(shape, dtype=torch.bfloat16 if bits else torch.float32, device="cuda")
        t[:, :, W - tail:] = dev_bf16(x) if bits else dev(x)
        return t

    k, v = whole(inp["k"], bits=True), whole(inp["v"], bits=True)
    g, beta = whole(inp["g"]), whole(inp["beta"])
    states = dev(pool)
    announce(f"refresh {sh} n_req=1 W={W} (identity steps but the last {tail})")
    D.dasc_refresh(sh, 0, dev_i32(inv), states, dev_i32([0]), k, v, g, beta, W)
    torch.cuda.synchronize()
    got = states.cpu().numpy()
    del k, v, g, beta
    om = (inv < 0).reshape(H, 128)
    pairs = [(0, h) for h in range(H) if om[h].any()]
    assert pairs
    err = check(sh, pool, got, 0, inv, inp, pairs)
    announce(f"maximum window {arch}: max rel err {err:.2e}")
