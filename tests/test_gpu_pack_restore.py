"""GPU parity of dasc_pack / dasc_restore against the oracle: bit-exact."""

import math

import numpy as np
import pytest

import paper_2608_30386_amd as D
from oracle import pack as OK
from oracle import plan as OP
from tests.gpu_util import announce, dev, dev_i32, host_words, plans, shape_of
from workloads import WORKLOADS, log_lambda, states_host

pytestmark = pytest.mark.gpu

SPECIAL = np.array([0x80000000, 0x7FC00001, 0xFFBFFFFF, 0x7F800001, 0x7F800000, 0xFF800000,
                    0x00000001, 0x807FFFFF], dtype=np.uint32)


def _plant(words: np.ndarray, rng) -> np.ndarray:
    flat = words.reshape(-1)
    pos = rng.choice(flat.size, size=min(flat.size, 4096), replace=False)
    flat[pos] = SPECIAL[np.arange(pos.size) % SPECIAL.size]
    return words


def _roundtrip(sh, plan, states_np, src, dst, n_slots, T=1, slice_rows=None, rng=None):
    """Pack then restore on the GPU; compare every word with the oracle."""
    import torch

    n_pool, rows, dv = states_np.shape[0], sh.rows, sh.dv
    R = int(plan["n_rows"])
    C = R if slice_rows is None else slice_rows
    words = states_np.reshape(n_pool, rows, dv).view(np.uint32)
    st = dev(states_np.reshape(n_pool, sh.n_layers, sh.n_heads, sh.dk, dv))
    sentinel = np.full((T, n_slots, max(C, 1), dv), 0x5A5A5A5A, dtype=np.uint32)[:, :, :C]
    ck = dev(sentinel.view(np.float32).copy())
    unit_row = dev_i32(plan["unit_row"])
    inv_row = dev_i32(plan["inv_row"])
    announce(f"pack {sh} R={R} n={len(src)} T={T}")
    D.dasc_pack(sh, st, dev_i32(src), unit_row, ck, dev_i32(dst), n_ranks=T, slice_rows=C)
    torch.cuda.synchronize()
    want = OK.pack(words, src, plan["unit_row"], sentinel, dst, slice_rows=C)
    got = host_words(ck)
    assert np.array_equal(got, want), "pack differs from the oracle"

    garbage = np.full((n_pool, rows, dv), 0x3C3C3C3C, dtype=np.uint32)
    out = dev(garbage.view(np.float32).reshape(n_pool, sh.n_layers, sh.n_heads, sh.dk, dv).copy())
    back_dst = list(np.random.default_rng(0).permutation(n_pool)[: len(dst)])
    announce(f"restore {sh} R={R} n={len(dst)} T={T}")
    D.dasc_restore(sh, ck, dev_i32(dst), inv_row, out, dev_i32(back_dst), n_rows=R, n_ranks=T,
                   slice_rows=C)
    torch.cuda.synchronize()
    want_r = OK.restore(want, dst, plan["unit_row"], garbage, back_dst, slice_rows=C)
    got_r = host_words(out).reshape(n_pool, rows, dv)
    assert np.array_equal(got_r, want_r), "restore differs from the oracle"
    # restore(pack(S)) = S with omitted rows cleared
    mask = (plan["inv_row"] >= 0)[:, None]
    for s, d in zip(src, back_dst):
        assert np.array_equal(got_r[d], np.where(mask, words[s], np.uint32(0)))


def test_tiny_kda_roundtrip():
    wl = WORKLOADS["tiny_kda"]
    lib, _ = plans(wl)
    rng = np.random.default_rng(0)
    st = states_host(wl, wl.n_ckpt)
    _plant(st.view(np.uint32), rng)
    _roundtrip(shape_of(wl), lib, st, src=[3, 1, 0, 2], dst=[0, 5, 2, 3], n_slots=6)


def test_kimi_layer_roundtrip_full_size():
    wl = WORKLOADS["kimi_layer"]
    lib, _ = plans(wl)
    st = states_host(wl, wl.n_ckpt)
    _plant(st.view(np.uint32), np.random.default_rng(1))
    n = wl.n_ckpt
    _roundtrip(shape_of(wl), lib, st, src=list(range(n)), dst=list(range(n))[::-1], n_slots=n)


@pytest.mark.parametrize("dv,dk", [(4, 8), (12, 8), (16, 16), (20, 4), (64, 32), (1024, 8), (2048, 4)])
def test_odd_row_widths(dv, dk):
    # dv/4 = 1 .. 512 vectors per row, powers of two and not
    rng = np.random.default_rng(dv)
    L, H = 2, 3
    g = OP.static_log_decay(rng.uniform(math.log(1e-4), 0, size=(L, H, dk)))
    sh = D.Shape("kda", L, H, H, dk, dv)
    lib = D.dasc_plan(sh, g, "threshold", 0, 64)
    st = rng.standard_normal((3, L, H, dk, dv), dtype=np.float32)
    _plant(st.view(np.uint32), rng)
    _roundtrip(sh, lib, st, src=[2, 0], dst=[1, 0], n_slots=3)


def test_heads_with_none_and_all_rows_and_gdn():
    g_keep, g_omit = math.log(1e-3) / 1e4, math.log(1e-3) / 2.0
    g = np.full((2, 4, 16), g_omit)
    g[0, 1] = g_keep          # whole head kept
    g[1, 2, ::3] = g_keep     # some rows
    sh = D.Shape("kda", 2, 4, 4, 16, 32)
    lib = D.dasc_plan(sh, g, "threshold", 0, 16)
    assert lib["unit_count"][0, 0] == 0 and lib["unit_count"][0, 1] == 16
    st = np.random.default_rng(3).standard_normal((2, 2, 4, 16, 32), dtype=np.float32)
    _roundtrip(sh, lib, st, src=[0, 1], dst=[1, 0], n_slots=2)
    gg = np.full((3, 4), g_omit)
    gg[0, 2] = gg[2, 0] = gg[2, 3] = g_keep
    shg = D.Shape("gdn", 3, 4, 2, 16, 32)
    libg = D.dasc_plan(shg, gg, "threshold", 0, 16)
    stg = np.random.default_rng(4).standard_normal((2, 3, 4, 16, 32), dtype=np.float32)
    _roundtrip(shg, libg, stg, src=[1, 0], dst=[0, 1], n_slots=2)


@pytest.mark.parametrize("T", [2, 8])
def test_rank_sliced_layout(T):
    wl = WORKLOADS["kimi_layer"]
    sh = shape_of(wl)
    p = D.dasc_plan(sh, D.dasc_static_log_decay(log_lambda(wl)), wl.keep_mode, wl.keep_k,
                    wl.w_max, T)
    st = states_host(wl, 8)
    _roundtrip(sh, p, st, src=list(range(8)), dst=list(range(8)), n_slots=8, T=T,
               slice_rows=int(p["slice_rows"]))


def test_empty_plan_and_no_checkpoints():
    import torch

    sh = D.Shape("kda", 1, 2, 2, 16, 16)
    g = np.full((1, 2, 16), math.log(1e-3) / 2.0)
    p = D.dasc_plan(sh, g, "threshold", 0, 1024)
    assert p["n_rows"] == 0
    st = torch.randn(2, 1, 2, 16, 16, device="cuda")
    ck = torch.zeros(1, 2, 1, 16, device="cuda")
    announce("pack with R = 0")
    D.dasc_pack(sh, st, dev_i32([0]), dev_i32(np.zeros(0)), ck, dev_i32([0]), slice_rows=1)
    torch.cuda.synchronize()
    assert torch.equal(ck, torch.zeros_like(ck))          # nothing packed
    out = torch.full_like(st, 7.0)
    announce("restore with R = 0 (all rows zero-filled)")
    D.dasc_restore(sh, ck, dev_i32([0]), dev_i32(p["inv_row"]), out, dev_i32([1]), n_rows=0)
    torch.cuda.synchronize()
    assert torch.equal(out[1], torch.zeros_like(out[1]))
    assert torch.equal(out[0], torch.full_like(out[0], 7.0))


def test_out_of_range_device_indices_are_skipped():
    import torch

    wl = WORKLOADS["tiny_kda"]
    lib, _ = plans(wl)
    sh = shape_of(wl)
    st = dev(states_host(wl, 2))
    R = int(lib["n_rows"])
    ck = torch.full((1, 3, R, sh.dv), 9.0, device="cuda")
    unit_row = lib["unit_row"].copy()
    unit_row[0] = 10_000                      # not a dense row of this state
    announce("pack with out-of-range slot and row indices")
    D.dasc_pack(sh, st, dev_i32([0, 5, 1]), dev_i32(unit_row), ck, dev_i32([0, 1, 7]))
    torch.cuda.synchronize()
    h = ck.cpu()
    assert torch.equal(h[0, 1], torch.full_like(h[0, 1], 9.0))     # bad source slot: skipped
    assert torch.equal(h[0, 2], torch.full_like(h[0, 2], 9.0))     # bad destination slot: skipped
    assert torch.equal(h[0, 0, 0], torch.full_like(h[0, 0, 0], 9.0))  # bad row: not written
    assert torch.equal(h[0, 0, 1:], st[0].reshape(-1, sh.dv)[unit_row[1:]].cpu())


# ---- App. B Scheme 1: the padded layout ------------------------------------------------

def _padded_roundtrip(sh, plan, states_np, src, dst, n_slots):
    import torch

    n_pool, rows, dv, L = states_np.shape[0], sh.rows, sh.dv, sh.n_layers
    R = int(plan["n_rows"])
    off, r_max = plan["layer_off_rows"], int(plan["r_max_rows"])
    rpu = int(plan["rows_per_unit"])
    words = states_np.reshape(n_pool, rows, dv).view(np.uint32)
    st = dev(states_np.reshape(n_pool, L, sh.n_heads, sh.dk, dv))
    sentinel = np.full((L, n_slots, max(r_max, 1), dv), 0x5A5A5A5A, dtype=np.uint32)
    ck = dev(sentinel.view(np.float32).copy())
    announce(f"pack_padded {sh} R={R} r_max_rows={r_max} n={len(src)}")
    D.dasc_pack_padded(sh, st, dev_i32(src), dev_i32(plan["unit_row"]), dev_i32(off), ck,
                       dev_i32(dst))
    torch.cuda.synchronize()
    want = OK.pack_padded(words, src, plan["unit_row"], plan["layer_off"], rpu, sentinel, dst)
    assert np.array_equal(host_words(ck), want), "padded pack differs from the oracle"
    garbage = np.full((n_pool, rows, dv), 0x3C3C3C3C, dtype=np.uint32)
    out = dev(garbage.view(np.float32).reshape(n_pool, L, sh.n_heads, sh.dk, dv).copy())
    back = list(range(len(dst)))[::-1]
    announce(f"restore_padded {sh} R={R} n={len(dst)}")
    D.dasc_restore_padded(sh, ck, dev_i32(dst), dev_i32(off), dev_i32(plan["inv_row"]), out,
                          dev_i32(back), n_rows=R)
    torch.cuda.synchronize()
    want_r = OK.restore_padded(want, dst, plan["unit_row"], plan["layer_off"], rpu, garbage, back)
    assert np.array_equal(host_words(out).reshape(n_pool, rows, dv), want_r), \
        "padded restore differs from the oracle"
    return L * r_max, R


def test_padded_layout_full_model_kda():
    wl = WORKLOADS["kimi_model"]
    lib, _ = plans(wl)
    sh = shape_of(wl)
    st = states_host(wl, 4)
    padded_rows, R = _padded_roundtrip(sh, lib, st, src=[3, 1, 0, 2], dst=[2, 0, 4, 1], n_slots=5)
    announce(f"kimi_model padded rows {padded_rows} vs ragged {R}: gain {padded_rows / R:.2f}")
    assert math.isclose(padded_rows / R, lib["layout_gain"], rel_tol=1e-12)


def test_padded_layout_gdn_and_uneven_layers():
    wl = WORKLOADS["qwen_gdn"]
    lib, _ = plans(wl)
    _padded_roundtrip(shape_of(wl), lib, states_host(wl, 2), src=[1, 0], dst=[0, 1], n_slots=2)
    rng = np.random.default_rng(9)
    L, H, dk, dv = 5, 3, 16, 20                      # ragged row width, an empty layer
    sh = D.Shape("kda", L, H, H, dk, dv)
    g = D.dasc_static_log_decay(rng.uniform(math.log(1e-4), 0, size=(L, H, dk)))
    g[2] = math.log(1e-3) / 1.0                       # layer 2: nothing kept
    g[4, 0] = math.log(1e-3) / 1e4                    # layer 4, head 0: everything kept
    plan = D.dasc_plan(sh, g, "threshold", 0, 64)
    st = _plant((0.1 * rng.standard_normal((3, L, H, dk, dv))).astype(np.float32).view(np.uint32),
                rng).view(np.float32)
    _padded_roundtrip(sh, plan, st, src=[2, 0, 1], dst=[1, 2, 0], n_slots=4)
