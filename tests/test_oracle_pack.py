"""Pins for the pack / restore oracle (CPU only): bit moves, checked on raw words."""

import math

import numpy as np
import pytest

from oracle import pack as K
from oracle import plan as P

SPECIAL_WORDS = np.array([
    0x80000000,  # -0.0
    0x7FC00001,  # quiet NaN with payload
    0xFFBFFFFF,  # negative NaN, another payload
    0x7F800001,  # signalling NaN
    0x7F800000,  # +inf
    0xFF800000,  # -inf
    0x00000001,  # smallest subnormal
    0x807FFFFF,  # largest negative subnormal
], dtype=np.uint32)


def _plan(arch, L, H, dk, dv, w, seed=0, T=1):
    rng = np.random.default_rng(seed)
    shape = (L, H, dk) if arch == "kda" else (L, H)
    g = P.static_log_decay(rng.uniform(math.log(1e-4), 0.0, size=shape))
    return P.build_plan(g, arch, L, H, dk, dv, w_max=w, n_ranks=T)


def _words(rng, n, rows, dv, plant=True):
    s = rng.integers(0, 2**32, size=(n, rows, dv), dtype=np.uint64).astype(np.uint32)
    if plant:
        flat = s.reshape(-1)
        pos = rng.choice(flat.size, size=SPECIAL_WORDS.size * 4, replace=False)
        flat[pos] = np.tile(SPECIAL_WORDS, 4)
    return s


@pytest.mark.parametrize("arch", ["kda", "gdn"])
def test_all_kept_pack_is_reshape_and_roundtrip_identity(arch):
    L, H, dk, dv = 2, 3, 4, 8
    p = _plan(arch, L, H, dk, dv, w=0)               # dense plan keeps every unit
    rng = np.random.default_rng(1)
    st = _words(rng, 3, L * H * dk, dv)
    ck = np.zeros((1, 3, p["n_rows"], dv), dtype=np.uint32)
    ck = K.pack(st, [0, 1, 2], p["unit_row"], ck, [0, 1, 2])
    np.testing.assert_array_equal(ck[0], st)
    back = K.restore(ck, [0, 1, 2], p["unit_row"], np.zeros_like(st), [0, 1, 2])
    np.testing.assert_array_equal(back, st)


@pytest.mark.parametrize("arch,w", [("kda", 16), ("kda", 256), ("gdn", 64)])
def test_restore_of_pack_is_masked_state(arch, w):
    L, H, dk, dv = 3, 4, 8, 4
    p = _plan(arch, L, H, dk, dv, w=w, seed=5)
    rng = np.random.default_rng(2)
    n_pool, n_slots = 5, 6
    st = _words(rng, n_pool, L * H * dk, dv)
    src, dst = [4, 0, 2], [5, 1, 3]
    ck0 = _words(rng, 1, n_slots * max(p["n_rows"], 1), dv, plant=False).reshape(1, n_slots, -1, dv)
    ck0 = ck0[:, :, : p["n_rows"]]
    ck = K.pack(st, src, p["unit_row"], ck0, dst)
    # untouched checkpoint slots keep their bits
    for s in set(range(n_slots)) - set(dst):
        np.testing.assert_array_equal(ck[0, s], ck0[0, s])
    garbage = _words(rng, n_pool, L * H * dk, dv, plant=False)
    back = K.restore(ck, dst, p["unit_row"], garbage, [1, 3, 0])
    kept_rows = p["inv_row"] >= 0
    for i, (s, d) in enumerate(zip(src, [1, 3, 0])):
        want = np.where(kept_rows[:, None], st[s], np.uint32(0))   # omitted -> +0.0 bits
        np.testing.assert_array_equal(back[d], want)
    # pools slots restore did not target keep their bits
    for d in set(range(n_pool)) - {1, 3, 0}:
        np.testing.assert_array_equal(back[d], garbage[d])
    # pack(restore(P)) = P
    again = K.pack(back, [1, 3, 0], p["unit_row"], np.zeros_like(ck), dst)
    for d in dst:
        np.testing.assert_array_equal(again[0, d], ck[0, d])


def test_special_bit_patterns_survive():
    L, H, dk, dv = 1, 2, 4, 4
    p = _plan("kda", L, H, dk, dv, w=0)
    st = np.tile(SPECIAL_WORDS, L * H * dk * dv // SPECIAL_WORDS.size).reshape(1, L * H * dk, dv)
    ck = K.pack(st, [0], p["unit_row"], np.zeros((1, 1, p["n_rows"], dv), np.uint32), [0])
    assert ck.tobytes() == st.tobytes()
    back = K.restore(ck, [0], p["unit_row"], np.zeros_like(st), [0])
    assert back.tobytes() == st.tobytes()


def test_heads_with_zero_and_all_rows_kept():
    # head 0 keeps nothing, head 1 keeps everything, head 2 keeps channel 1 only
    g_keep, g_omit = math.log(1e-3) / 1e4, math.log(1e-3) / 2.0
    g = np.full((1, 3, 4), g_omit)
    g[0, 1, :] = g_keep
    g[0, 2, 1] = g_keep
    p = P.build_plan(g, "kda", 1, 3, 4, 4, w_max=16)
    np.testing.assert_array_equal(p["unit_row"], [4, 5, 6, 7, 9])
    np.testing.assert_array_equal(p["off"], [0, 0, 4, 5])
    rng = np.random.default_rng(4)
    st = _words(rng, 1, 12, 4)
    ck = K.pack(st, [0], p["unit_row"], np.zeros((1, 1, 5, 4), np.uint32), [0])
    np.testing.assert_array_equal(ck[0, 0], st[0, [4, 5, 6, 7, 9]])


@pytest.mark.parametrize("arch,T", [("kda", 3), ("kda", 8), ("gdn", 4)])
def test_rank_sliced_layout_reconcatenates(arch, T):
    L, H, dk, dv = 2, 8, 8, 4
    p = _plan(arch, L, H, dk, dv, w=16, seed=9, T=T)
    rng = np.random.default_rng(6)
    st = _words(rng, 2, L * H * dk, dv)
    flat = K.pack(st, [0, 1], p["unit_row"], np.zeros((1, 2, p["n_rows"], dv), np.uint32), [0, 1])
    C = p["slice_rows"]
    sl = K.pack(st, [0, 1], p["unit_row"], np.zeros((T, 2, C, dv), np.uint32), [0, 1], slice_rows=C)
    for s in (0, 1):
        np.testing.assert_array_equal(K.concat_slices(sl, s, p["n_rows"], C), flat[0, s])
    back = K.restore(sl, [0, 1], p["unit_row"], np.zeros_like(st), [0, 1], slice_rows=C)
    back_flat = K.restore(flat, [0, 1], p["unit_row"], np.zeros_like(st), [0, 1])
    np.testing.assert_array_equal(back, back_flat)


# ---- App. B Scheme 1: the padded layout ------------------------------------------------

@pytest.mark.parametrize("arch,w", [("kda", 64), ("kda", 512), ("gdn", 64)])
def test_padded_layout_matches_ragged_and_round_trips(arch, w):
    rng = np.random.default_rng(7)
    L, H, dk, dv, n = 4, 3, 8, 4, 3
    p = _plan(arch, L, H, dk, dv, w, seed=5)
    rpu = p["rows_per_unit"]
    # the plan's padded geometry against a brute-force count of kept dense rows per layer
    kept_rows = (p["inv_row"].reshape(L, -1) >= 0).sum(axis=1)
    assert p["r_max_rows"] == kept_rows.max()
    np.testing.assert_array_equal(p["layer_off_rows"], np.concatenate([[0], np.cumsum(kept_rows)]))
    r_max_rows = int(p["r_max_rows"])
    st = _words(rng, n, L * H * dk, dv)
    sentinel = np.uint32(0xDEADBEEF)
    ckpt = np.full((L, n + 1, r_max_rows, dv), sentinel, np.uint32)
    src, dst = [2, 0, 1], [1, 3, 0]
    pad = K.pack_padded(st, src, p["unit_row"], p["layer_off"], rpu, ckpt, dst)
    # the valid entries of each layer are that layer's range of the ragged checkpoint
    rag = K.pack(st, src, p["unit_row"], np.zeros((1, n + 1, p["n_rows"], dv), np.uint32), dst)
    for i, d in enumerate(dst):
        for l in range(L):
            lo, hi = int(p["layer_off"][l]) * rpu, int(p["layer_off"][l + 1]) * rpu
            assert np.array_equal(pad[l, d, : hi - lo], rag[0, d, lo:hi])
            assert np.all(pad[l, d, hi - lo:] == sentinel)           # padding untouched
    assert np.all(pad[:, 2] == sentinel)                               # unused slot
    # Load: the same restored state as from the ragged layout (masked source state)
    back = K.restore_padded(pad, dst, p["unit_row"], p["layer_off"], rpu,
                            np.zeros((n, L * H * dk, dv), np.uint32), [0, 1, 2])
    mask = p["inv_row"] >= 0
    for i in range(n):
        assert np.array_equal(back[i][mask], st[src[i]][mask])
        assert np.all(back[i][~mask] == 0)
    # capacity: padded over ragged rows is the layout gain R_max / r_bar of Eq. 6
    if p["n_units"]:
        assert math.isclose(L * r_max_rows / (p["n_rows"]), p["layout_gain"], rel_tol=1e-12)
