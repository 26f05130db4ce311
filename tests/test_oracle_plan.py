"""Pins for the plan oracle against what the paper and arithmetic fix (CPU only)."""

import json
import math
import os

import numpy as np
import pytest

from oracle import plan as P

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _rand_plan_inputs(rng, arch, L, H, dk):
    shape = (L, H, dk) if arch == "kda" else (L, H)
    a_log = rng.uniform(math.log(1e-4), 0.0, size=shape)
    return P.static_log_decay(a_log)


# ---- Eq. 2 / Eq. 3 -------------------------------------------------------------

def test_softplus_identities():
    # softplus(x) - softplus(-x) = x and softplus(0) = ln 2
    for x in [-30.0, -2.5, -0.3, 0.0, 0.3, 1.7, 40.0]:
        assert abs((P.softplus(x) - P.softplus(-x)) - x) <= 4e-16 * max(1.0, abs(x))
    assert P.softplus(0.0) == math.log(2.0)
    # against the textbook form ln(1 + e^x) where that form is accurate
    for x in [-3.0, -0.3, 0.0, 0.7, 5.0]:
        assert abs(P.softplus(x) - math.log(1.0 + math.exp(x))) <= 1e-15 * max(1.0, abs(x))


def test_static_decay_closed_form():
    # A_log = 0 and dt_bias = 0.3 cancel a = -0.3: g = -softplus(0) = -ln 2
    g = P.static_log_decay(np.zeros(3), np.full(3, 0.3))
    assert np.all(g == -math.log(2.0))
    # g scales linearly in exp(A_log) = lambda and is always negative
    lam = np.array([1e-4, 1e-2, 0.5, 1.0])
    g = P.static_log_decay(np.log(lam))
    sp = math.log1p(math.exp(-0.3))
    np.testing.assert_allclose(g, -lam * sp, rtol=4e-15)  # exp(log(lam)) rounds
    assert np.all(g < 0)


def test_horizon_meaning():
    # Eq. 3: after H_s tokens the decay factor e^{g H_s} equals eps
    g = -np.array([1e-4, 3e-3, 0.05, 0.7, 5.0])
    for eps in (1e-3, 1e-2):
        Hs = P.horizon(g, eps)
        np.testing.assert_allclose(np.exp(g * Hs), eps, rtol=1e-13)
    # exact power-of-two case: g = ln(eps)/16 gives H_s = 16 exactly
    g16 = math.log(1e-3) / 16.0
    assert P.horizon(np.array([g16]))[0] == 16.0
    with pytest.raises(ValueError):
        P.horizon(np.array([0.0]))
    with pytest.raises(ValueError):
        P.horizon(np.array([0.1]))


# ---- Sec. 4.1 selection ------------------------------------------------------------

def test_dense_is_w_max_zero_and_large_w_keeps_nothing():
    # App. C.1: dense is the same cache path with W_max = 0 (every unit retained)
    rng = np.random.default_rng(1)
    for arch in ("kda", "gdn"):
        g = _rand_plan_inputs(rng, arch, 3, 4, 8)
        p = P.build_plan(g, arch, 3, 4, 8, 8, w_max=0)
        assert p["keep"].all() and p["n_rows"] == 3 * 4 * 8
        np.testing.assert_array_equal(p["unit_row"], np.arange(3 * 4 * 8))
        assert p["w_replay"] == 0
        big = int(math.ceil(float(p["horizon"].max()))) + 1
        p = P.build_plan(g, arch, 3, 4, 8, 8, w_max=big)
        assert not p["keep"].any() and p["n_rows"] == 0
        assert (p["inv_row"] == -1).all()


def test_threshold_is_strict():
    g16 = math.log(1e-3) / 16.0          # H_s = 16 exactly
    g = np.array([[[g16, g16 * 0.5, g16 * 2.0]]])   # H_s = 16, 32, 8
    p = P.build_plan(g, "kda", 1, 1, 3, 4, w_max=16)
    np.testing.assert_array_equal(p["keep"][0, 0], [False, True, False])


@pytest.mark.parametrize("arch", ["kda", "gdn"])
def test_offsets_and_maps_against_brute_force(arch):
    rng = np.random.default_rng(7)
    L, H, dk, dv = 3, 4, 8, 4
    for trial in range(6):
        g = _rand_plan_inputs(rng, arch, L, H, dk)
        w = int(rng.choice([0, 4, 16, 64, 256, 4096]))
        p = P.build_plan(g, arch, L, H, dk, dv, w_max=w)
        Hs = p["horizon"]
        # independent route: a row is kept iff its unit's H_s > W_max; rows in dense order
        row_keep = (Hs > w) if arch == "kda" else np.repeat((Hs > w)[..., None], dk, axis=-1)
        row_keep = row_keep.reshape(-1)
        np.testing.assert_array_equal(p["unit_row"], np.flatnonzero(row_keep))
        assert p["n_rows"] == row_keep.sum() == p["off"][-1]
        inv = p["inv_row"]
        np.testing.assert_array_equal(inv[p["unit_row"]], np.arange(p["n_rows"]))
        assert (inv >= 0).sum() == p["n_rows"]
        per_lh = row_keep.reshape(L * H, dk).sum(axis=1)
        np.testing.assert_array_equal(np.diff(p["off"]), per_lh)
        # App. B: o_0 = 0, o_{l+1} = o_l + r_l (units)
        r_l = (Hs > w).reshape(L, -1).sum(axis=1)
        np.testing.assert_array_equal(p["layer_off"], np.concatenate([[0], np.cumsum(r_l)]))


def test_topk_modes_brute_force_with_ties():
    H = np.array([[[5.0, 9.0, 9.0, 1.0, 9.0, 2.0],
                   [3.0, 3.0, 3.0, 3.0, 3.0, 3.0]]])
    keep = P.select(H, "kda", "topk_head", w_max=0, keep_k=2)
    np.testing.assert_array_equal(keep[0, 0], [False, True, True, False, False, False])
    np.testing.assert_array_equal(keep[0, 1], [True, True, False, False, False, False])
    keep = P.select(H, "kda", "topk_layer", w_max=0, keep_k=5)
    # layer ranking: 9,9,9 (idx 1,2,4), then 5 (idx 0), then ties at 3 -> lowest idx 6
    want = np.zeros(12, dtype=bool)
    want[[1, 2, 4, 0, 6]] = True
    np.testing.assert_array_equal(keep.reshape(-1), want)
    rng = np.random.default_rng(3)
    for _ in range(20):
        Hs = np.round(rng.uniform(1, 10, size=(2, 3, 5)), 0)      # many ties
        k = int(rng.integers(0, 16))
        keep = P.select(Hs, "kda", "topk_layer", w_max=0, keep_k=k)
        for l in range(2):
            flat, kf = Hs[l].reshape(-1), keep[l].reshape(-1)
            assert kf.sum() == k
            for i in np.flatnonzero(kf):
                for j in np.flatnonzero(~kf):
                    assert flat[i] > flat[j] or (flat[i] == flat[j] and i < j)


# ---- Eq. 7 ----------------------------------------------------------------------

def test_replay_window_golden():
    cases = json.load(open(os.path.join(GOLD, "replay_window.json")))["cases"]
    for c in cases:
        assert P.replay_window(c["h"], c["w_max"]) == c["w"], c


def test_w_replay_is_max_over_omitted_only():
    g16 = math.log(1e-3) / 16.0
    # H_s = 16 (omitted at W_max=64 -> W 16), 5.3-ish, and 200 (kept -> ignored)
    g = np.array([[g16, math.log(1e-3) / 5.3, math.log(1e-3) / 200.0]])
    p = P.build_plan(g, "gdn", 1, 3, 4, 4, w_max=64)
    np.testing.assert_array_equal(p["keep"][0], [False, False, True])
    assert p["w_replay"] == 16
    np.testing.assert_array_equal(p["w_units"][0], [16, 8, 0])


# ---- Sec. 4.3 rank slices ----------------------------------------------------------

@pytest.mark.parametrize("arch,T", [("kda", 1), ("kda", 4), ("kda", 8), ("gdn", 4)])
def test_rank_slices_and_send_matrix(arch, T):
    rng = np.random.default_rng(11 + T)
    L, H, dk = 3, 8, 8
    g = _rand_plan_inputs(rng, arch, L, H, dk)
    p = P.build_plan(g, arch, L, H, dk, 4, w_max=16, n_ranks=T)
    R_units = p["n_units"]
    C = p["slice_units"]
    assert C == -(-R_units // T)
    rb = p["rank_begin"] // p["rows_per_unit"]
    assert rb[0] == 0 and rb[-1] == R_units and np.all(np.diff(rb) <= C)
    send = p["send"]
    assert send.sum() == R_units
    # row sums: units whose head is computed on rank o (brute force)
    owned = np.zeros(T, dtype=np.int64)
    for l in range(L):
        for h in range(H):
            owned[h // (H // T)] += int(p["unit_count"][l, h])
    np.testing.assert_array_equal(send.sum(axis=1), owned)
    np.testing.assert_array_equal(send.sum(axis=0), np.diff(rb))


# ---- Eq. 6 / App. B ratios -----------------------------------------------------------

def test_compression_ratios_closed_form():
    # L = 2 layers of n_l = 4 units (GDN heads); keep 1 and 3 heads
    g_keep, g_omit = math.log(1e-3) / 1000.0, math.log(1e-3) / 2.0
    g = np.array([[g_keep, g_omit, g_omit, g_omit], [g_keep, g_keep, g_keep, g_omit]])
    p = P.build_plan(g, "gdn", 2, 4, 2, 2, w_max=16, conv_bytes=10)
    assert p["c_temp_rag"] == 8 / 4
    assert p["c_temp_pad"] == 8 / (2 * 3)
    assert p["layout_gain"] == 3 / 2
    assert math.isclose(p["c_temp_rag"] / p["c_temp_pad"], p["layout_gain"], rel_tol=1e-15)
    ub = 2 * 2 * 4
    assert p["c_ckpt"] == (8 * ub + 10) / (4 * ub + 10)


# Sec. 4.3 / Eq. 6 / Eq. 8 at T > 1, worked by hand.  One KDA layer, H = 2 heads of
# dk = 5 channels, dv = 4 (a unit is 4 fp32 = 16 B), T = 4 ranks, 8 conv bytes per rank.
# Head 0 keeps channels {0, 1, 2, 4}, head 1 keeps {1, 3, 4}: 7 of 10 units retained.
#   C = ceil(7 / 4) = 2 units per rank slice; rank_begin = [0, 2, 4, 6, 7].
#   Owners: head h is computed on rank floor(h * 4 / 2) = 2h, so packed units 0..3 (head 0)
#   belong to rank 0 and 4..6 (head 1) to rank 2; unit p is stored on rank floor(p / 2):
#   send[0][0] = 2, send[0][1] = 2, send[2][2] = 2, send[2][3] = 1.
#   Dense per-rank bytes: ceil(10 / 4) = 3 units = 48 B, + 8 conv = 56.
#   Ragged per-rank bytes (the bottleneck after balancing): C = 2 units = 32 B, + 8 = 40.
#   C_ckpt = 56 / 40 = 1.4; Eq. 8 with a 4000 B budget: floor(4000 / 40) - 1 = 99 slots.
# Rounding either quotient down instead (floor for ceil) gives C = 1 and 2 dense units:
# slot bytes 24 and 40, C_ckpt 40 / 24 = 1.67 (or 2.33 / 1.0 when only one is floored),
# 165 slots -- every figure below would fail.
HAND_T4 = {"C": 2, "rank_begin": [0, 2, 4, 6, 7], "slot_bytes_rank": 40,
           "dense_slot_bytes_rank": 56, "c_ckpt": 1.4, "slots_4000": 99,
           "send": [[2, 2, 0, 0], [0, 0, 0, 0], [0, 0, 2, 1], [0, 0, 0, 0]]}


def hand_t4_decay():
    """Static log-decay of the hand-worked T = 4 case (kept: H_s = 1000, omitted: H_s = 2,
    against W_max = 16)."""
    keep = np.array([[[1, 1, 1, 0, 1], [0, 1, 0, 1, 1]]], dtype=bool)
    return np.where(keep, math.log(1e-3) / 1000.0, math.log(1e-3) / 2.0)


def test_rank_bottleneck_hand_worked_t4():
    p = P.build_plan(hand_t4_decay(), "kda", 1, 2, 5, 4, w_max=16, n_ranks=4, conv_bytes=8)
    assert p["n_units"] == 7
    assert p["slice_units"] == HAND_T4["C"] and p["slice_rows"] == HAND_T4["C"]
    np.testing.assert_array_equal(p["rank_begin"], HAND_T4["rank_begin"])
    np.testing.assert_array_equal(p["send"], HAND_T4["send"])
    assert p["slot_bytes_rank"] == HAND_T4["slot_bytes_rank"]
    assert p["dense_slot_bytes_rank"] == HAND_T4["dense_slot_bytes_rank"]
    assert p["c_ckpt"] == HAND_T4["c_ckpt"]
    assert p["c_temp_rag"] == 10 / 7
    assert P.matched_slots(4000, p["slot_bytes_rank"]) == HAND_T4["slots_4000"]


def test_matched_hbm_slots_golden():
    gold = json.load(open(os.path.join(GOLD, "matched_hbm.json")))
    for arch in ("kda", "gdn"):
        b = gold[arch]["budget_bytes"]
        per_slot = b // gold[arch]["dense_physical_slots"]
        assert per_slot * gold[arch]["dense_physical_slots"] == b
        assert P.matched_slots(b, per_slot) == gold[arch]["deployable_slots"]
        # the same budget through a dense plan (W_max = 0) at the model's per-rank shape
        s = gold["derived_shapes"][arch]
        shape = (s["n_layers"], s["n_heads"], s["dk"]) if arch == "kda" else (s["n_layers"], s["n_heads"])
        g = np.full(shape, -0.1)
        p = P.build_plan(g, arch, s["n_layers"], s["n_heads"], s["dk"], s["dv"], w_max=0,
                         n_ranks=s["tp"], conv_bytes=s["conv_bytes_per_rank"])
        assert p["dense_slot_bytes_rank"] == per_slot
        assert p["slot_bytes_rank"] == per_slot
        assert P.matched_slots(b, p["slot_bytes_rank"]) == 127
        assert p["c_ckpt"] == 1.0


# ---- Sec. 4.3 stage 1: head-bundle permutation across TP ranks -------------------------

def _bundle_loads(unit_count, arch, B, dk):
    L, H = unit_count.shape
    g, rpu = H // B, (1 if arch == "kda" else dk)
    return [[int(unit_count[l, b * g:(b + 1) * g].sum()) * rpu for b in range(B)] for l in range(L)]


def _check_permutation(unit_count, arch, B, T, dk, res):
    """head_perm moves whole bundles, gives every rank B/T bundles per layer, and the
    reported per-rank rows are what the permuted placement holds."""
    L, H = unit_count.shape
    g, cap = H // B, B // T
    rpu = 1 if arch == "kda" else dk
    perm = res["head_perm"]
    rows = [0] * T
    for l in range(L):
        assert sorted(perm[l].tolist()) == list(range(H))
        for pos_b in range(B):
            heads = perm[l, pos_b * g:(pos_b + 1) * g].tolist()
            assert heads[0] % g == 0 and heads == list(range(heads[0], heads[0] + g))
            rows[pos_b // cap] += int(unit_count[l, heads].sum()) * rpu
    assert rows == res["rank_rows"].tolist()
    ident = [0] * T
    for l in range(L):
        for b, x in enumerate(_bundle_loads(unit_count, arch, B, dk)[l]):
            ident[b // cap] += x
    assert ident == res["rank_rows_identity"].tolist()


def _optimum(loads, T, cap):
    """Smallest worst-rank load over every placement with B/T bundles per rank per layer
    (brute force; tiny inputs only)."""
    import itertools

    L, B = len(loads), len(loads[0])
    per_layer = []
    for l in range(L):
        opts = set()
        for owner in itertools.product(range(T), repeat=B):
            if all(owner.count(r) == cap for r in range(T)):
                opts.add(tuple(sum(loads[l][b] for b in range(B) if owner[b] == r) for r in range(T)))
        per_layer.append(sorted(opts))
    best = None
    for combo in itertools.product(*per_layer):
        worst = max(sum(c[r] for c in combo) for r in range(T))
        best = worst if best is None else min(best, worst)
    return best


def test_tp_permutation_hand_worked():
    # Two KDA layers, four heads, T = 2 (two heads per rank and layer).  Retained rows
    # [8, 1, 1, 0] and [8, 0, 0, 0]: the identity puts 8 + 1 + 8 = 17 rows on rank 0 and
    # 1 on rank 1.  Largest first: (0, 0) -> rank 0, (1, 0) -> rank 1 (now 8 / 8),
    # (0, 1) -> rank 0 (tie, lower rank), (0, 2) -> rank 1, the empty bundles fill the
    # remaining places: 9 / 9 rows, the optimum (18 rows over two ranks).
    uc = np.array([[8, 1, 1, 0], [8, 0, 0, 0]])
    res = P.tp_permutation(uc, "kda", 4, 2, 16)
    assert res["rank_rows"].tolist() == [9, 9]
    assert res["rank_rows_identity"].tolist() == [17, 1]
    assert res["head_perm"].tolist() == [[0, 1, 2, 3], [1, 2, 0, 3]]
    _check_permutation(uc, "kda", 4, 2, 16, res)


def test_tp_permutation_trivial_cases():
    rng = np.random.default_rng(3)
    uc = rng.integers(0, 17, size=(3, 8))
    one = P.tp_permutation(uc, "kda", 8, 1, 16)            # one rank: nothing to move
    assert one["head_perm"].tolist() == [list(range(8))] * 3
    assert one["rank_rows"].tolist() == [int(uc.sum())]
    flat = P.tp_permutation(np.full((2, 8), 5), "kda", 8, 4, 16)   # already balanced
    assert flat["head_perm"].tolist() == [list(range(8))] * 2
    assert flat["rank_rows"].tolist() == [20, 20, 20, 20]


@pytest.mark.parametrize("seed", range(12))
def test_tp_permutation_brute_force(seed):
    rng = np.random.default_rng(100 + seed)
    arch = "kda" if seed % 2 == 0 else "gdn"
    L, T = (2, 2) if seed % 3 else (1, 3)
    B = 4 if T == 2 else 6
    g = 1 if arch == "kda" else 2                           # value heads per bundle
    hi = 17 if arch == "kda" else 2
    uc = rng.integers(0, hi, size=(L, B * g))
    if seed % 4 == 1:
        uc[0, :g] = hi - 1                                   # one heavy bundle
    res = P.tp_permutation(uc, arch, B, T, 16)
    _check_permutation(uc, arch, B, T, 16, res)
    loads = _bundle_loads(uc, arch, B, 16)
    opt = _optimum(loads, T, B // T)
    worst = max(res["rank_rows"])
    assert opt <= worst <= max(res["rank_rows_identity"])
    # placing items largest first onto the least loaded rank is optimal when no bundle
    # exceeds a third of the balanced load (the classic LPT bound is then tight here)
    total = sum(map(sum, loads))
    if max(map(max, loads)) * 3 <= total / T and B // T >= 2:
        assert worst <= opt + max(map(max, loads)) // 3
