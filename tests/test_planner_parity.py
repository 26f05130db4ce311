"""The C++ host planner (libdasc.so) against the plan oracle: bit-exact (CPU only)."""

import math

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import paper_2608_30386_amd as D
from oracle import plan as OP
from workloads import WORKLOADS, log_lambda


def _compare(sh, a_log, mode, k, w, T=1, conv=0, eps=1e-3):
    g_lib = D.dasc_static_log_decay(a_log)
    g_orc = OP.static_log_decay(a_log)
    assert g_lib.tobytes() == g_orc.tobytes(), "Eq. 2 differs in the last bit"
    lib = D.dasc_plan(sh, g_lib, mode, k, w, T, eps, conv)
    orc = OP.build_plan(g_orc, sh.arch, sh.n_layers, sh.n_heads, sh.dk, sh.dv, w, mode, k, eps, T, conv)
    assert lib["horizon"].tobytes() == orc["horizon"].tobytes()
    np.testing.assert_array_equal(lib["keep"], orc["keep"])
    for name in ("unit_count", "off", "layer_off", "layer_off_rows", "unit_row", "inv_row", "w_units",
                 "rank_begin", "send"):
        np.testing.assert_array_equal(lib[name], orc[name], err_msg=name)
    for name in ("n_rows", "n_units", "rows_per_unit", "w_replay", "slice_units", "slice_rows",
                 "r_max_rows", "slot_bytes_rank", "dense_slot_bytes_rank"):
        assert lib[name] == orc[name], name
    for name in ("c_temp_rag", "c_temp_pad", "layout_gain", "c_ckpt"):
        a, b = lib[name], orc[name]
        assert (math.isnan(a) and math.isnan(b)) or a == b, (name, a, b)
    return lib


@pytest.mark.parametrize("name", list(WORKLOADS))
def test_workload_plans_bit_exact(name):
    wl = WORKLOADS[name]
    sh = D.Shape(wl.arch, wl.n_layers, wl.n_heads, wl.n_qk_heads, wl.dk, wl.dv)
    p = _compare(sh, log_lambda(wl), wl.keep_mode, wl.keep_k, wl.w_max, wl.n_ranks)
    if name == "kimi_layer":
        assert p["n_rows"] == 1556                       # 38% of 4096 rows
    if name == "qwen_gdn":
        assert p["n_units"] == 36 * 12 and p["n_rows"] == 36 * 12 * 128
    if name == "kimi_model":
        from workloads.synth import planted_counts
        np.testing.assert_array_equal(p["unit_count"], planted_counts(wl))
        assert (p["unit_count"] == 0).any() and (p["unit_count"] == 128).any()


@settings(max_examples=40, deadline=None)
@given(arch=st.sampled_from(["kda", "gdn"]), L=st.integers(1, 4), H=st.sampled_from([1, 2, 4, 8]),
       dk=st.sampled_from([1, 3, 8, 16]), w=st.sampled_from([0, 4, 16, 64, 512, 1024, 5000]),
       mode=st.sampled_from(["threshold", "topk_head", "topk_layer"]),
       T=st.sampled_from([1, 2, 4, 8]), seed=st.integers(0, 2**31), ties=st.booleans())
def test_random_plans_bit_exact(arch, L, H, dk, w, mode, T, seed, ties):
    if arch == "gdn" and mode == "topk_head":
        mode = "topk_layer"
    rng = np.random.default_rng(seed)
    shape = (L, H, dk) if arch == "kda" else (L, H)
    a_log = rng.uniform(math.log(1e-4), math.log(2.0), size=shape)
    if ties:
        a_log = np.round(a_log, 0)                       # many equal horizons
    per = dk if mode == "topk_head" else (H * dk if arch == "kda" else H)
    k = int(rng.integers(0, per + 1))
    sh = D.Shape(arch, L, H, H, dk, 4)
    _compare(sh, a_log, mode, k, w, T, conv=int(rng.integers(0, 5000)))


def test_dense_plan_is_identity_map():
    sh = D.Shape("kda", 2, 4, 4, 8, 8)
    g = D.dasc_static_log_decay(np.full((2, 4, 8), -1.0))
    p = D.dasc_plan(sh, g, "threshold", 0, 0)
    np.testing.assert_array_equal(p["unit_row"], np.arange(64))
    np.testing.assert_array_equal(p["inv_row"], np.arange(64))
    assert p["w_replay"] == 0 and p["c_temp_rag"] == 1.0


def test_matched_slots_paper_budget():
    # App. C.1: 694,681,600 B per rank = 128 dense slots -> 127 deployable
    assert D.dasc_matched_slots(694_681_600, 694_681_600 // 128) == 127
    assert D.dasc_matched_slots(1_236_271_104, 1_236_271_104 // 128) == 127


def _compare_perm(sh, unit_count, T):
    lib = D.dasc_tp_permutation(sh, unit_count, T)
    orc = OP.tp_permutation(np.asarray(unit_count).reshape(sh.n_layers, sh.n_heads), sh.arch,
                            sh.n_qk_heads, T, sh.dk)
    for name in ("head_perm", "rank_rows", "rank_rows_identity"):
        np.testing.assert_array_equal(lib[name], orc[name], err_msg=name)
    return lib


@pytest.mark.parametrize("name,T", [("kimi_model", 8), ("kimi_model", 4), ("qwen_gdn", 8),
                                    ("kimi_layer", 8), ("tiny_kda", 2)])
def test_workload_tp_permutation_bit_exact(name, T):
    wl = WORKLOADS[name]
    sh = D.Shape(wl.arch, wl.n_layers, wl.n_heads, wl.n_qk_heads, wl.dk, wl.dv)
    plan = D.dasc_plan(sh, D.dasc_static_log_decay(log_lambda(wl)), wl.keep_mode, wl.keep_k,
                       wl.w_max, 1, wl.eps)
    res = _compare_perm(sh, plan["unit_count"], T)
    assert res["rank_rows"].sum() == res["rank_rows_identity"].sum() == plan["n_rows"]
    assert res["rank_rows"].max() <= res["rank_rows_identity"].max()


@settings(max_examples=60, deadline=None)
@given(arch=st.sampled_from(["kda", "gdn"]), L=st.integers(1, 5), B=st.sampled_from([1, 2, 4, 8]),
       g=st.sampled_from([1, 2, 3]), T=st.sampled_from([1, 2, 4, 8]), dk=st.sampled_from([1, 4, 16]),
       seed=st.integers(0, 2**31), ties=st.booleans())
def test_random_tp_permutation_bit_exact(arch, L, B, g, T, dk, seed, ties):
    if B % T:
        T = 1
    rng = np.random.default_rng(seed)
    H = B * g
    hi = dk if arch == "kda" else 1
    uc = rng.integers(0, hi + 1, size=(L, H))
    if ties:
        uc = np.full((L, H), hi // 2) + (rng.random((L, H)) < 0.1)
        uc = np.minimum(uc, hi)
    sh = D.Shape(arch, L, H, B, dk, 4)
    _compare_perm(sh, uc, T)


def test_rank_bottleneck_hand_worked_t4_library():
    # the hand-worked T = 4 case of the oracle pins, through the C ABI
    from tests.test_oracle_plan import HAND_T4, hand_t4_decay

    sh = D.Shape("kda", 1, 2, 2, 5, 4)
    p = D.dasc_plan(sh, hand_t4_decay(), "threshold", 0, 16, 4, 1e-3, 8)
    assert p["n_units"] == 7 and p["slice_units"] == HAND_T4["C"]
    np.testing.assert_array_equal(p["rank_begin"], HAND_T4["rank_begin"])
    np.testing.assert_array_equal(p["send"], HAND_T4["send"])
    assert p["slot_bytes_rank"] == HAND_T4["slot_bytes_rank"]
    assert p["dense_slot_bytes_rank"] == HAND_T4["dense_slot_bytes_rank"]
    assert p["c_ckpt"] == HAND_T4["c_ckpt"]
    assert D.dasc_matched_slots(4000, p["slot_bytes_rank"]) == HAND_T4["slots_4000"]
