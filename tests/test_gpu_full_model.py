"""GPU parity at the full-model size and in the launch configuration the bench times:
24 KDA layers x 32 heads, 256 checkpoints, T = 8 rank slices, plus the INT8 and
padded layouts on the same states, checked word for word against the oracle on sampled checkpoints."""

import numpy as np
import pytest

import paper_2608_30386_amd as D
from oracle import pack as OK
from oracle import quant as OQ
from tests.gpu_util import announce, dev_i32, plans, shape_of
from workloads import WORKLOADS, states_device

pytestmark = pytest.mark.gpu

SAMPLES = (0, 37, 128, 201, 255)


def test_full_model_pack_restore_all_layouts():
    import torch

    wl = WORKLOADS["kimi_model"]
    lib, _ = plans(wl)
    sh = shape_of(wl)
    n, T, R, C, dv = wl.n_ckpt, wl.n_ranks, int(lib["n_rows"]), int(lib["slice_rows"]), wl.dv
    rows = sh.rows
    announce(f"full-model states {n} x {rows} rows")
    states = states_device(wl, n, "cuda")
    src = np.arange(n)
    dst = (src * 101 + 7) % n                          # a permutation of the slots
    back = (src * 37 + 11) % n
    ckpt = torch.full((T, n, C, dv), -7.0, device="cuda")
    announce(f"pack n={n} T={T} R={R}")
    D.dasc_pack(sh, states, dev_i32(src), dev_i32(lib["unit_row"]), ckpt, dev_i32(dst), n_ranks=T,
                slice_rows=C)
    active = torch.full_like(states, 3.0)
    announce("restore")
    D.dasc_restore(sh, ckpt, dev_i32(dst), dev_i32(lib["inv_row"]), active, dev_i32(back), n_rows=R,
                   n_ranks=T, slice_rows=C)
    torch.cuda.synchronize()
    for i in SAMPLES:
        words = states[i].reshape(1, rows, dv).cpu().numpy().view(np.uint32)
        want = OK.pack(words, [0], lib["unit_row"], np.full((T, 1, C, dv), np.float32(-7.0).view(np.uint32)),
                       [0], slice_rows=C)
        got = ckpt[:, int(dst[i])].cpu().numpy().view(np.uint32)
        assert np.array_equal(got, want[:, 0]), f"pack of checkpoint {i} differs"
        want_r = OK.restore(want, [0], lib["unit_row"], np.zeros((1, rows, dv), np.uint32), [0],
                            slice_rows=C)
        got_r = active[int(back[i])].reshape(rows, dv).cpu().numpy().view(np.uint32)
        assert np.array_equal(got_r, want_r[0]), f"restore of checkpoint {i} differs"
    del ckpt

    q = torch.full((n, R, dv), 77, dtype=torch.int8, device="cuda")
    s = torch.full((n, R), -1.0, device="cuda")
    announce(f"pack_q8 / restore_q8 n={n}")
    D.dasc_pack_q8(sh, states, dev_i32(src), dev_i32(lib["unit_row"]), q, s, dev_i32(dst))
    D.dasc_restore_q8(sh, q, s, dev_i32(dst), dev_i32(lib["inv_row"]), active, dev_i32(back), n_rows=R)
    torch.cuda.synchronize()
    for i in SAMPLES:
        x = states[i].reshape(1, rows, dv).cpu().numpy()
        wq, ws = OQ.pack_q8(x, [0], lib["unit_row"])
        assert np.array_equal(q[int(dst[i])].cpu().numpy(), wq[0]), f"codes of checkpoint {i} differ"
        assert np.array_equal(s[int(dst[i])].cpu().numpy().view(np.uint32), ws[0].view(np.uint32))
        want = OQ.restore_q8(wq, ws, lib["unit_row"], rows)
        got = active[int(back[i])].reshape(rows, dv).cpu().numpy()
        assert np.array_equal(got.view(np.uint32), want[0].view(np.uint32)), f"restore_q8 {i} differs"
    del q, s

    off_rows, r_max = lib["layer_off_rows"], int(lib["r_max_rows"])
    ck_pad = torch.full((sh.n_layers, n, r_max, dv), -5.0, device="cuda")
    announce(f"pack_padded / restore_padded n={n} r_max={r_max}")
    D.dasc_pack_padded(sh, states, dev_i32(src), dev_i32(lib["unit_row"]), dev_i32(off_rows), ck_pad,
                       dev_i32(dst))
    D.dasc_restore_padded(sh, ck_pad, dev_i32(dst), dev_i32(off_rows), dev_i32(lib["inv_row"]), active,
                          dev_i32(back), n_rows=R)
    torch.cuda.synchronize()
    off_units, rpu = lib["layer_off"], int(lib["rows_per_unit"])
    for i in SAMPLES:
        words = states[i].reshape(1, rows, dv).cpu().numpy().view(np.uint32)
        blank = np.full((sh.n_layers, 1, r_max, dv), np.float32(-5.0).view(np.uint32))
        want = OK.pack_padded(words, [0], lib["unit_row"], off_units, rpu, blank, [0])
        got = ck_pad[:, int(dst[i])].cpu().numpy().view(np.uint32)
        assert np.array_equal(got, want[:, 0]), f"padded pack of checkpoint {i} differs"
        want_r = OK.restore_padded(want, [0], lib["unit_row"], off_units, rpu,
                                   np.zeros((1, rows, dv), np.uint32), [0])
        got_r = active[int(back[i])].reshape(rows, dv).cpu().numpy().view(np.uint32)
        assert np.array_equal(got_r, want_r[0]), f"padded restore of checkpoint {i} differs"
    announce(f"full-model pack/restore/q8/padded bit-exact on checkpoints {SAMPLES}")
