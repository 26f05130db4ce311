"""GPU parity at the full-model size and in the launch configuration the bench times:
24 KDA layers x 32 heads, 256 checkpoints, T = 8 rank slices, plus the INT8 and
padded layouts on the same states.  Every one of the 256 checkpoints is checked word for
word against the oracle, slot by slot (the oracle packs and restores each source state
on the host)."""

import numpy as np
import pytest

import paper_2608_30386_amd as D
from oracle import pack as OK
from oracle import quant as OQ
from tests.gpu_util import announce, dev_i32, plans, shape_of
from workloads import WORKLOADS, states_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def model():
    wl = WORKLOADS["kimi_model"]
    lib, _ = plans(wl)
    sh = shape_of(wl)
    n = wl.n_ckpt
    announce(f"full-model states {n} x {sh.rows} rows")
    states = states_device(wl, n, "cuda")
    src = np.arange(n)
    dst = (src * 101 + 7) % n                          # a permutation of the checkpoint slots
    back = (src * 37 + 11) % n                         # and of the pool slots
    yield wl, lib, sh, states, src, dst, back
    del states


def _host_state(states, i, rows, dv):
    return states[i].reshape(1, rows, dv).cpu().numpy()


def test_full_model_ragged_sliced_every_checkpoint(model):
    import torch

    wl, lib, sh, states, src, dst, back = model
    n, T, R, C, dv, rows = wl.n_ckpt, wl.n_ranks, int(lib["n_rows"]), int(lib["slice_rows"]), wl.dv, sh.rows
    ckpt = torch.full((T, n, C, dv), -7.0, device="cuda")
    announce(f"pack n={n} T={T} R={R}")
    D.dasc_pack(sh, states, dev_i32(src), dev_i32(lib["unit_row"]), ckpt, dev_i32(dst), n_ranks=T,
                slice_rows=C)
    active = torch.full_like(states, 3.0)
    announce("restore")
    D.dasc_restore(sh, ckpt, dev_i32(dst), dev_i32(lib["inv_row"]), active, dev_i32(back), n_rows=R,
                   n_ranks=T, slice_rows=C)
    torch.cuda.synchronize()
    blank = np.full((T, 1, C, dv), np.float32(-7.0).view(np.uint32))
    for i in range(n):
        words = _host_state(states, i, rows, dv).view(np.uint32)
        want = OK.pack(words, [0], lib["unit_row"], blank, [0], slice_rows=C)
        got = ckpt[:, int(dst[i])].cpu().numpy().view(np.uint32)
        assert np.array_equal(got, want[:, 0]), f"pack of checkpoint {i} differs"
        want_r = OK.restore(want, [0], lib["unit_row"], np.zeros((1, rows, dv), np.uint32), [0],
                            slice_rows=C)
        got_r = active[int(back[i])].reshape(rows, dv).cpu().numpy().view(np.uint32)
        assert np.array_equal(got_r, want_r[0]), f"restore of checkpoint {i} differs"
    announce(f"full-model ragged T={T}: all {n} checkpoints bit-exact")


def test_full_model_int8_every_checkpoint(model):
    import torch

    wl, lib, sh, states, src, dst, back = model
    n, R, dv, rows = wl.n_ckpt, int(lib["n_rows"]), wl.dv, sh.rows
    q = torch.full((n, R, dv), 77, dtype=torch.int8, device="cuda")
    s = torch.full((n, R), -1.0, device="cuda")
    active = torch.full_like(states, 3.0)
    announce(f"pack_q8 / restore_q8 n={n}")
    D.dasc_pack_q8(sh, states, dev_i32(src), dev_i32(lib["unit_row"]), q, s, dev_i32(dst))
    D.dasc_restore_q8(sh, q, s, dev_i32(dst), dev_i32(lib["inv_row"]), active, dev_i32(back), n_rows=R)
    torch.cuda.synchronize()
    for i in range(n):
        x = _host_state(states, i, rows, dv)
        wq, ws = OQ.pack_q8(x, [0], lib["unit_row"])
        assert np.array_equal(q[int(dst[i])].cpu().numpy(), wq[0]), f"codes of checkpoint {i} differ"
        assert np.array_equal(s[int(dst[i])].cpu().numpy().view(np.uint32), ws[0].view(np.uint32)), \
            f"scales of checkpoint {i} differ"
        want = OQ.restore_q8(wq, ws, lib["unit_row"], rows)
        got = active[int(back[i])].reshape(rows, dv).cpu().numpy()
        assert np.array_equal(got.view(np.uint32), want[0].view(np.uint32)), f"restore_q8 {i} differs"
    announce(f"full-model INT8: all {n} checkpoints bit-exact (codes, scales, restored words)")


def test_full_model_padded_every_checkpoint(model):
    import torch

    wl, lib, sh, states, src, dst, back = model
    n, R, dv, rows = wl.n_ckpt, int(lib["n_rows"]), wl.dv, sh.rows
    off_rows, r_max = lib["layer_off_rows"], int(lib["r_max_rows"])
    ck_pad = torch.full((sh.n_layers, n, r_max, dv), -5.0, device="cuda")
    active = torch.full_like(states, 3.0)
    announce(f"pack_padded / restore_padded n={n} r_max={r_max}")
    D.dasc_pack_padded(sh, states, dev_i32(src), dev_i32(lib["unit_row"]), dev_i32(off_rows), ck_pad,
                       dev_i32(dst))
    D.dasc_restore_padded(sh, ck_pad, dev_i32(dst), dev_i32(off_rows), dev_i32(lib["inv_row"]), active,
                          dev_i32(back), n_rows=R)
    torch.cuda.synchronize()
    off_units, rpu = lib["layer_off"], int(lib["rows_per_unit"])
    blank = np.full((sh.n_layers, 1, r_max, dv), np.float32(-5.0).view(np.uint32))
    for i in range(n):
        words = _host_state(states, i, rows, dv).view(np.uint32)
        want = OK.pack_padded(words, [0], lib["unit_row"], off_units, rpu, blank, [0])
        got = ck_pad[:, int(dst[i])].cpu().numpy().view(np.uint32)
        assert np.array_equal(got, want[:, 0]), f"padded pack of checkpoint {i} differs"
        want_r = OK.restore_padded(want, [0], lib["unit_row"], off_units, rpu,
                                   np.zeros((1, rows, dv), np.uint32), [0])
        got_r = active[int(back[i])].reshape(rows, dv).cpu().numpy().view(np.uint32)
        assert np.array_equal(got_r, want_r[0]), f"padded restore of checkpoint {i} differs"
    announce(f"full-model padded: all {n} checkpoints bit-exact")
