"""Pins for the recurrence oracle (CPU only).

Each pin is a fact the paper's Eq. 1 or plain algebra fixes, chosen so that a
plausible slip (dropped decay, erase before decay, wrong sign, transposed
operand, wrong key head) fails at least one of them.
"""

import numpy as np
import pytest

from oracle import recurrence as R


def _inputs(rng, B, W, dk, dv, per_channel=True, lam_hi=1.0):
    k = rng.standard_normal((B, W, dk))
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((B, W, dv))
    lam = np.exp(rng.uniform(np.log(1e-3), np.log(lam_hi), size=(B, 1, dk if per_channel else 1)))
    z = rng.standard_normal((B, W, dk if per_channel else 1))
    g = -lam * np.logaddexp(0, z)
    if not per_channel:
        g = g[..., 0]
    beta = 1 / (1 + np.exp(-rng.standard_normal((B, W))))
    S0 = 0.1 * rng.standard_normal((B, dk, dv))
    return S0, k, v, g, beta


def test_beta_zero_is_pure_decay():
    rng = np.random.default_rng(0)
    S0, k, v, g, _ = _inputs(rng, 3, 9, 6, 5)
    beta = np.zeros((3, 9))
    want = np.exp(g.sum(axis=1))[:, :, None] * S0          # Diag(prod alpha) S_0
    for f in (R.replay_naive, lambda *a: R.replay_chunked(*a, chunk=4)):
        np.testing.assert_allclose(f(S0, k, v, g, beta), want, rtol=1e-13, atol=1e-15)


def test_alpha_one_beta_zero_is_identity():
    rng = np.random.default_rng(1)
    S0, k, v, g, _ = _inputs(rng, 2, 7, 4, 4)
    out = R.replay_naive(S0, k, v, np.zeros_like(g), np.zeros((2, 7)))
    np.testing.assert_array_equal(out, S0)


def test_unit_beta_unit_key_reads_back_value():
    # beta_t = 1, |k_t| = 1: the write makes S_t^T k_t = v_t exactly (after decay).
    # Fails if erase came before decay or the erase sign flipped.
    rng = np.random.default_rng(2)
    S0, k, v, g, _ = _inputs(rng, 4, 6, 8, 5)
    beta = np.ones((4, 6))
    for W in range(1, 7):
        S = R.replay_naive(S0, k[:, :W], v[:, :W], g[:, :W], beta[:, :W])
        got = np.einsum("bc,bcj->bj", k[:, W - 1], S)
        np.testing.assert_allclose(got, v[:, W - 1], rtol=0, atol=1e-13)


def test_orthonormal_keys_closed_form():
    # alpha = 1 and orthonormal keys: S_W = (I - sum beta_s k_s k_s^T) S_0 + sum beta_s k_s v_s^T
    rng = np.random.default_rng(3)
    dk, dv, W = 8, 5, 6
    Q, _ = np.linalg.qr(rng.standard_normal((dk, dk)))
    k = Q[:, :W].T[None]                                    # W orthonormal keys
    v = rng.standard_normal((1, W, dv))
    beta = rng.uniform(0.1, 0.9, size=(1, W))
    S0 = rng.standard_normal((1, dk, dv))
    P = sum(beta[0, s] * np.outer(k[0, s], k[0, s]) for s in range(W))
    O = sum(beta[0, s] * np.outer(k[0, s], v[0, s]) for s in range(W))
    want = (np.eye(dk) - P) @ S0[0] + O
    g0 = np.zeros((1, W, dk))
    for f in (R.replay_naive, lambda *a: R.replay_chunked(*a, chunk=4)):
        np.testing.assert_allclose(f(S0, k, v, g0, beta)[0], want, atol=1e-13)
    # from a zero state it is a plain outer-product sum
    np.testing.assert_allclose(R.replay_naive(np.zeros_like(S0), k, v, g0, beta)[0], O, atol=1e-14)


def test_paper_orientation_matches_transposed_form():
    # Eq. 1 written literally on [dv, dk] equals the transposed per-token form
    rng = np.random.default_rng(4)
    for dk, dv, W in [(1, 1, 3), (2, 3, 5), (4, 4, 8), (3, 2, 7)]:
        S0, k, v, g, beta = _inputs(rng, 2, W, dk, dv)
        a = R.replay_paper_form(np.swapaxes(S0, -1, -2), k, v, g, beta)
        b = R.replay_naive(S0, k, v, g, beta)
        np.testing.assert_allclose(np.swapaxes(a, -1, -2), b, rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("chunk", [1, 3, 8, 16, 64])
@pytest.mark.parametrize("per_channel", [True, False])
def test_chunked_equals_naive(chunk, per_channel):
    rng = np.random.default_rng(5)
    S0, k, v, g, beta = _inputs(rng, 3, 37, 16, 12, per_channel=per_channel)   # ragged tail
    a = R.replay_chunked(S0, k, v, g, beta, chunk=chunk)
    b = R.replay_naive(S0, k, v, g, beta)
    assert np.abs(a - b).max() <= 1e-12 * np.abs(b).max()


def test_chunked_strong_decay_no_overflow():
    # per-token log-gates near -5 over 64 tokens: exp(G) spans e^-320; still finite & equal
    rng = np.random.default_rng(6)
    S0, k, v, _, beta = _inputs(rng, 2, 64, 8, 8)
    g = -rng.uniform(3.0, 5.5, size=(2, 64, 8))
    a = R.replay_chunked(S0, k, v, g, beta, chunk=64)
    b = R.replay_naive(S0, k, v, g, beta)
    assert np.all(np.isfinite(a))
    assert np.abs(a - b).max() <= 1e-12 * np.abs(b).max()


def test_channel_constant_kda_equals_gdn():
    rng = np.random.default_rng(7)
    S0, k, v, g, beta = _inputs(rng, 2, 11, 6, 4, per_channel=False)
    g_kda = np.repeat(g[..., None], 6, axis=-1)
    np.testing.assert_allclose(R.replay_naive(S0, k, v, g_kda, beta),
                               R.replay_naive(S0, k, v, g, beta), rtol=1e-14, atol=0)


def test_value_columns_evolve_independently_and_homogeneity():
    rng = np.random.default_rng(8)
    S0, k, v, g, beta = _inputs(rng, 2, 13, 8, 6)
    full = R.replay_naive(S0, k, v, g, beta)
    part = R.replay_naive(S0[..., 2:5], k, v[..., 2:5], g, beta)
    np.testing.assert_allclose(part, full[..., 2:5], rtol=1e-14, atol=1e-16)
    c = -2.5
    np.testing.assert_allclose(R.replay_naive(c * S0, k, c * v, g, beta), c * full, rtol=1e-13, atol=1e-15)


def test_refresh_writes_only_omitted_rows_and_shares_key_heads():
    rng = np.random.default_rng(9)
    n_req, H, Hqk, W, dk, dv = 2, 4, 2, 10, 4, 4
    st = rng.standard_normal((n_req, H, dk, dv)).astype(np.float32)
    inv = np.arange(H * dk)
    inv[[1, 2, 9]] = -1                       # head 0 rows 1,2 and head 2 row 1 omitted
    kf = rng.standard_normal((n_req, Hqk, W, dk)).astype(np.float32)
    from workloads import bf16_bits_from_f32
    kb = bf16_bits_from_f32(kf)
    vb = bf16_bits_from_f32(rng.standard_normal((n_req, H, W, dv)).astype(np.float32))
    g = (-0.3 * rng.uniform(0, 2, size=(n_req, H, W, dk))).astype(np.float32)
    beta = rng.uniform(0, 1, size=(n_req, H, W)).astype(np.float32)
    out, om = R.refresh(st, inv, kb, vb, g, beta, n_qk_heads=Hqk)
    out = out.reshape(n_req, H, dk, dv)
    kept = ~om
    for n in range(n_req):
        for h in range(H):
            np.testing.assert_array_equal(out[n, h][kept[h]], st[n, h][kept[h]].astype(np.float64))
    # heads 1 and 3 have nothing omitted: untouched
    np.testing.assert_array_equal(out[:, [1, 3]], st[:, [1, 3]])
    # grouped key heads == the same keys duplicated per value head
    kdup = np.repeat(kb, H // Hqk, axis=1)
    out2 = R.refresh(st, inv, kdup, vb, g, beta, n_qk_heads=H)[0].reshape(out.shape)
    np.testing.assert_array_equal(out, out2)
    # value head 2 must read key head 1: swapping key heads changes it
    out3 = R.refresh(st, inv, kb[:, ::-1], vb, g, beta, n_qk_heads=Hqk)[0].reshape(out.shape)
    assert not np.allclose(out3[:, 2], out[:, 2])


def test_refresh_gdn_zero_init_equals_restored():
    # an omitted GDN head restores as zeros, so both start states agree
    rng = np.random.default_rng(10)
    n_req, H, Hqk, W, dk, dv = 2, 4, 2, 9, 4, 4
    st = rng.standard_normal((n_req, H, dk, dv)).astype(np.float32)
    inv = np.arange(H * dk)
    inv[4:8] = -1
    st[:, 1] = 0.0
    from workloads import bf16_bits_from_f32
    kb = bf16_bits_from_f32(rng.standard_normal((n_req, Hqk, W, dk)).astype(np.float32))
    vb = bf16_bits_from_f32(rng.standard_normal((n_req, H, W, dv)).astype(np.float32))
    g = (-rng.uniform(0, 1, size=(n_req, H, W))).astype(np.float32)
    beta = rng.uniform(0, 1, size=(n_req, H, W)).astype(np.float32)
    a, _ = R.refresh(st, inv, kb, vb, g, beta, Hqk, init="restored")
    b, _ = R.refresh(st, inv, kb, vb, g, beta, Hqk, init="zero")
    np.testing.assert_array_equal(a, b)
