"""Pins of the training-side gather-scatter oracle (Section 3.2, Eq. 6-7,
Appendix B) against brute force, closed forms, adjointness and finite
differences."""
import numpy as np
import pytest

from oracle import gather_scatter as gs


def _depths(rng, rows, R):
    return rng.integers(1, R + 1, size=rows).astype(np.int32)


def test_active_set_brute_force():
    rng = np.random.default_rng(11)
    B, T, R = 3, 7, 4
    m = _depths(rng, B * T, R)
    for i in range(0, R + 2):
        rows = [r for r in range(B * T) if m[r] >= i]
        assert gs.active_rows(m, i).tolist() == rows
        slot = gs.compact_slot(m, i)
        for r in range(B * T):
            assert slot[r] == (rows.index(r) if r in rows else -1)
        off = [0]
        for b in range(B):
            off.append(off[-1] + sum(1 for t in range(T) if m[b * T + t] >= i))
        assert gs.sequence_offsets(m, T, i).tolist() == off


def test_active_set_keeps_sequences_causal():
    rng = np.random.default_rng(12)
    B, T, R = 5, 33, 8
    m = _depths(rng, B * T, R)
    for i in range(1, R + 1):
        idx = gs.active_rows(m, i)
        off = gs.sequence_offsets(m, T, i)
        for b in range(B):
            seg = idx[off[b]:off[b + 1]]
            assert np.all(seg // T == b)
            assert np.all(np.diff(seg) > 0)


def test_edge_cases():
    assert gs.active_rows(np.zeros(0, np.int32), 1).shape == (0,)
    m = np.array([1, 1, 1], np.int32)
    assert gs.active_rows(m, 2).shape == (0,)
    assert gs.active_rows(m, 1).tolist() == [0, 1, 2]
    H = np.arange(6.0).reshape(3, 2)
    # no active rows: the scatter is the identity
    assert np.array_equal(gs.scatter(H, np.zeros((0, 2)), np.zeros(0, np.int64)), H)


def test_gather_scatter_is_lossless_for_rowwise_block():
    """A row-wise block on the compact rows, scattered back, equals the dense
    update masked to the active rows (the compression loses nothing)."""
    rng = np.random.default_rng(13)
    rows, d, R = 50, 6, 5
    m = _depths(rng, rows, R)
    H = rng.standard_normal((rows, d))
    A = rng.standard_normal((d, d))
    for i in range(1, R + 1):
        idx = gs.active_rows(m, i)
        got = gs.scatter(H, np.tanh(gs.gather(H, idx) @ A), idx)
        mask = (m >= i).astype(np.float64)[:, None]
        want = H + mask * np.tanh(H @ A)
        np.testing.assert_allclose(got, want, rtol=0, atol=1e-14)


def test_loops_closed_form():
    """Block output c_i for every active row: after R loops a token of depth m
    holds h0 + c_1 + ... + c_min(m, R)."""
    rng = np.random.default_rng(14)
    rows, d, R = 40, 3, 6
    m = _depths(rng, rows, R + 2)
    H0 = rng.standard_normal((rows, d))
    c = rng.standard_normal((R + 1, d))
    got = gs.loop_forward(H0, m, lambda i, X: np.broadcast_to(c[i], X.shape), R)
    for r in range(rows):
        want = H0[r] + c[1:min(int(m[r]), R) + 1].sum(axis=0)
        np.testing.assert_allclose(got[r], want, rtol=0, atol=1e-13)


def test_adjointness():
    rng = np.random.default_rng(15)
    rows, d = 30, 4
    m = _depths(rng, rows, 4)
    idx = gs.active_rows(m, 3)
    H = rng.standard_normal((rows, d))
    G = rng.standard_normal((idx.shape[0], d))
    lhs = np.sum(gs.gather(H, idx) * G)
    rhs = np.sum(H * gs.gather_backward(G, idx, rows))
    assert abs(lhs - rhs) < 1e-12
    Y = rng.standard_normal((idx.shape[0], d))
    dH = rng.standard_normal((rows, d))
    dprev, dY = gs.scatter_backward(dH, idx)
    assert abs(np.sum(gs.scatter(H, Y, idx) * dH) - (np.sum(H * dprev) + np.sum(Y * dY))) < 1e-12


def test_backward_matches_finite_differences():
    """dL/dH0 through three loops of a nonlinear row-wise block, composed from
    the backward pieces, against central differences."""
    rng = np.random.default_rng(16)
    rows, d, R = 12, 3, 3
    m = _depths(rng, rows, R)
    A = rng.standard_normal((d, d)) * 0.7
    W = rng.standard_normal((rows, d))
    H0 = rng.standard_normal((rows, d))

    def block(i, X):
        return np.tanh(X @ A)

    def loss(H):
        return float(np.sum(W * gs.loop_forward(H, m, block, R)))

    # forward, keeping each loop's compact input
    H, saved = H0, []
    for i in range(1, R + 1):
        idx = gs.active_rows(m, i)
        X = gs.gather(H, idx)
        saved.append((idx, X))
        H = gs.scatter(H, block(i, X), idx)
    dH = W.copy()
    for idx, X in reversed(saved):
        dprev, dY = gs.scatter_backward(dH, idx)
        dX = (dY * (1.0 - np.tanh(X @ A) ** 2)) @ A.T
        dH = dprev + gs.gather_backward(dX, idx, rows)
    eps = 1e-6
    fd = np.zeros_like(H0)
    for r in range(rows):
        for k in range(d):
            e = np.zeros_like(H0)
            e[r, k] = eps
            fd[r, k] = (loss(H0 + e) - loss(H0 - e)) / (2 * eps)
    np.testing.assert_allclose(dH, fd, rtol=1e-6, atol=1e-8)


def test_ste():
    rng = np.random.default_rng(17)
    s = rng.standard_normal(64) * 3
    g = rng.standard_normal(64)
    m = rng.integers(1, 9, 64)
    assert np.array_equal(gs.ste_value(m), m.astype(np.float64))
    eps = 1e-6
    fd = g * (gs.sigmoid(s + eps) - gs.sigmoid(s - eps)) / (2 * eps)
    np.testing.assert_allclose(gs.ste_grad(s, g), fd, rtol=1e-7, atol=1e-12)
    # sigma'(0) = 1/4; far tails vanish
    assert gs.ste_grad(np.zeros(1), np.ones(1))[0] == pytest.approx(0.25, abs=0)
    assert gs.ste_grad(np.array([40.0, -40.0]), np.ones(2)).max() < 1e-16
    # far tails keep full relative precision: sigma'(s) ~ exp(-|s|)
    far = gs.ste_grad(np.array([60.0, -60.0]), np.ones(2))
    np.testing.assert_allclose(far, np.exp(-60.0) * np.ones(2), rtol=1e-12)
