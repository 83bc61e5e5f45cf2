"""Pins of the oracle's LoRE calibration fit (Eq. 10): the minimiser of
sum_t || y_t - B A x_t ||^2 over rank-r maps, checked against planted maps, the exact-fit
case r >= n, Eckart-Young's closed-form loss, monotonicity in r, stationarity, and
random perturbations."""
import numpy as np
import pytest


def _planted(r_, n, d, rank, seed, noise=0.0):
    X = r_.standard_normal((n, d))
    W0 = r_.standard_normal((d, rank)) @ r_.standard_normal((rank, d))
    Y = X @ W0.T + noise * r_.standard_normal((n, d))
    return X, Y, W0


def test_planted_map_is_recovered_with_enough_tokens(orc):
    r_ = np.random.default_rng(0)
    X, Y, W0 = _planted(r_, 60, 24, 5, 0)
    A, B, loss = orc.lore_fit(X, Y, 5)
    assert A.shape == (5, 24) and B.shape == (24, 5)
    assert loss < 1e-18 * (Y * Y).sum()
    assert np.abs(B @ A - W0).max() < 1e-9 * np.abs(W0).max()


def test_planted_map_with_fewer_tokens_fits_exactly_with_minimum_norm(orc):
    r_ = np.random.default_rng(1)
    X, Y, W0 = _planted(r_, 15, 40, 4, 1)
    A, B, loss = orc.lore_fit(X, Y, 4)
    W = B @ A
    assert loss < 1e-18 * (Y * Y).sum()
    assert np.allclose(X @ W.T, Y, atol=1e-9 * np.abs(Y).max())
    P = np.linalg.pinv(X) @ X  # projector on the tokens' row space
    assert np.allclose(W @ P, W, atol=1e-9 * np.abs(W).max())
    assert np.linalg.norm(W) <= np.linalg.norm(W0) + 1e-9


@pytest.mark.parametrize("n,d", [(12, 30), (30, 30)])
def test_rank_at_least_n_fits_any_residual(orc, n, d):
    r_ = np.random.default_rng(2)
    X, Y = r_.standard_normal((n, d)), r_.standard_normal((n, d))
    for r in (n, n + 3):
        _, _, loss = orc.lore_fit(X, Y, min(r, d))
        assert loss < 1e-18 * (Y * Y).sum()


def test_loss_is_the_tail_of_the_residual_spectrum(orc):
    """n <= d with X of full rank: every target is reachable, so the best rank-r loss is the
    sum of the squared singular values of Y beyond the r-th (Eckart-Young)."""
    r_ = np.random.default_rng(3)
    n, d = 20, 48
    X = r_.standard_normal((n, d))
    Y = r_.standard_normal((n, d)) * np.linspace(3, 0.1, d)
    ev = np.sort(np.linalg.eigvalsh(Y @ Y.T))[::-1]  # sigma_i(Y)^2
    for r in (1, 4, 9, 19):
        _, _, loss = orc.lore_fit(X, Y, r)
        assert abs(loss - ev[r:].sum()) <= 1e-9 * ev.sum()


def test_loss_does_not_increase_with_rank(orc):
    r_ = np.random.default_rng(4)
    X, Y, _ = _planted(r_, 70, 32, 12, 4, noise=0.3)
    losses = [orc.lore_fit(X, Y, r)[2] for r in range(0, 33, 2)]
    assert all(b <= a * (1 + 1e-12) + 1e-12 for a, b in zip(losses, losses[1:]))
    assert losses[0] == pytest.approx((Y * Y).sum(), rel=1e-12)


def test_fit_is_a_stationary_point_and_beats_perturbations(orc):
    r_ = np.random.default_rng(5)
    X, Y, _ = _planted(r_, 80, 24, 10, 5, noise=0.5)
    r = 4
    A, B, loss = orc.lore_fit(X, Y, r)
    R = Y.T - B @ (A @ X.T)
    gA = -2 * B.T @ R @ X
    gB = -2 * R @ (A @ X.T).T
    scale = np.abs(Y).max() * np.abs(X).max() * X.shape[0]
    assert np.abs(gA).max() < 1e-8 * scale and np.abs(gB).max() < 1e-8 * scale
    assert loss == pytest.approx(orc.lore_loss(X, Y, A, B), rel=1e-12)
    for _ in range(20):
        dA = r_.standard_normal(A.shape) * 1e-3
        dB = r_.standard_normal(B.shape) * 1e-3
        assert orc.lore_loss(X, Y, A + dA, B + dB) >= loss


def test_token_order_does_not_matter(orc):
    r_ = np.random.default_rng(6)
    X, Y, _ = _planted(r_, 50, 20, 6, 6, noise=0.2)
    p = r_.permutation(50)
    A, B, l1 = orc.lore_fit(X, Y, 3)
    A2, B2, l2 = orc.lore_fit(X[p], Y[p], 3)
    assert l1 == pytest.approx(l2, rel=1e-10)
    assert np.allclose(B @ A, B2 @ A2, atol=1e-9 * np.abs(B @ A).max())
