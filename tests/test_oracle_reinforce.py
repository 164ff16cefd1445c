"""Pins of the rollout reward math oracle (Sec. 3.2): closed forms of the
discounted return and the EMA, library suffix sums, the RLOO invariants and a
finite-difference check of the loss derivative."""
import numpy as np
import pytest

from oracle import reinforce as orf


def _geometric(r, gamma, n):
    return r * n if gamma == 1.0 else r * (1.0 - gamma ** n) / (1.0 - gamma)


@pytest.mark.parametrize("gamma", [0.0, 0.5, 0.99, 1.0])
def test_constant_rewards_give_geometric_series(gamma):
    T, K = 37, 3
    R = np.full((T, K), -0.25)
    G = orf.discounted_returns(R, gamma)
    for t in range(T):
        assert np.allclose(G[t], _geometric(-0.25, gamma, T - t), rtol=1e-13, atol=1e-15)


def test_gamma_zero_and_one():
    R = np.random.default_rng(0).normal(size=(20, 4))
    assert np.array_equal(orf.discounted_returns(R, 0.0), R)
    suffix = np.flip(np.cumsum(np.flip(R, 0), 0), 0)
    assert np.allclose(orf.discounted_returns(R, 1.0), suffix, rtol=1e-13, atol=1e-13)


def test_rloo_invariants():
    rng = np.random.default_rng(1)
    R = rng.normal(size=(16, 6))
    lp = -rng.uniform(10, 100, size=(16, 6))
    out = orf.reinforce_terms(R, lp, 0.99, 0.01, 0.0, 0.9)
    # leave-one-out advantages sum to zero over the rollouts of a step
    assert np.allclose(out["advantage"].sum(1), 0.0, atol=1e-12)
    # baseline of rollout k excludes rollout k: changing G_k leaves b_k unchanged
    G = out["returns"].copy()
    G2 = G.copy()
    G2[:, 2] += 5.0
    assert np.allclose(orf.rloo_baseline(G2)[:, 2], orf.rloo_baseline(G)[:, 2])
    out2 = orf.reinforce_terms(R[:, :2], lp[:, :2], 0.99, 0.0, 0.0, 0.9)
    A = out2["advantage"]
    assert np.allclose(A[:, 0], out2["returns"][:, 0] - out2["returns"][:, 1])
    assert np.allclose(A[:, 0], -A[:, 1])


def test_single_rollout_uses_the_ema_and_the_ema_closed_form():
    rng = np.random.default_rng(2)
    R = rng.normal(size=(10, 1))
    out = orf.reinforce_terms(R, -np.ones((10, 1)), 0.9, 0.0, 0.3, 0.8)
    assert np.all(out["baseline"] == 0.3)
    m = out["returns"].mean()
    e = 0.3
    for n in range(1, 6):
        e = orf.reinforce_terms(R, -np.ones((10, 1)), 0.9, 0.0, e, 0.8)["ema"]
        assert abs(e - (0.8 ** n * 0.3 + (1 - 0.8 ** n) * m)) < 1e-13


def test_loss_derivative_by_finite_differences():
    rng = np.random.default_rng(3)
    R = rng.normal(size=(6, 3))
    lp = -rng.uniform(1, 5, size=(6, 3))
    base = orf.reinforce_terms(R, lp, 0.95, 0.05, 0.0, 0.9)
    h = 1e-6
    for t, k in [(0, 0), (3, 1), (5, 2)]:
        lp2 = lp.copy()
        lp2[t, k] += h
        d = (orf.reinforce_terms(R, lp2, 0.95, 0.05, 0.0, 0.9)["loss"] - base["loss"]) / h
        assert abs(d - base["weight"][t, k]) < 1e-8
    # the entropy surrogate is the mean of -log pi
    assert abs(base["entropy"] + lp.mean()) < 1e-13
