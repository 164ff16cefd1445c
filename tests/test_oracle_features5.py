"""Pins of the fifth feature sigma_i (Sec. 3.1.1: variance of the attention
mass across heads) and of the LayerNorm MLP variant (App. D), against closed
forms and hand-worked values."""
import math

import numpy as np

from oracle import features as of
from oracle import policy as op
from oracle import unit as ounit


def test_head_variance_closed_forms():
    a = np.array([[0.1, 0.5, 0.25], [0.3, 0.5, 0.75]])
    # two heads: ((a - b) / 2)^2
    assert np.allclose(of.head_variance(a), ((a[0] - a[1]) / 2) ** 2, rtol=0, atol=1e-15)
    # one head, or identical heads: zero
    assert np.all(of.head_variance(a[:1]) == 0)
    assert np.all(of.head_variance(np.tile(a[:1], (4, 1))) == 0)
    # three heads by hand: (0.1, 0.2, 0.6) has mean 0.3 and variance 0.14 / 3
    v = of.head_variance(np.array([[0.1], [0.2], [0.6]]))
    assert abs(v[0] - 0.14 / 3) < 1e-15


def test_five_feature_order():
    L = 4
    x = of.feature_matrix5(np.full(L, 1.0), np.zeros((L, 2)), np.full(L, 7.0), np.zeros(L),
                           np.zeros(L), np.arange(L), 8)
    assert x.shape == (L, 5)
    assert np.all(x[:, 0] == 1.0) and np.all(x[:, 1] == 0) and np.all(x[:, 2] == 7.0)
    assert np.all(x[:, 3] == 0) and np.allclose(x[:, 4], np.arange(L) / 8)


def test_unit_records_sigma_of_the_last_step():
    rng = np.random.default_rng(0)
    K, V = rng.normal(size=(20, 8)), rng.normal(size=(20, 8))
    st = ounit.new_student(K, V, np.arange(20), G=2, scale=0.5, window=4)
    q = rng.normal(size=(2, 8))
    att = ounit.decode_step(st, q, rng.normal(size=8), rng.normal(size=8))
    assert st.sigma.shape == (21,)
    assert np.allclose(st.sigma, ((att.a[0] - att.a[1]) / 2) ** 2, rtol=0, atol=1e-18)
    kept = ounit.evict(st, -np.arange(21.0), 10)
    assert np.allclose(st.sigma, ((att.a[0] - att.a[1]) / 2)[kept] ** 2, rtol=0, atol=1e-18)


def _blob(W1, b1, g1, be1, wo, bo):
    return np.concatenate([np.ravel(W1), b1, g1, be1, wo, [bo]])


def test_layer_norm_two_units_by_hand():
    # x = (1, 0, 0, 0): z = (1, 3); mean 2, variance 1; normalised (-1, 1) / sqrt(1 + eps)
    W1 = np.array([[1.0, 0, 0, 0], [3.0, 0, 0, 0]])
    p = _blob(W1, [0.0, 0.0], [1.0, 1.0], [0.0, 0.0], [1.0, 1.0], 0.0)
    s = op.scores(p, [[1.0, 0, 0, 0]], (2,), layer_norm=True)
    assert abs(s[0] - 1.0 / math.sqrt(1.0 + 1e-5)) < 1e-15
    # gain and bias act after the normalisation
    p2 = _blob(W1, [0.0, 0.0], [2.0, 3.0], [0.5, -0.25], [1.0, 1.0], 0.0)
    s2 = op.scores(p2, [[1.0, 0, 0, 0]], (2,), layer_norm=True)
    r = 1.0 / math.sqrt(1.0 + 1e-5)
    assert abs(s2[0] - (max(-2 * r + 0.5, 0) + max(3 * r - 0.25, 0))) < 1e-15


def test_layer_norm_moments_and_shift_invariance():
    rng = np.random.default_rng(5)
    h1, h2, L = 16, 8, 50
    x = rng.normal(size=(L, 5))
    W1, b1 = rng.normal(size=(h1, 5)), rng.normal(size=h1)
    z = x @ W1.T + b1
    n = op.layer_norm_rows(z, np.ones(h1), np.zeros(h1))
    var = z.var(axis=1)
    assert np.allclose(n.mean(axis=1), 0, atol=1e-13)
    assert np.allclose(n.var(axis=1), var / (var + 1e-5), rtol=1e-12)
    W2, b2 = rng.normal(size=(h2, h1)), rng.normal(size=h2)
    g1, be1, g2, be2 = (rng.uniform(0.5, 2, h1), rng.normal(size=h1), rng.uniform(0.5, 2, h2),
                        rng.normal(size=h2))
    wo, bo = rng.normal(size=h2), 0.3

    def blob(b1_):
        return np.concatenate([W1.ravel(), b1_, g1, be1, W2.ravel(), b2, g2, be2, wo, [bo]])

    s = op.scores(blob(b1), x, (h1, h2), layer_norm=True)
    # adding one constant to every first-layer pre-activation changes nothing ...
    s_shift = op.scores(blob(b1 + 7.5), x, (h1, h2), layer_norm=True)
    assert np.allclose(s, s_shift, rtol=1e-11, atol=1e-11)
    # ... which is exactly what LayerNorm removes: without it the scores move
    plain = np.concatenate([W1.ravel(), b1, W2.ravel(), b2, wo, [bo]])
    plain_shift = np.concatenate([W1.ravel(), b1 + 7.5, W2.ravel(), b2, wo, [bo]])
    assert not np.allclose(op.scores(plain, x, (h1, h2)), op.scores(plain_shift, x, (h1, h2)))
