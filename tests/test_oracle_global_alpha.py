"""Pins of the paper's global alpha (Sec. 3.1.1: the attention mass a token
received in the most recent forward pass, averaged over all heads and layers)
and of the most-recent-step alpha it is built from."""
import numpy as np

from oracle import features
from oracle import unit as ounit



def test_hand_example_with_a_position_missing_from_one_unit():
    # unit A holds positions 0, 1, 2; unit B evicted position 1
    g = features.global_alpha([[0.5, 0.3, 0.2], [0.9, 0.1]], [[0, 1, 2], [0, 2]], 2)
    assert np.allclose(g[0], [0.7, 0.15, 0.15], rtol=0, atol=1e-15)
    assert np.allclose(g[1], [0.7, 0.15], rtol=0, atol=1e-15)


def test_single_unit_and_identical_units_are_unchanged():
    rng = np.random.default_rng(1)
    al = rng.random(7)
    ps = rng.permutation(20)[:7]
    assert np.array_equal(features.global_alpha([al], [ps], 1)[0], al)
    out = features.global_alpha([al, al, al], [ps, ps, ps], 3)
    for o in out:
        assert np.allclose(o, al, rtol=1e-15, atol=0)


def _sequence(n_units, G, d, rng, n0=12, evict=3):
    """One sequence's KV units (layers x KV heads) after different evictions:
    each unit keeps its own subset of the n0 prefix positions."""
    sts = []
    for u in range(n_units):
        keep = np.sort(rng.permutation(n0)[: n0 - evict])
        K = rng.standard_normal((n0, d))[keep]
        V = rng.standard_normal((n0, d))[keep]
        sts.append(ounit.new_student(K, V, keep, G=G, scale=d ** -0.5, window=4, next_pos=n0,
                                     alpha_recent=True))
    return sts


def test_recent_alpha_is_the_step_mass_and_the_global_mean_matches_all_heads():
    rng = np.random.default_rng(7)
    G, d, U = 4, 8, 6              # e.g. 3 layers x 2 KV heads
    sts = _sequence(U, G, d, rng)
    atts = None
    for t in range(3):
        atts = []
        for st in sts:
            q = rng.standard_normal((G, d))
            atts.append(ounit.decode_step(st, q, rng.standard_normal(d), rng.standard_normal(d)))
    for st, att in zip(sts, atts):
        # not accumulated: alpha is this step's head-mean mass, which sums to 1
        assert np.allclose(st.alpha, att.a.mean(axis=0), rtol=1e-14, atol=0)
        assert abs(st.alpha.sum() - 1.0) <= 1e-12
    g = features.global_alpha([st.alpha for st in sts], [st.pos for st in sts], U)
    # the definition from the raw weights: mean over every query head of every
    # unit, a head whose unit lacks the position contributing 0
    allpos = sorted(set(int(p) for st in sts for p in st.pos))
    direct = {}
    for p in allpos:
        acc = 0.0
        for st, att in zip(sts, atts):
            hit = np.nonzero(st.pos == p)[0]
            for j in range(G):
                acc += att.a[j, hit[0]] if hit.size else 0.0
        direct[p] = acc / (U * G)
    for st, gu in zip(sts, g):
        assert np.allclose(gu, [direct[int(p)] for p in st.pos], rtol=1e-13, atol=0)
    # conservation over the union of positions held by the sequence's units
    assert abs(sum(direct.values()) - 1.0) <= 1e-12


def test_cumulative_alpha_is_unchanged_by_the_mode_flag_default():
    rng = np.random.default_rng(3)
    G, d = 2, 4
    K, V = rng.standard_normal((5, d)), rng.standard_normal((5, d))
    st = ounit.new_student(K, V, np.arange(5), G=G, scale=0.5, window=4)
    masses = []
    for t in range(3):
        att = ounit.decode_step(st, rng.standard_normal((G, d)), rng.standard_normal(d), rng.standard_normal(d))
        masses.append(np.concatenate([att.a.mean(axis=0)]))
    # cumulative: the rows present at every step hold the sum of their masses
    expect = masses[0][:5] + masses[1][:5] + masses[2][:5]
    assert np.allclose(st.alpha[:5], expect, rtol=1e-14, atol=0)
