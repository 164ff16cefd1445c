"""Pins for the CPU oracle: facts fixed by the paper and by mathematics that do
not come from the oracle itself (closed forms, invariants, brute force, library
routines).  Each test names the slip it is there to catch."""
import itertools
import json
import math
import os

import numpy as np
import pytest
import scipy.stats

from oracle import attention, features, kl, policy, select, unit

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
RNG = np.random.default_rng(20260802)


def _ev(x):
    if isinstance(x, list):
        return np.array([_ev(v) for v in x], dtype=np.float64)
    return float(eval(str(x), {"__builtins__": {}}, {"math": math}))


# ------------------------------------------------------------------ attention

def test_attention_weights_sum_to_one():
    for L in (1, 7, 300):
        q, K, V = RNG.normal(size=(4, 16)), RNG.normal(size=(L, 16)) * 3, RNG.normal(size=(L, 16))
        att = attention.attend(q, K, V, 0.25)
        assert np.all(np.abs(att.a.sum(axis=1) - 1.0) <= 1e-12)
        assert np.all(att.a >= 0)


def test_attention_single_row_is_that_value_with_zero_entropy():
    q, K, V = RNG.normal(size=(3, 8)), RNG.normal(size=(1, 8)), RNG.normal(size=(1, 8))
    att = attention.attend(q, K, V, 0.5)
    assert np.array_equal(att.o, np.repeat(V, 3, axis=0))
    assert np.all(att.H == 0.0)


def test_attention_equal_keys_give_uniform_weights_mean_value_and_log_L():
    L = 37
    K = np.tile(RNG.normal(size=(1, 8)), (L, 1))
    V = RNG.normal(size=(L, 8))
    att = attention.attend(RNG.normal(size=(2, 8)), K, V, 1.0)
    assert np.allclose(att.a, 1.0 / L, rtol=0, atol=1e-15)
    assert np.allclose(att.o, V.mean(axis=0)[None, :], rtol=0, atol=1e-13)
    assert np.allclose(att.H, math.log(L), rtol=1e-14)


def test_attention_two_key_closed_form_catches_sign_and_scale_slips():
    # logits (0, x): a1 = e^x / (1 + e^x); H = ln(1 + e^x) - x a1
    for x in (-3.0, -0.2, 0.7, 5.0):
        scale = 0.5
        q = np.array([[2.0 * x]])              # scale * q.k = x for k = (1)
        K = np.array([[0.0], [1.0]])
        V = np.array([[10.0], [-4.0]])
        att = attention.attend(q, K, V, scale)
        a1 = math.exp(x) / (1.0 + math.exp(x))
        assert math.isclose(att.a[0, 1], a1, rel_tol=1e-14)
        assert math.isclose(att.H[0], math.log1p(math.exp(x)) - x * a1, rel_tol=1e-13)
        assert math.isclose(att.o[0, 0], 10.0 * (1 - a1) - 4.0 * a1, rel_tol=1e-13)


def test_attention_is_permutation_invariant():
    q, K, V = RNG.normal(size=(4, 16)), RNG.normal(size=(50, 16)), RNG.normal(size=(50, 16))
    perm = RNG.permutation(50)
    a1 = attention.attend(q, K, V, 0.3)
    a2 = attention.attend(q, K[perm], V[perm], 0.3)
    assert np.allclose(a1.o, a2.o, rtol=0, atol=1e-13)
    assert np.allclose(a1.H, a2.H, rtol=1e-13)
    assert np.allclose(a1.a[:, perm], a2.a, rtol=0, atol=1e-15)


def test_entropy_bounds_and_one_dominant_logit():
    for L in (2, 10, 4097):
        q, K = RNG.normal(size=(4, 32)), RNG.normal(size=(L, 32)) * RNG.uniform(0.1, 8)
        att = attention.attend(q, K, np.zeros((L, 32)), 1 / math.sqrt(32))
        assert np.all(att.H >= 0) and np.all(att.H <= math.log(L) + 1e-12)
    K = np.zeros((20, 4))
    K[7] = 1.0
    att = attention.attend(np.array([[400.0, 0, 0, 0]]), K, np.zeros((20, 4)), 1.0)
    assert att.H[0] < 1e-100


def test_eviction_error_bound_of_the_reward_motivation():
    """Sec. 3.1.4: renormalising attention over the kept set moves the output by
    at most 2 * max||v|| * (evicted attention mass)."""
    for trial in range(50):
        L, d = int(RNG.integers(2, 60)), 8
        q, K, V = RNG.normal(size=(1, d)), RNG.normal(size=(L, d)) * 2, RNG.normal(size=(L, d))
        keep = np.sort(RNG.choice(L, size=int(RNG.integers(1, L + 1)), replace=False))
        full = attention.attend(q, K, V, 0.5)
        part = attention.attend(q, K[keep], V[keep], 0.5)
        eps = 1.0 - full.a[0, keep].sum()
        C = np.sqrt((V ** 2).sum(axis=1)).max()
        assert np.linalg.norm(full.o[0] - part.o[0]) <= 2 * C * eps + 1e-12


# ------------------------------------------------------------------ features

def _student(L=40, d=16, G=4, window=64, seed=1):
    r = np.random.default_rng(seed)
    K, V = r.normal(size=(L, d)), r.normal(size=(L, d))
    return unit.new_student(K, V, np.arange(L), G=G, scale=1 / math.sqrt(d), window=window), r


def test_feature_step_sums():
    st, r = _student()
    G, d = 4, 16
    for t in range(5):
        a0, (z0, n0) = st.alpha.copy(), st.hist.sums()
        att = unit.decode_step(st, r.normal(size=(G, d)), r.normal(size=d), r.normal(size=d))
        z1, n1 = st.hist.sums()
        z0 = np.append(z0, 0.0); n0 = np.append(n0, 0.0); a0 = np.append(a0, 0.0)
        assert math.isclose((st.alpha - a0).sum(), 1.0, rel_tol=1e-12)
        assert math.isclose((z1 - z0).sum(), G, rel_tol=1e-12)
        assert math.isclose((n1 - n0).sum(), att.H.sum(), rel_tol=1e-12)


def test_window_entropy_is_a_weighted_mean_of_window_entropies():
    st, r = _student(window=8)
    Hs = []
    for t in range(20):
        att = unit.decode_step(st, r.normal(size=(4, 16)) * r.uniform(0.2, 3), r.normal(size=16), r.normal(size=16))
        Hs.append(att.H)
        Z, N = st.hist.sums()
        Hi = features.entropy_feature(Z, N)
        win = np.concatenate(Hs[-8:])
        assert np.all(Hi >= win.min() - 1e-12) and np.all(Hi <= win.max() + 1e-12)


def test_window_64_equals_unbounded_before_step_64_and_differs_after():
    s1, r1 = _student(window=64, seed=5)
    s2, r2 = _student(window=0, seed=5)
    for t in range(70):
        q, k, v = r1.normal(size=(4, 16)), r1.normal(size=16), r1.normal(size=16)
        r2.normal(size=(4, 16)); r2.normal(size=16); r2.normal(size=16)
        unit.decode_step(s1, q, k, v)
        unit.decode_step(s2, q, k, v)
        z1, n1 = s1.hist.sums()
        z2, n2 = s2.hist.sums()
        if t < 64:
            assert np.allclose(z1, z2, rtol=1e-12) and np.allclose(n1, n2, rtol=1e-12)
    assert not np.allclose(z1, z2, rtol=1e-6)


def test_add_retire_bookkeeping_equals_window_definition():
    st, r = _student(L=60, window=16, seed=9)
    for t in range(80):
        unit.decode_step(st, r.normal(size=(4, 16)), r.normal(size=16) * 2, r.normal(size=16))
        if t % 7 == 3:       # evict a few rows now and then
            s = r.normal(size=st.L)
            unit.evict(st, s, st.L - 3)
        Z, N = st.hist.sums()
        assert np.allclose(st.Z, Z, rtol=1e-9, atol=1e-15)
        assert np.allclose(st.N, N, rtol=1e-9, atol=1e-15)


def test_position_feature_in_unit_interval():
    st, r = _student()
    unit.decode_step(st, r.normal(size=(4, 16)), r.normal(size=16), r.normal(size=16))
    x = unit.feature_matrix(st)
    assert np.all(x[:, 3] >= 0) and np.all(x[:, 3] < 1)
    assert x[-1, 3] == (st.next_pos - 1) / st.next_pos


# ------------------------------------------------------------------ golden

def test_two_token_golden_example():
    g = json.load(open(os.path.join(GOLDEN, "two_token_example.json")))
    inp, exp = g["inputs"], g["expected"]
    K, V = np.array(inp["K"]), np.array(inp["V"])
    qs = [np.array([[_ev(x) for x in q]]) for q in inp["q_steps"]]
    for window, tag in ((2, "w2"), (1, "w1")):
        st = unit.new_student(K, V, inp["positions"], G=1, scale=inp["scale"], window=window)
        a0 = unit.decode_step(st, qs[0])
        assert np.allclose(a0.a[0], _ev(exp["step0_weights"]), rtol=1e-14)
        assert math.isclose(a0.H[0], _ev(exp["step0_entropy"]), rel_tol=1e-14)
        assert math.isclose(a0.o[0, 0], _ev(exp["step0_out"]), rel_tol=1e-14)
        a1 = unit.decode_step(st, qs[1])
        assert math.isclose(a1.H[0], _ev(exp["step1_entropy"]), rel_tol=1e-14)
        assert math.isclose(a1.o[0, 0], _ev(exp["step1_out"]), rel_tol=1e-14)
        assert np.allclose(st.alpha, _ev(exp["alpha"]), rtol=1e-14)
        Z, N = st.hist.sums()
        x = unit.feature_matrix(st)
        if tag == "w2":
            assert np.allclose(Z, _ev(exp["window2_Z"]), rtol=1e-14)
            assert np.allclose(N, _ev(exp["window2_N"]), rtol=1e-14)
            assert np.allclose(x, _ev(exp["features_w2"]), rtol=1e-14, atol=0)
            s = unit.scores(st, np.array(inp["policy_params"], float), tuple(inp["policy_hidden"]))
            assert np.allclose(s, _ev(exp["scores_w2"]), rtol=1e-14)
            assert list(select.top_budget(s, st.pos, inp["budget"])) == exp["kept"]
            zero = np.zeros(13); zero[-1] = 0.5
            s0 = unit.scores(st, zero, (2,))
            assert list(select.top_budget(s0, st.pos, inp["budget"])) == exp["kept_all_zero_policy"]
        else:
            assert np.allclose(features.entropy_feature(Z, N), _ev(exp["window1_H"]), rtol=1e-14)


# ------------------------------------------------------------------ policy

def test_policy_zero_weights_give_output_bias():
    n = 4 * 32 + 32 + 32 + 1
    p = np.zeros(n); p[-1] = -0.75
    assert np.all(policy.scores(p, RNG.normal(size=(9, 4)), (32,)) == -0.75)


def test_policy_one_hot_probes_fix_layout_and_feature_order():
    hidden = (3,)
    x = RNG.normal(size=(11, 4)) + 2.0
    for f in range(4):
        for k in range(3):
            p = np.zeros(4 * 3 + 3 + 3 + 1)
            p[k * 4 + f] = 1.0           # W1[k][f]
            p[12 + 3 + k] = 1.0          # w_out[k]
            assert np.array_equal(policy.scores(p, x, hidden), np.maximum(x[:, f], 0))


def test_policy_two_hidden_layers_probe():
    hidden = (2, 3)
    n = 2 * 4 + 2 + 3 * 2 + 3 + 3 + 1
    p = np.zeros(n)
    p[1] = 1.0                  # W1[0][1] picks feature 1 into hidden unit 0
    p[8 + 1] = -1.0             # b1[1] = -1 -> hidden unit 1 = relu(-1) = 0
    p[10 + 2 * 2 + 0] = 3.0     # W2[2][0] = 3
    p[10 + 6 + 2] = 0.5         # b2[2] = 0.5
    p[10 + 6 + 3 + 2] = 2.0     # w_out[2] = 2
    p[-1] = 1.0
    x = RNG.normal(size=(5, 4))
    assert np.allclose(policy.scores(p, x, hidden), 2.0 * np.maximum(3.0 * np.maximum(x[:, 1], 0) + 0.5, 0) + 1.0)


# ------------------------------------------------------------------ select

def test_select_brute_force_max_sum_subset_with_earliest_tiebreak():
    for trial in range(300):
        L = int(RNG.integers(1, 11))
        B = int(RNG.integers(1, L + 1))
        s = RNG.integers(-3, 4, size=L).astype(float)   # many ties on purpose
        pos = np.sort(RNG.choice(1000, size=L, replace=False))
        best = None
        for sub in itertools.combinations(range(L), B):
            # maximise the sum; among equal sums prefer the lexicographically earliest positions
            cand = (s[list(sub)].sum(), tuple(sorted((-pos[i] for i in sub), reverse=True)))
            if best is None or cand > best[0]:
                best = (cand, sub)
        assert tuple(select.top_budget(s, pos, B)) == tuple(sorted(best[1]))


def test_select_size_and_separation():
    for trial in range(100):
        L = int(RNG.integers(1, 500)); B = int(RNG.integers(1, 600))
        s = RNG.normal(size=L)
        kept = select.top_budget(s, np.arange(L), B)
        assert len(kept) == min(B, L)
        ev = np.setdiff1d(np.arange(L), kept)
        if len(ev):
            assert s[kept].min() >= s[ev].max()


def test_select_all_equal_keeps_earliest_and_nan_ranks_last():
    s = np.zeros(10)
    pos = np.array([5, 3, 9, 0, 1, 2, 8, 7, 6, 4])
    assert sorted(pos[select.top_budget(s, pos, 4)]) == [0, 1, 2, 3]
    s = np.array([np.nan, -np.inf, -0.0, 0.0, np.nan])
    kept = select.top_budget(s, np.arange(5), 3)
    assert list(kept) == [1, 2, 3]
    kept = select.top_budget(s, np.arange(5), 2)      # -0.0 == +0.0: earlier wins
    assert list(kept) == [2, 3]
    assert list(select.top_budget(np.array([np.nan, np.nan, 1.0]), np.array([7, 2, 9]), 2)) == [1, 2]


# ------------------------------------------------------------------ KL

def test_kl_zero_for_identical_and_nonnegative():
    h = RNG.normal(size=(5, 64)); W = RNG.normal(size=(300, 64)) * 0.1
    assert np.all(kl.kl_reward(h, h, W) == 0.0)
    h2 = h + RNG.normal(size=h.shape)
    assert np.all(kl.kl_reward(h, h2, W) > 0)


def test_kl_shift_invariance_and_two_symbol_closed_form():
    z = RNG.normal(size=(3, 50))
    assert np.allclose(kl.kl_from_logits(z, z + 7.25), 0.0, atol=1e-14)
    for p, q in ((0.3, 0.6), (0.99, 0.01), (0.5, 0.5001)):
        lz = np.log([[p, 1 - p]]); lq = np.log([[q, 1 - q]])
        want = p * math.log(p / q) + (1 - p) * math.log((1 - p) / (1 - q))
        # binary64 log-softmax differences carry ~1e-16 absolute error per term
        assert math.isclose(kl.kl_from_logits(lz, lq)[0], want, rel_tol=1e-10, abs_tol=1e-14)


def test_kl_matches_scipy_entropy_and_pinsker():
    for _ in range(10):
        a, b = RNG.normal(size=(1, 1000)) * 2, RNG.normal(size=(1, 1000)) * 2
        P = np.exp(a - a.max()); P /= P.sum()
        Q = np.exp(b - b.max()); Q /= Q.sum()
        got = kl.kl_from_logits(a, b)[0]
        assert math.isclose(got, scipy.stats.entropy(P[0], Q[0]), rel_tol=1e-10)
        assert got >= 0.5 * np.abs(P - Q).sum() ** 2


# ------------------------------------------------------------------ unit

def test_budget_at_least_len_reproduces_the_teacher_exactly():
    r = np.random.default_rng(3)
    L, d, G = 30, 8, 2
    K, V = r.normal(size=(L, d)), r.normal(size=(L, d))
    st = unit.new_student(K, V, np.arange(L), G=G, scale=0.3)
    te = unit.new_teacher(K, V, np.arange(L), scale=0.3)
    params = r.normal(size=4 * 32 + 32 + 32 + 1) * 0.1
    for t in range(10):
        q, k, v = r.normal(size=(G, d)), r.normal(size=d), r.normal(size=d)
        a_s = unit.decode_step(st, q, k, v)
        a_t = unit.teacher_step(te, q, k, v)
        assert np.array_equal(a_s.o, a_t.o)
        _, kept = unit.score_evict(st, params, (32,), budget=st.L + int(r.integers(0, 3)))
        assert np.array_equal(kept, np.arange(st.L))
    assert np.array_equal(st.K, te.K) and np.array_equal(st.pos, te.pos)


def test_eviction_carries_rows_and_state():
    r = np.random.default_rng(4)
    L, d, G = 50, 8, 2
    st = unit.new_student(r.normal(size=(L, d)), r.normal(size=(L, d)), np.arange(L), G=G, scale=0.3)
    unit.decode_step(st, r.normal(size=(G, d)), r.normal(size=d), r.normal(size=d))
    before = (st.K.copy(), st.V.copy(), st.pos.copy(), st.alpha.copy(), st.hist.z.copy())
    s = r.normal(size=st.L)
    kept = unit.evict(st, s, 20)
    assert st.L == 20 and len(set(st.pos.tolist())) == 20
    for arr, old in zip((st.K, st.V, st.pos, st.alpha, st.hist.z), before):
        assert np.array_equal(arr, old[kept])


def test_dynamic_budget_schedule():
    from oracle import select as osel
    # the paper's protocol: ratio 0.25, minimum 32
    assert osel.dynamic_budget(0.25, 8193) == 2048
    assert osel.dynamic_budget(0.25, 100) == 32 and osel.dynamic_budget(0.25, 128) == 32
    assert osel.dynamic_budget(0.25, 132) == 33
    assert osel.dynamic_budget(0.125, 16384, 32) == 2048
    # non-decreasing in the sequence length, and a cache that follows it loses at
    # most one row per step once it is at the budget
    L, prev = 300, 0
    for T in range(301, 2000):
        B = osel.dynamic_budget(0.25, T)
        assert B >= prev
        prev = B
        newL = min(B, L + 1)
        if T > 301:
            assert L + 1 - newL <= 1
        L = newL
    with pytest.raises(ValueError):
        osel.dynamic_budget(0.0, 10)
