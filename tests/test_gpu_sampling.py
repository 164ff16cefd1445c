"""GPU parity of training-mode selection (Sec. 3.1.2 Gumbel-perturbed ranking;
App. C exact log-partition and subset log-probability): the HIP path through
the C ABI against the oracle.

Tolerances.  log Z and log pi: the device recursion adds positive terms in
float32 with one rounding per update and float32 weights, so the relative
error of Z is at most about (K + L) 2^-24 (K = min(B, L - B)); the tests allow
(K + L + 64) 2^-23 on log Z.  End to end, log pi also inherits the score
deviation: |d log pi| <= 2 B max|d s| / tau on top of that.  Sampled kept sets
are compared with the near-tie band widened by the float32 rounding of the
perturbed score (4 ulp of |s / tau| + |g| + |s~|)."""
import math

import numpy as np
import pytest
import torch

from oracle import sampling as osmp
from oracle import select as osel
from oracle import unit as ounit
from paper_2608_08878_amd import binding as B
from paper_2608_08878_amd.buffers import subset_log_prob
from synth import gpu as sg
from synth import philox as px
from synth import workloads as W

from . import harness as H
from .test_gpu_step import _buffers, _policy, _policy_from, _step_tensors, _tiny_state_after_one_step

pytestmark = pytest.mark.gpu

SCORE_STREAM = 41


def _scores(units, L, scale, step=0, shift=0.0):
    idx = np.arange(units * L, dtype=np.uint64)
    z = px.normal(W.WORKLOADS[1].seed, SCORE_STREAM, step, idx)
    return px.to_f32(z * scale + shift).reshape(units, L)


def _logz_tol(L, B):
    K = 0 if B >= L else min(B, L - B)
    return (K + L + 64) * 2.0 ** -23


def _dev(a, dtype=torch.float32):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dtype).cuda()


SMALL = [(b, tau) for tau in (1.0, 0.6)
         for b in (1, 2, 3, 5, 8, 9, 40, 64, 65, 100, 150, 151, 200, 236, 290, 292, 295, 298,
                   299, 300, 310)]


@pytest.mark.parametrize("B_,tau", SMALL)
def test_log_partition_small_rows(B_, tau):
    units, L = 3, 300
    s = _scores(units, L, 2.0, step=B_)
    nk = min(B_, L)
    rng = np.random.default_rng(B_)
    kept = np.stack([np.sort(rng.choice(L, nk, replace=False)) for _ in range(units)]).astype(np.int32)
    print(f"logz small B={B_} tau={tau}", flush=True)
    lz, lp = subset_log_prob(_dev(s), B_, tau, kept=_dev(kept, torch.int32))
    torch.cuda.synchronize()
    lz, lp = lz.cpu().numpy(), lp.cpu().numpy()
    for u in range(units):
        ref = osmp.log_partition(s[u], B_, tau)
        assert abs(lz[u] - ref) <= _logz_tol(L, B_), (u, lz[u], ref)
        refp = osmp.log_prob(s[u], kept[u], B_, tau)
        assert abs(lp[u] - refp) <= _logz_tol(L, B_), (u, lp[u], refp)
    if B_ >= L:
        assert np.all(lp == 0.0)


# (units, L, B, tau): one eviction per step, a 64-token block, compression steps
# of the decode workloads, two bands (K > 4096) and the largest single band.
LARGE = [(4, 2049, 2048, 1.0), (2, 3341, 3277, 1.0), (2, 4097, 1024, 1.0), (2, 8193, 2048, 1.0),
         (1, 9000, 4500, 0.8), (1, 16385, 4096, 1.0), (1, 12000, 11990, 1.3)]


@pytest.mark.parametrize("units,L,B_,tau", LARGE)
def test_log_partition_workload_sizes(units, L, B_, tau):
    s = _scores(units, L, 3.0, step=L)
    nk = min(B_, L)
    kept = np.stack([np.arange(u, u + nk) % L for u in range(units)]).astype(np.int32)
    print(f"logz L={L} B={B_} units={units}", flush=True)
    lz, lp = subset_log_prob(_dev(s), B_, tau, kept=_dev(kept, torch.int32))
    torch.cuda.synchronize()
    lz, lp = lz.cpu().numpy(), lp.cpu().numpy()
    for u in range(units):
        ref = osmp.log_partition(s[u], B_, tau)
        assert abs(lz[u] - ref) <= _logz_tol(L, B_), (u, lz[u] - ref)
        refp = float(s[u][kept[u]].astype(np.float64).sum() / tau) - ref
        assert abs(lp[u] - refp) <= _logz_tol(L, B_), (u, lp[u] - refp)


def test_log_partition_special_rows():
    L = 400
    rows = [np.full(L, 0.37, np.float32),                               # all equal
            np.concatenate([np.full(5, 50.0), np.full(L - 5, -3000.0)]).astype(np.float32),
            _scores(1, L, 40.0)[0]]                                      # wide spread
    s = np.stack(rows)
    for B_ in (1, 6, 100, 395, 399):
        lz, _ = subset_log_prob(_dev(s), B_, 0.5)
        torch.cuda.synchronize()
        lz = lz.cpu().numpy()
        r = float(np.float32(0.37)) / 0.5
        closed = math.lgamma(L + 1) - math.lgamma(B_ + 1) - math.lgamma(L - B_ + 1) + B_ * r
        assert abs(lz[0] - closed) <= _logz_tol(L, B_) + 1e-9 * abs(closed), (B_, lz[0], closed)
        for u in (1, 2):
            ref = osmp.log_partition(s[u], B_, 0.5)
            assert abs(lz[u] - ref) <= _logz_tol(L, B_) * max(1.0, 1e-4 * abs(ref)), (u, B_, lz[u], ref)


def test_log_partition_non_finite_and_bad_indices_give_nan():
    L = 200
    s = _scores(3, L, 1.0)
    s[1, 17] = np.nan
    s[2, 3] = np.inf
    kept = np.tile(np.arange(50, dtype=np.int32), (3, 1))
    kept[0, 10] = L                        # outside the row
    lz, lp = subset_log_prob(_dev(s), 50, 1.0, kept=_dev(kept, torch.int32))
    torch.cuda.synchronize()
    lz, lp = lz.cpu().numpy(), lp.cpu().numpy()
    assert np.isnan(lp[0]) and np.isnan(lz[0])
    assert np.isnan(lz[1]) and np.isnan(lp[1]) and np.isnan(lz[2]) and np.isnan(lp[2])


# ------------------------------------------------------------------ sampled selection

def _band(s_tau, g, st):
    return 1e-6 + 4 * 2.0 ** -24 * (np.abs(s_tau) + np.abs(g) + np.abs(st))


def _sampled_check(s_or, pos, kept_pos_gpu, budget, tau, seed, unit, draw):
    """Kept set of the device against the oracle's sampled top-B, with the
    widened near-tie band.  Returns (ok, oracle kept rows, n_ambiguous, n_flips)."""
    g = osmp.gumbel(seed, unit, draw, pos)
    st = osmp.perturbed_scores(s_or, tau, g)
    L = len(st)
    kept_o = osmp.sample_top_budget(s_or, pos, budget, tau, g)
    if budget >= L:
        return set(kept_pos_gpu) == set(pos.tolist()), kept_o, 0, 0
    order = osel.ranking(st, pos)
    thr = st[order[budget - 1]]
    band = _band(s_or / tau, g, st)
    amb = np.abs(st - thr) <= band + band[order[budget - 1]]
    ko = np.zeros(L, bool)
    ko[kept_o] = True
    kg = np.isin(pos, np.asarray(list(kept_pos_gpu)))
    mism = ko != kg
    return bool(not np.any(mism & ~amb)), kept_o, int(amb.sum()), int((mism & amb).sum())


def _check_layout(pre_u, kept_u, post_u, budget):
    L = len(pre_u["pos"])
    assert len(set(kept_u.tolist())) == min(budget, L)
    layout = H.slot_map_of(kept_u, L)
    assert np.array_equal(kept_u, layout)
    for name in ("k", "v", "pos", "alpha", "num", "den", "vnorm"):
        assert np.array_equal(post_u[name], pre_u[name][layout]), name


def test_gumbel_noise_alone_decides_with_constant_scores():
    """Zero weights: every score is b_out, so the kept set is the top-B of the
    Gumbel draws alone (pins the device generator's counter layout and
    transform), and log pi = -log C(L, B) exactly."""
    wl, buf = _tiny_state_after_one_step()
    U, L, budget, tau, seed, draw = wl.units, buf.kv.len, 100, 0.7, 0x0123_4567_89AB_CDEF, 5
    p, pol = _policy_from([0, 0, 0, 0, 0, 0, 0.25])
    pre = [H.download_unit(buf, u) for u in range(U)]
    scores = torch.empty((U, L), dtype=torch.float32, device="cuda")
    kept = torch.empty((U, budget), dtype=torch.int32, device="cuda")
    logp = torch.empty(U, dtype=torch.float64, device="cuda")
    buf.sample_evict(pol, budget, B.make_gumbel(tau, seed, draw), scores, kept, logp)
    torch.cuda.synchronize()
    sc, kp, lp = H.to_np(scores), H.to_np(kept), logp.cpu().numpy()
    for u in range(U):
        assert np.all(sc[u] == np.float32(0.25))
        post = H.download_unit(buf, u)
        ok, kept_o, amb, flips = _sampled_check(np.full(L, 0.25), pre[u]["pos"], post["pos"],
                                                budget, tau, seed, u, draw)
        assert ok and flips == 0, (u, amb, flips)
        _check_layout(pre[u], kp[u], post, budget)
        want = -(math.lgamma(L + 1) - math.lgamma(budget + 1) - math.lgamma(L - budget + 1))
        assert abs(lp[u] - want) <= _logz_tol(L, budget), (u, lp[u], want)


def _sampled_end_to_end(wl, n0, budget, tau, seed, draw, check_units=None):
    U = wl.units
    buf = _buffers(wl)
    buf.reserve_workspace(wl.capacity)
    sg.init_cache(wl, buf.k, buf.v, U, buf.cap)
    buf.feat_init(n0, 0)
    params, pol = _policy(wl)
    pnp = H.to_np(params)
    q, kn, vn = _step_tensors(wl)
    sg.queries(wl, 0, q)
    sg.new_rows(wl, 0, kn, vn, U)
    buf.decode_step(q, kn, vn)
    torch.cuda.synchronize()
    L = buf.kv.len
    units = range(U) if check_units is None else check_units
    pre = {u: H.download_unit(buf, u) for u in units}
    scores = torch.empty((U, L), dtype=torch.float32, device="cuda")
    kept = torch.empty((U, min(budget, L)), dtype=torch.int32, device="cuda")
    logp = torch.empty(U, dtype=torch.float64, device="cuda")
    buf.sample_evict(pol, budget, B.make_gumbel(tau, seed, draw), scores, kept, logp)
    torch.cuda.synchronize()
    sc, kp, lp = H.to_np(scores), H.to_np(kept), logp.cpu().numpy()
    total_flips = 0
    for u in units:
        st = H.oracle_student(wl, u, n0=n0)
        ounit.decode_step(st, *H.step_inputs_np(wl, 0, u))
        s_or = ounit.scores(st, pnp, wl.hidden)
        ok, worst = H.vec_ok(sc[u], s_or)
        assert ok, (u, "scores", worst)
        post = H.download_unit(buf, u)
        _check_layout(pre[u], kp[u], post, budget)
        ok, kept_o, amb, flips = _sampled_check(s_or, pre[u]["pos"], post["pos"], budget, tau, seed,
                                                u, draw)
        assert ok, (u, amb, flips)
        total_flips += flips
        if flips == 0:
            ref = osmp.log_prob(s_or, kept_o, budget, tau)
            ds = float(np.abs(sc[u].astype(np.float64) - s_or).max()) / tau
            tol = _logz_tol(L, budget) + 2 * min(budget, L) * ds + 1e-9 * abs(ref)
            assert abs(lp[u] - ref) <= tol, (u, lp[u], ref, tol)
    return total_flips


@pytest.mark.parametrize("cid,n0,budget,tau", [(2, 300, 100, 1.0), (2, 3000, 700, 0.5),
                                               (4, 3340, 3277, 1.0), (5, 2048, 2048, 1.0),
                                               (5, 2048, 512, 2.0)])
def test_sampled_selection_end_to_end(cid, n0, budget, tau):
    wl = W.WORKLOADS[cid].scaled(batch=1, n_layers=1, n_kv_heads=2, n_q_heads=8, n0=n0,
                                 budget=budget, steps=1)
    print(f"sampled end-to-end workload {cid} n0={n0} B={budget} tau={tau}", flush=True)
    flips = _sampled_end_to_end(wl, n0, budget, tau, seed=1000 + cid, draw=n0)
    assert flips <= 1


def test_sampled_selection_long_cache_workspace_path():
    """L > 8192 goes through the workspace-key path (row keys in memory)."""
    wl = W.WORKLOADS[5].scaled(batch=1, n_layers=1, n_kv_heads=2, n_q_heads=8, n0=8192,
                               budget=2048, steps=1)
    print("sampled long cache n0=8192 B=2048", flush=True)
    assert _sampled_end_to_end(wl, 8192, 2048, 1.0, seed=77, draw=3) <= 1


def test_sampling_is_deterministic_and_draws_differ():
    res = []
    for draw in (4, 4, 5):
        wl, buf = _tiny_state_after_one_step()
        U, L = wl.units, buf.kv.len
        _, pol = _policy(wl)
        kept = torch.empty((U, 100), dtype=torch.int32, device="cuda")
        scores = torch.empty((U, L), dtype=torch.float32, device="cuda")
        logp = torch.empty(U, dtype=torch.float64, device="cuda")
        buf.sample_evict(pol, 100, B.make_gumbel(1.0, 99, draw), scores, kept, logp)
        torch.cuda.synchronize()
        res.append((H.to_np(kept).copy(), logp.cpu().numpy().copy()))
    assert np.array_equal(res[0][0], res[1][0]) and np.array_equal(res[0][1], res[1][1])
    assert not np.array_equal(res[0][0], res[2][0])


def test_vanishing_temperature_reproduces_deterministic_selection():
    out = []
    for mode in ("det", "sample"):
        wl, buf = _tiny_state_after_one_step()
        U = wl.units
        _, pol = _policy(wl)
        kept = torch.empty((U, 100), dtype=torch.int32, device="cuda")
        if mode == "det":
            buf.score_evict(pol, 100, None, kept)
        else:
            # s / tau is so large that adding g cannot change its float32 value
            buf.sample_evict(pol, 100, B.make_gumbel(1e-20, 5, 1), None, kept, None)
        torch.cuda.synchronize()
        out.append(H.to_np(kept).copy())
    assert np.array_equal(out[0], out[1])


def _sampled_run(wl, n0, budget, tau, seed, draws, fused):
    U = wl.units
    buf = _buffers(wl)
    buf.reserve_workspace(wl.capacity)
    sg.init_cache(wl, buf.k, buf.v, U, buf.cap)
    buf.feat_init(n0, 0)
    _, pol = _policy(wl)
    q, kn, vn = _step_tensors(wl)
    snaps = []
    for t, draw in enumerate(draws):
        sg.queries(wl, t, q)
        sg.new_rows(wl, t, kn, vn, U)
        L = buf.kv.len + 1
        scores = torch.empty((U, L), dtype=torch.float32, device="cuda")
        kept = torch.empty((U, min(budget, L)), dtype=torch.int32, device="cuda")
        logp = torch.empty(U, dtype=torch.float64, device="cuda")
        g = B.make_gumbel(tau, seed, draw)
        if fused:
            out = buf.decode_sample_evict(pol, budget, g, q, kn, vn, None, scores, kept, logp)
        else:
            out = buf.decode_step(q, kn, vn)
            buf.sample_evict(pol, budget, g, scores, kept, logp)
        torch.cuda.synchronize()
        snaps.append({"out": H.to_np(out).copy(), "scores": H.to_np(scores).copy(),
                      "kept": H.to_np(kept).copy(), "logp": logp.cpu().numpy().copy(),
                      "state": [H.download_unit(buf, u) for u in range(U)]})
    return snaps


@pytest.mark.parametrize("cid,n0,budget", [(5, 2048, 2048), (5, 3000, 900), (4, 3340, 3277)])
def test_fused_sampled_step_equals_decode_then_sample(cid, n0, budget):
    """dc_decode_sample_evict (one launch where the cache fits) against
    dc_decode_step + dc_sample_evict: every output bit and the post-step state,
    over three steps with a new draw each; the fused kept set against the
    oracle's sampled selection at the first step."""
    wl = W.WORKLOADS[cid].scaled(batch=1, n_layers=1, n_kv_heads=2, n_q_heads=8, n0=n0,
                                 budget=budget, steps=3)
    print(f"fused sampled workload {cid} n0={n0} B={budget}", flush=True)
    a = _sampled_run(wl, n0, budget, 0.9, 4242, (7, 8, 9), True)
    b = _sampled_run(wl, n0, budget, 0.9, 4242, (7, 8, 9), False)
    for t, (x, y) in enumerate(zip(a, b)):
        for name in ("out", "scores", "kept", "logp"):
            assert np.array_equal(x[name], y[name]), (t, name)
        for u, (su, tu) in enumerate(zip(x["state"], y["state"])):
            for name in su:
                assert np.array_equal(su[name], tu[name]), (t, u, name)
    params, _ = _policy(wl)
    pnp = H.to_np(params)
    for u in range(wl.units):
        st = H.oracle_student(wl, u, n0=n0)
        ounit.decode_step(st, *H.step_inputs_np(wl, 0, u))
        s_or = ounit.scores(st, pnp, wl.hidden)
        ok, worst = H.vec_ok(a[0]["scores"][u], s_or)
        assert ok, (u, worst)
        ok, _, amb, flips = _sampled_check(s_or, st.pos, a[0]["state"][u]["pos"], budget, 0.9, 4242,
                                           u, 7)
        assert ok, (u, amb, flips)
