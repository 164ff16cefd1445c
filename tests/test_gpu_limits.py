"""GPU parity at the documented maximum sizes: a 40960-row cache (the largest
the selection takes) through decode and a compression step, and the exact
log-partition at 40960 rows with K = 20480 (five bands of the recursion)."""
import numpy as np
import pytest
import torch

from oracle import sampling as osmp
from oracle import unit as ounit
from paper_2608_08878_amd.buffers import subset_log_prob
from synth import gpu as sg
from synth import workloads as W

from . import harness as H
from .test_gpu_sampling import _dev, _logz_tol, _scores
from .test_gpu_step import _buffers, _check_decode, _check_evict, _policy, _step_tensors

pytestmark = pytest.mark.gpu


def test_maximum_cache_length_decode_and_compression():
    # 40959 rows + the appended one = 40960; keep 10000 (10000 moves, within the 16384 cap)
    wl = W.WORKLOADS[2].scaled(batch=1, n_layers=1, n_kv_heads=1, n_q_heads=4, n0=40959,
                               budget=10000, steps=1)
    U = wl.units
    buf = _buffers(wl)
    buf.reserve_workspace(wl.capacity)
    sg.init_cache(wl, buf.k, buf.v, U, buf.cap)
    buf.feat_init(wl.n0, 0)
    params, pol = _policy(wl)
    pnp = H.to_np(params)
    q, kn, vn = _step_tensors(wl)
    sg.queries(wl, 0, q)
    sg.new_rows(wl, 0, kn, vn, U)
    print("maximum length: decode 40960 rows", flush=True)
    out = buf.decode_step(q, kn, vn)
    torch.cuda.synchronize()
    assert buf.kv.len == 40960
    pre = [H.download_unit(buf, u) for u in range(U)]
    scores = torch.empty((U, 40960), dtype=torch.float32, device="cuda")
    kept = torch.empty((U, wl.budget), dtype=torch.int32, device="cuda")
    print("maximum length: select 10000 of 40960", flush=True)
    buf.score_evict(pol, wl.budget, scores, kept)
    torch.cuda.synchronize()
    outn, sc, kp = H.to_np(out), H.to_np(scores), H.to_np(kept)
    for u in range(U):
        st = H.oracle_student(wl, u)
        att = ounit.decode_step(st, *H.step_inputs_np(wl, 0, u))
        _check_decode(wl, outn[u], pre[u], st, att, u)
        s_or = ounit.scores(st, pnp, wl.hidden)
        _check_evict(wl, wl.budget, pre[u], sc[u], kp[u], H.download_unit(buf, u), s_or, u)


@pytest.mark.parametrize("B_", [20480, 35000, 1])
def test_log_partition_at_maximum_length(B_):
    L = 40960
    s = _scores(1, L, 2.0, step=B_ + 7)
    kept = np.arange(min(B_, L), dtype=np.int32)[None, :]
    print(f"log-partition L={L} B={B_}", flush=True)
    lz, lp = subset_log_prob(_dev(s), B_, 1.0, kept=_dev(kept, torch.int32))
    torch.cuda.synchronize()
    ref = osmp.log_partition(s[0], B_, 1.0)
    assert abs(lz.item() - ref) <= _logz_tol(L, B_), (lz.item(), ref)
    refp = float(s[0][kept[0]].astype(np.float64).sum()) - ref
    assert abs(lp.item() - refp) <= _logz_tol(L, B_)


def _sequence_rows(buf, u, L):
    return {"pos": H.to_np(buf.pos[u, :L]).astype(np.int64), "alpha": H.to_np(buf.alpha[u, :L])}


@pytest.mark.parametrize("hidden", [(32,), (64, 64)])
def test_more_units_than_one_grid_dimension_holds(hidden):
    """65544 units (8193 sequences x 8 KV heads): the grids whose rows are units
    run in slices of 65535 rows.  A ragged cache (chunked decode, row-key
    selection with per-unit budgets) with the paper's alpha (recent mass, then
    the cross-unit mean); the sequences on both sides of the slice boundary
    and the first one are checked against the oracle."""
    from oracle import features as ofeat
    from paper_2608_08878_amd.buffers import DecodeBuffers, make_policy
    wl = W.WORKLOADS[2].scaled(batch=8193, n_layers=1, n_kv_heads=8, n_q_heads=32, n0=30,
                               budget=20, steps=1, hidden=hidden)
    U, per_seq = wl.units, 8
    assert U == 65544
    buf = DecodeBuffers(wl.batch, wl.n_layers, wl.n_q_heads, wl.n_kv_heads, wl.head_dim, 40,
                        wl.dtype, wl.ent_window, 0.0, True, ragged=True, alpha_recent=True)
    buf.reserve_workspace(40)
    sg.init_cache(wl, buf.k, buf.v, U, buf.cap)
    buf.feat_init(wl.n0, 0)
    params = torch.empty(wl.n_params, dtype=torch.float32, device="cuda")
    sg.fill_normal(params, wl, W.S_POLICY, 0, 0.1)
    pol = make_policy(params, hidden)
    pnp = H.to_np(params)
    budgets = torch.tensor([12 + (u % 9) for u in range(U)], dtype=torch.int32, device="cuda")
    q, kn, vn = _step_tensors(wl)
    sg.queries(wl, 0, q)
    sg.new_rows(wl, 0, kn, vn, U)
    print(f"{U} units: decode", flush=True)
    out = buf.decode_step(q, kn, vn)
    torch.cuda.synchronize()
    L = 31
    recent = {u: _sequence_rows(buf, u, L) for b in (0, 8191, 8192) for u in range(8 * b, 8 * b + 8)}
    print(f"{U} units: global alpha, selection", flush=True)
    buf.global_alpha()
    torch.cuda.synchronize()
    glob = {u: H.to_np(buf.alpha[u, :L]) for u in recent}
    scores = torch.empty((U, L), dtype=torch.float32, device="cuda")
    kept = torch.empty((U, 20), dtype=torch.int32, device="cuda")
    buf.score_evict_units(pol, budgets, 20, None, scores, kept, None)
    torch.cuda.synchronize()
    outn, sc = H.to_np(out), H.to_np(scores)
    bud = H.to_np(budgets)
    for b in (0, 8191, 8192):
        us = list(range(8 * b, 8 * b + 8))
        sts = []
        for u in us:
            st = H.oracle_student(wl, u)
            st.alpha_recent = True
            att = ounit.decode_step(st, *H.step_inputs_np(wl, 0, u))
            assert H.rel_err_rows(outn[u], att.o) <= H.OUT_TOL, u
            order = np.argsort(recent[u]["pos"])
            ok, worst = H.vec_ok(recent[u]["alpha"][order], st.alpha)
            assert ok, (u, "recent alpha", worst)
            sts.append(st)
        g = ofeat.global_alpha([st.alpha for st in sts], [st.pos for st in sts], per_seq)
        for u, st, gu in zip(us, sts, g):
            order = np.argsort(recent[u]["pos"])
            ok, worst = H.vec_ok(glob[u][order], gu)
            assert ok, (u, "global alpha", worst)
            st.alpha = gu
            s_or = ounit.scores(st, pnp, hidden)
            ok, worst = H.vec_ok(sc[u][order], s_or)
            assert ok, (u, "scores", worst)
            nk = int(bud[u])
            post_pos = H.to_np(buf.pos[u, :nk]).astype(np.int64)
            ok, amb, flips = H.selection_check(s_or, st.pos, post_pos, nk)
            assert ok, (u, amb, flips)
    lens = H.to_np(buf.unit_len)
    assert np.array_equal(lens, np.minimum(31, H.to_np(budgets)))
