"""GPU parity of the paper's alpha (Sec. 3.1.1): decode steps that leave each
row's most recent mass (alpha_recent), the cross-unit average over all heads
and layers of a sequence (dc_global_alpha), and the scoring and eviction that
then use it, against the oracle, step by step.  Units of a sequence evict
different rows, so positions go missing from some of them."""
import numpy as np
import pytest
import torch

from oracle import features as ofeat
from oracle import unit as ounit
from paper_2608_08878_amd.buffers import DecodeBuffers
from synth import gpu as sg
from synth import workloads as W

from . import harness as H
from .test_gpu_step import _check_decode, _policy, _step_tensors

pytestmark = pytest.mark.gpu


def _download(buf, u, L):
    return {"k": H.to_np(buf.k[u, :L]).astype(np.float64), "v": H.to_np(buf.v[u, :L]).astype(np.float64),
            "pos": H.to_np(buf.pos[u, :L]).astype(np.int64), "alpha": H.to_np(buf.alpha[u, :L]),
            "num": H.to_np(buf.num[u, :L]), "den": H.to_np(buf.den[u, :L]),
            "vnorm": H.to_np(buf.vnorm[u, :L])}


def _global_run(steps, budgets=None, budget=200, n0=300, batch=2, n_layers=2, n_kv=2):
    ragged = budgets is not None
    wl = W.WORKLOADS[2].scaled(batch=batch, n_layers=n_layers, n_kv_heads=n_kv,
                               n_q_heads=4 * n_kv, n0=n0,
                               budget=max(budgets) if ragged else budget, steps=steps)
    U, per_seq = wl.units, n_layers * n_kv
    buf = DecodeBuffers(wl.batch, wl.n_layers, wl.n_q_heads, wl.n_kv_heads, wl.head_dim,
                        wl.capacity, wl.dtype, wl.ent_window, 0.0, True, ragged=ragged,
                        alpha_recent=True)
    buf.reserve_workspace(wl.capacity)
    sg.init_cache(wl, buf.k, buf.v, U, buf.cap)
    buf.feat_init(n0, 0)
    params, pol = _policy(wl)
    pnp = H.to_np(params)
    sts = []
    for u in range(U):
        st = H.oracle_student(wl, u)
        st.alpha_recent = True
        sts.append(st)
    q, kn, vn = _step_tensors(wl)
    bud = torch.tensor(budgets, dtype=torch.int32, device="cuda") if ragged else None
    for t in range(steps):
        sg.queries(wl, t, q)
        sg.new_rows(wl, t, kn, vn, U)
        out = buf.decode_step(q, kn, vn)
        torch.cuda.synchronize()
        lens = H.to_np(buf.unit_len).astype(int) if ragged else [buf.kv.len] * U
        outn = H.to_np(out)
        pre = [_download(buf, u, lens[u]) for u in range(U)]
        for u in range(U):
            att = ounit.decode_step(sts[u], *H.step_inputs_np(wl, t, u))
            # the step's own mass (not accumulated), with the other state; until a
            # near-tie parts them, device and oracle store the rows in the same slots
            _check_decode(wl, outn[u], pre[u], sts[u], att, (t, u))
            assert abs(sts[u].alpha.sum() - 1.0) <= 1e-12
        buf.global_alpha()
        torch.cuda.synchronize()
        for b in range(wl.batch):
            us = range(b * per_seq, (b + 1) * per_seq)
            g = ofeat.global_alpha([sts[u].alpha for u in us], [sts[u].pos for u in us], per_seq)
            for u, gu in zip(us, g):
                sts[u].alpha = gu
        for u in range(U):
            ga = H.to_np(buf.alpha[u, :lens[u]])
            ok, worst = H.vec_ok(ga, sts[u].alpha)
            assert ok, (t, u, "global alpha", worst)
            pre[u]["alpha"] = H.to_np(buf.alpha[u, :lens[u]])
        Lb = buf.kv.len
        maxb = max(budgets) if ragged else budget
        scores = torch.empty((U, Lb), dtype=torch.float32, device="cuda")
        kept = torch.empty((U, min(maxb, Lb)), dtype=torch.int32, device="cuda")
        if ragged:
            buf.score_evict_units(pol, bud, maxb, None, scores, kept, None)
        else:
            buf.score_evict(pol, budget, scores, kept)
        torch.cuda.synchronize()
        sc, kp = H.to_np(scores), H.to_np(kept)
        diverged = False
        for u in range(U):
            s_or = ounit.scores(sts[u], pnp, wl.hidden)
            ok, worst = H.vec_ok(sc[u, :lens[u]], s_or)
            assert ok, (t, u, "scores", worst)
            Bu = budgets[u] if ragged else budget
            nk = min(Bu, lens[u])
            post = _download(buf, u, nk)
            ok, amb, flips = H.selection_check(s_or, sts[u].pos, post["pos"], nk)
            assert ok, (t, u, amb, flips)
            layout = H.oracle_slot_map(sc[u, :lens[u]], pre[u]["pos"], nk)
            assert np.array_equal(kp[u, :nk], layout), (t, u)
            for name in ("k", "v", "pos", "alpha", "num", "den", "vnorm"):
                assert np.array_equal(post[name], pre[u][name][layout]), (t, u, name)
            ounit.evict(sts[u], s_or, Bu)
            diverged |= flips > 0
        if diverged:
            print("trajectories parted at a near-tie at step", t)
            return t
    if per_seq > 1:     # positions differ across the units of a sequence by now
        assert any(not np.array_equal(np.sort(sts[0].pos), np.sort(sts[u].pos))
                   for u in range(1, per_seq))
    return steps


def test_global_alpha_trajectory():
    assert _global_run(steps=5) >= 2


def test_global_alpha_on_ragged_caches_with_per_unit_budgets():
    # sequence 0: one unit keeps its whole cache (the hybrid's full head)
    assert _global_run(steps=4, budgets=[150, 10 ** 6, 220, 180, 200, 120, 260, 90]) >= 2


def test_global_alpha_of_a_single_unit_sequence_is_its_own_mass():
    assert _global_run(steps=3, batch=3, n_layers=1, n_kv=1) >= 1


def test_recent_and_global_alpha_on_the_float32_path():
    """The float32 / d = 64 kernels (workload 1's shape, no append): three steps
    with alpha_recent, each followed by the cross-unit mean."""
    wl = W.WORKLOADS[1].scaled(batch=2, n_layers=2, n_kv_heads=2, n_q_heads=4, steps=3)
    U, per_seq = wl.units, wl.n_layers * wl.n_kv_heads
    buf = DecodeBuffers(wl.batch, wl.n_layers, wl.n_q_heads, wl.n_kv_heads, wl.head_dim,
                        wl.capacity, wl.dtype, wl.ent_window, 0.0, True, alpha_recent=True)
    sg.init_cache(wl, buf.k, buf.v, U, buf.cap)
    buf.feat_init(wl.n0, 0)
    sts = []
    for u in range(U):
        st = H.oracle_student(wl, u)
        st.alpha_recent = True
        sts.append(st)
    q, _, _ = _step_tensors(wl)
    for t in range(3):
        sg.queries(wl, t, q)
        buf.decode_step(q)
        torch.cuda.synchronize()
        for u in range(U):
            att = ounit.decode_step(sts[u], W.queries(wl, t, u))
            ok, worst = H.vec_ok(H.to_np(buf.alpha[u, :wl.n0]), sts[u].alpha)
            assert ok, (t, u, "recent alpha", worst)
            assert np.allclose(sts[u].alpha, att.a.mean(axis=0), rtol=1e-14, atol=0)
        buf.global_alpha()
        torch.cuda.synchronize()
        for b in range(wl.batch):
            us = range(b * per_seq, (b + 1) * per_seq)
            g = ofeat.global_alpha([sts[u].alpha for u in us], [sts[u].pos for u in us], per_seq)
            for u, gu in zip(us, g):
                sts[u].alpha = gu
                ok, worst = H.vec_ok(H.to_np(buf.alpha[u, :wl.n0]), gu)
                assert ok, (t, u, "global alpha", worst)
