"""GPU parity at every workload's stated size, step count and launch
configuration (the ones the benchmark times), in lockstep with the oracle on
sampled units: unit 0, the last unit and six seeded random units (every unit
of workload 2).  Before each step the sampled units' device state is replaced
by the oracle's (rows, alpha/N/Z, positions, the query ring), so a near-tie in
one step cannot carry into the next; the other units run on.

* workload 2: 8 units, 4097 -> 1024 at step 0 (chunked decode + stand-alone
  selection), then 255 single-launch steps 1025 -> 1024 in capacity-1025
  buffers, through the entropy window's retire (steps 64..255);
* workload 3: 4096 units, 16385 -> 4096, then 127 single-launch steps
  4097 -> 4096 in capacity-4097 buffers;
* workload 4: 1024 units, 32769 -> 3277 with the 4->64->64->1 policy, decode
  steps 1..63 in capacity-3341 buffers, then the block eviction 3341 -> 3277
  at step 64;
* workload 5: the student (2048 units, 8193 -> 2048, then 2049 -> 2048) and
  the never-pruned teacher (8193..8256 rows), all 64 steps.
"""
import gc

import numpy as np
import pytest
import torch

from oracle import unit as ounit
from synth import gpu as sg
from synth import workloads as W

from . import harness as H
from .test_gpu_step import _buffers, _check_decode, _policy, _step_tensors

pytestmark = pytest.mark.gpu


def _release():
    gc.collect()
    torch.cuda.empty_cache()


def _sample(U, seed):
    if U <= 8:
        return list(range(U))
    rng = np.random.default_rng(seed)
    return sorted({0, U - 1, *rng.choice(np.arange(1, U - 1), 6, replace=False).tolist()})


def _check_step_with_eviction(wl, buf, budget, sts, sample, outn, sc, kp, pnp, t):
    amb_total = 0
    for u in sample:
        st = sts[u]
        att = ounit.decode_step(st, *H.step_inputs_np(wl, t, u))
        assert H.rel_err_rows(outn[u], att.o) <= H.OUT_TOL, (t, u)
        s_or = ounit.scores(st, pnp, wl.hidden)
        ok, worst = H.vec_ok(sc[u], s_or)                # uploaded rows are in oracle order
        assert ok, (t, u, "scores", worst)
        post = H.download_unit(buf, u)
        ok, amb, flips = H.selection_check(s_or, st.pos, post["pos"], budget)
        assert ok, (t, u, amb, flips)
        amb_total += amb
        pre_pos = st.pos.copy()
        # exact: the oracle's selection and compaction on the GPU's own scores
        assert np.array_equal(kp[u], H.oracle_slot_map(sc[u], pre_pos, budget)), (t, u)
        slot_map = ounit.evict(st, s_or, budget)
        if flips == 0:
            # the oracle's own step: the same slot map, rows with its post-step state
            assert np.array_equal(kp[u], slot_map) and np.array_equal(post["pos"], st.pos), (t, u)
            Z, N = st.hist.sums()
            for name, ref in (("alpha", st.alpha), ("den", Z), ("num", N)):
                ok, worst = H.vec_ok(post[name], ref)
                assert ok, (t, u, name, worst)
            assert H.rel_err_rows(post["k"], st.K) == 0 and H.rel_err_rows(post["v"], st.V) == 0
    return amb_total


def _upload(buf, sts, sample):
    for u in sample:
        H.upload_unit(buf, u, sts[u])
    H.set_host_fields(buf, sts[sample[0]])


def _evict_step(wl, buf, pol, budget, q, kn, vn, sts, sample, pnp, t):
    U = wl.units
    L = buf.kv.len + 1
    scores = torch.empty((U, L), dtype=torch.float32, device="cuda")
    kept = torch.empty((U, min(L, budget)), dtype=torch.int32, device="cuda")
    out = buf.decode_evict(pol, budget, q, kn, vn, scores_out=scores, kept_out=kept)
    torch.cuda.synchronize()
    return _check_step_with_eviction(wl, buf, budget, sts, sample, H.to_np(out), H.to_np(scores),
                                     H.to_np(kept), pnp, t)


def _run_every_step_evicting(wl):
    """Workloads 2 and 3: compression at step 0, then a single-launch step with
    one eviction every step, in the benchmark's buffers."""
    U = wl.units
    buf = _buffers(wl, capacity=wl.n0 + 1)
    buf.reserve_workspace(wl.n0 + 1)
    sg.init_cache(wl, buf.k, buf.v, U, buf.cap)
    buf.feat_init(wl.n0, 0)
    params, pol = _policy(wl)
    pnp = H.to_np(params)
    sample = _sample(U, wl.seed)
    sts = {u: H.oracle_student(wl, u) for u in sample}
    q, kn, vn = _step_tensors(wl)
    amb = 0
    for t in range(wl.steps):
        if t > 0:
            _upload(buf, sts, sample)
        sg.queries(wl, t, q)
        sg.new_rows(wl, t, kn, vn, U)
        if t % 16 == 0 or t == 1 or t == 64:
            print(f"workload {wl.cid} step {t}: {buf.kv.len + 1} rows", flush=True)
        amb += _evict_step(wl, buf, pol, wl.budget, q, kn, vn, sts, sample, pnp, t)
        if t == 0:
            buf.shrink(wl.budget + 1)              # the benchmark's steady buffers
            buf.reserve_workspace(wl.budget + 1)
    assert buf.feat.step == wl.steps and buf.kv.len == wl.budget
    print(f"workload {wl.cid}: {wl.steps} steps, ambiguous selections excluded: {amb}")
    del buf
    _release()


def test_workload2_as_stated_all_steps():
    wl = W.WORKLOADS[2]
    assert (wl.units, wl.n0, wl.budget, wl.steps, wl.key_structure) == (8, 4096, 1024, 256, "heavy")
    _run_every_step_evicting(wl)


def test_workload3_full_size_all_steps():
    wl = W.WORKLOADS[3]
    assert (wl.units, wl.n0, wl.budget, wl.steps) == (4096, 16384, 4096, 128)
    _run_every_step_evicting(wl)


def test_workload4_full_size_through_the_block_eviction():
    wl = W.WORKLOADS[4]
    U, E = wl.units, wl.evict_every
    assert (U, wl.n0, wl.budget, E, wl.hidden) == (1024, 32768, 3277, 64, (64, 64))
    buf = _buffers(wl, capacity=wl.n0 + 1)
    buf.reserve_workspace(wl.n0 + 1)
    sg.init_cache(wl, buf.k, buf.v, U, buf.cap)
    buf.feat_init(wl.n0, 0)
    params, pol = _policy(wl)
    pnp = H.to_np(params)
    sample = _sample(U, wl.seed)
    sts = {u: H.oracle_student(wl, u) for u in sample}
    q, kn, vn = _step_tensors(wl)
    for t in range(E + 1):
        if t > 0:
            _upload(buf, sts, sample)
        sg.queries(wl, t, q)
        sg.new_rows(wl, t, kn, vn, U)
        if t % 16 == 0 or t == 1:
            print(f"workload 4 step {t}: {buf.kv.len + 1} rows", flush=True)
        if t % E == 0:                                   # eviction steps: 0 and 64
            _evict_step(wl, buf, pol, wl.budget, q, kn, vn, sts, sample, pnp, t)
            if t == 0:
                buf.shrink(wl.budget + E)                # the benchmark's cycle buffers
                buf.reserve_workspace(wl.budget + E)
        else:
            out = buf.decode_step(q, kn, vn)
            torch.cuda.synchronize()
            outn = H.to_np(out)
            for u in sample:
                att = ounit.decode_step(sts[u], *H.step_inputs_np(wl, t, u))
                _check_decode(wl, outn[u], H.download_unit(buf, u), sts[u], att, (t, u))
    assert buf.kv.len == wl.budget and all(st.L == wl.budget for st in sts.values())
    del buf
    _release()


def test_workload5_full_size_student_and_teacher_all_steps():
    wl = W.WORKLOADS[5]
    U = wl.units
    assert (U, wl.n0, wl.budget, wl.steps) == (2048, 8192, 2048, 64)
    stu = _buffers(wl, capacity=wl.n0 + 1)
    stu.reserve_workspace(wl.n0 + 1)
    sg.init_cache(wl, stu.k, stu.v, U, stu.cap)
    stu.feat_init(wl.n0, 0)
    tea = _buffers(wl, capacity=wl.n0 + wl.steps, features=False)
    sg.init_cache(wl, tea.k, tea.v, U, tea.cap, n0=wl.n0)
    tea.kv.len = wl.n0
    params, pol = _policy(wl)
    pnp = H.to_np(params)
    sample = _sample(U, wl.seed)
    sts = {u: H.oracle_student(wl, u) for u in sample}
    tes = {u: H.oracle_teacher(wl, u) for u in sample}
    q, kn, vn = _step_tensors(wl)
    for t in range(wl.steps):
        if t > 0:
            _upload(stu, sts, sample)
        sg.queries(wl, t, q)
        sg.new_rows(wl, t, kn, vn, U)
        if t % 16 == 0 or t == 1:
            print(f"workload 5 step {t}: teacher {tea.kv.len + 1} rows, student "
                  f"{stu.kv.len + 1} rows", flush=True)
        out_t = tea.decode_step(q, kn, vn, features=False)
        torch.cuda.synchronize()
        outn = H.to_np(out_t)
        for u in sample:
            att = ounit.teacher_step(tes[u], *H.step_inputs_np(wl, t, u))
            assert H.rel_err_rows(outn[u], att.o) <= H.OUT_TOL, (t, u)
        _evict_step(wl, stu, pol, wl.budget, q, kn, vn, sts, sample, pnp, t)
        if t == 0:
            stu.shrink(wl.budget + 1)
            stu.reserve_workspace(wl.budget + 1)
    assert tea.kv.len == wl.n0 + wl.steps and stu.kv.len == wl.budget
    del stu, tea
    _release()
