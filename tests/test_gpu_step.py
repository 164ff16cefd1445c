"""GPU parity: the HIP decode step (through the C ABI) against the CPU oracle."""
import math

import numpy as np
import pytest
import torch

from oracle import select as osel
from oracle import unit as ounit
from paper_2608_08878_amd.buffers import DecodeBuffers, make_policy
from synth import gpu as sg
from synth import philox as px
from synth import workloads as W

from . import harness as H

pytestmark = pytest.mark.gpu


def _buffers(wl, capacity=None, features=True, units_override=None):
    return DecodeBuffers(wl.batch, wl.n_layers, wl.n_q_heads, wl.n_kv_heads, wl.head_dim,
                         capacity or wl.capacity, wl.dtype, wl.ent_window, 0.0, features)


def _policy(wl):
    p = torch.empty(wl.n_params, dtype=torch.float32, device="cuda")
    sg.fill_normal(p, wl, W.S_POLICY, 0, 0.1)
    return p, make_policy(p, wl.hidden)


def test_generator_twin_matches_host():
    wl = W.WORKLOADS[3].scaled(batch=1, n_layers=1)
    U, cap = wl.units, 300
    k = torch.empty((U, cap, wl.head_dim), dtype=torch.bfloat16, device="cuda")
    v = torch.empty_like(k)
    sg.init_cache(wl, k, v, U, cap, n0=257)
    torch.cuda.synchronize()
    for u in (0, 5, U - 1):
        assert np.array_equal(H.to_np(k[u, :257]), W.key_rows(wl, u, np.arange(257)))
        assert np.array_equal(H.to_np(v[u, :257]), W.value_rows(wl, u, np.arange(257)))
    q = torch.empty((U, wl.group, wl.head_dim), dtype=torch.bfloat16, device="cuda")
    sg.queries(wl, 7, q)
    for u in (0, U - 1):
        assert np.array_equal(H.to_np(q[u]), W.queries(wl, 7, u))
    for cid in (1, 2, 4):
        w2 = W.WORKLOADS[cid].scaled(batch=1, n_layers=1)
        kk = torch.empty((w2.units, 80, w2.head_dim), dtype=H.torch_dtype(w2), device="cuda")
        sg.fill_rows(kk, w2, "k", w2.units, 80, 0, 80, 0)
        torch.cuda.synchronize()
        for u in (0, w2.units - 1):
            assert np.array_equal(H.to_np(kk[u]), W.key_rows(w2, u, np.arange(80))), cid
    p, _ = _policy(W.WORKLOADS[4])
    assert np.array_equal(H.to_np(p), W.policy_params(W.WORKLOADS[4]))
    # a large sample of raw normals (exercises every branch of the transforms)
    n = 1 << 22
    z = torch.empty(n, dtype=torch.float32, device="cuda")
    sg.fill_normal(z, wl, 9, 3, 1.0)
    assert np.array_equal(H.to_np(z), px.to_f32(px.normal(wl.seed, 9, 3, np.arange(n, dtype=np.uint64))))


def _run_config1():
    wl = W.WORKLOADS[1]
    U, G, D, L, Bgt = wl.units, wl.group, wl.head_dim, wl.n0, wl.budget
    buf = _buffers(wl)
    sg.init_cache(wl, buf.k, buf.v, U, buf.cap)
    buf.feat_init(L, 0)
    q = torch.empty((U, G, D), dtype=torch.float32, device="cuda")
    sg.queries(wl, 0, q)
    out = buf.decode_step(q)
    torch.cuda.synchronize()
    pre = [H.download_unit(buf, u) for u in range(U)]
    params, pol = _policy(wl)
    scores = torch.empty((U, L), dtype=torch.float32, device="cuda")
    kept = torch.empty((U, Bgt), dtype=torch.int32, device="cuda")
    buf.score_evict(pol, Bgt, scores, kept)
    torch.cuda.synchronize()
    post = [H.download_unit(buf, u) for u in range(U)]
    return wl, buf, H.to_np(out), pre, H.to_np(scores), H.to_np(kept), post, H.to_np(params)


def test_config1_single_step_matches_oracle():
    wl, buf, out, pre, scores, kept, post, params = _run_config1()
    assert buf.kv.len == wl.budget
    for u in range(wl.units):
        st = H.oracle_student(wl, u)
        att = ounit.decode_step(st, W.queries(wl, 0, u))
        # attention output (float32 path: far inside the bf16 tolerance)
        assert H.rel_err_rows(out[u], att.o) <= 1e-4
        # features after the step
        Z, N = st.hist.sums()
        for name, ref in (("alpha", st.alpha), ("den", Z), ("num", N),
                          ("vnorm", np.sqrt((st.V ** 2).sum(1)))):
            ok, worst = H.vec_ok(pre[u][name], ref)
            assert ok, (u, name, worst)
        assert np.array_equal(pre[u]["pos"], np.arange(wl.n0))
        s_or = ounit.scores(st, params, wl.hidden)
        ok, worst = H.vec_ok(scores[u], s_or)
        assert ok, (u, "scores", worst)
        # exact: the oracle's selection applied to the GPU's own float32 scores
        layout = H.oracle_slot_map(scores[u], pre[u]["pos"], wl.budget)
        assert np.array_equal(kept[u], layout)
        for name in ("k", "v", "pos", "alpha", "num", "den", "vnorm"):
            assert np.array_equal(post[u][name], pre[u][name][layout]), name
        # end to end against the oracle's own scores, with the near-tie band
        ok, amb, flips = H.selection_check(s_or, pre[u]["pos"], post[u]["pos"], wl.budget)
        assert ok, (u, amb, flips)


def _step_tensors(wl):
    U, G, D = wl.units, wl.group, wl.head_dim
    td = H.torch_dtype(wl)
    q = torch.empty((U, G, D), dtype=td, device="cuda")
    kn = torch.empty((U, D), dtype=td, device="cuda")
    vn = torch.empty_like(kn)
    return q, kn, vn


def _check_decode(wl, out_u, pre_u, st, att, tag):
    assert H.rel_err_rows(out_u, att.o) <= H.OUT_TOL, tag
    Z, N = st.hist.sums()
    assert np.array_equal(pre_u["pos"], st.pos), tag
    for name, ref in (("alpha", st.alpha), ("den", Z), ("num", N),
                      ("vnorm", np.sqrt((st.V ** 2).sum(1)))):
        ok, worst = H.vec_ok(pre_u[name], ref)
        assert ok, (tag, name, worst)


def _check_evict(wl, budget, pre_u, scores_u, kept_u, post_u, s_or, tag):
    ok, worst = H.vec_ok(scores_u, s_or)
    assert ok, (tag, "scores", worst)
    layout = H.oracle_slot_map(scores_u, pre_u["pos"], budget)
    assert np.array_equal(kept_u, layout), tag
    for name in ("k", "v", "pos", "alpha", "num", "den", "vnorm"):
        assert np.array_equal(post_u[name], pre_u[name][layout]), (tag, name)
    ok, amb, flips = H.selection_check(s_or, pre_u["pos"], post_u["pos"], budget)
    assert ok, (tag, amb, flips)
    return amb, flips


def test_multistep_lockstep_with_window_retire():
    """Mistral-shaped heads (G=4, d=128, bf16, heavy-hitter keys) on 2 units, 90
    steps: step 0 compresses 701 -> 256 rows, later steps evict one row; from
    step 64 on the entropy window retires.  Every step starts the device from
    the oracle's state (so a near-tie can never cascade) and compares."""
    wl = W.WORKLOADS[2].scaled(n_kv_heads=2, n_q_heads=8, n0=700, budget=256, steps=90)
    U = wl.units
    buf = _buffers(wl)
    params, pol = _policy(wl)
    pnp = H.to_np(params)
    sts = [H.oracle_student(wl, u) for u in range(U)]
    q, kn, vn = _step_tensors(wl)
    amb_total = 0
    for t in range(wl.steps):
        for u in range(U):
            H.upload_unit(buf, u, sts[u])
        H.set_host_fields(buf, sts[0])
        sg.queries(wl, t, q)
        sg.new_rows(wl, t, kn, vn, U)
        out = buf.decode_step(q, kn, vn)
        torch.cuda.synchronize()
        outn = H.to_np(out)
        pre = [H.download_unit(buf, u) for u in range(U)]
        L = buf.kv.len
        scores = torch.empty((U, L), dtype=torch.float32, device="cuda")
        kept = torch.empty((U, min(L, wl.budget)), dtype=torch.int32, device="cuda")
        buf.score_evict(pol, wl.budget, scores, kept)
        torch.cuda.synchronize()
        post = [H.download_unit(buf, u) for u in range(U)]
        sc, kp = H.to_np(scores), H.to_np(kept)
        for u in range(U):
            att = ounit.decode_step(sts[u], *H.step_inputs_np(wl, t, u))
            _check_decode(wl, outn[u], pre[u], sts[u], att, (t, u))
            s_or = ounit.scores(sts[u], pnp, wl.hidden)
            amb, _ = _check_evict(wl, wl.budget, pre[u], sc[u], kp[u], post[u], s_or, (t, u))
            amb_total += amb
            ounit.evict(sts[u], s_or, wl.budget)
    print("ambiguous selections excluded:", amb_total)


def test_free_running_trajectory_until_first_near_tie():
    """Device and oracle each run their own trajectory from the same inputs;
    they must agree until a selection lands inside the near-tie band."""
    wl = W.WORKLOADS[2].scaled(n_kv_heads=2, n_q_heads=8, n0=400, budget=160, steps=72)
    U = wl.units
    buf = _buffers(wl)
    sg.init_cache(wl, buf.k, buf.v, U, buf.cap)
    buf.feat_init(wl.n0, 0)
    params, pol = _policy(wl)
    pnp = H.to_np(params)
    sts = [H.oracle_student(wl, u) for u in range(U)]
    q, kn, vn = _step_tensors(wl)
    for t in range(wl.steps):
        sg.queries(wl, t, q)
        sg.new_rows(wl, t, kn, vn, U)
        out = buf.decode_step(q, kn, vn)
        torch.cuda.synchronize()
        outn = H.to_np(out)
        pre = [H.download_unit(buf, u) for u in range(U)]      # same slot order as the oracle
        buf.score_evict(pol, wl.budget)
        torch.cuda.synchronize()
        diverged = False
        for u in range(U):
            att = ounit.decode_step(sts[u], *H.step_inputs_np(wl, t, u))
            _check_decode(wl, outn[u], pre[u], sts[u], att, (t, u))
            s_or = ounit.scores(sts[u], pnp, wl.hidden)
            post = H.download_unit(buf, u)
            ok, amb, flips = H.selection_check(s_or, sts[u].pos, post["pos"], wl.budget)
            assert ok, (t, u, amb, flips)
            ounit.evict(sts[u], s_or, wl.budget)
            diverged |= flips > 0
        if diverged:
            print("trajectories parted at a near-tie at step", t)
            return


@pytest.mark.parametrize("units_batch,n0", [((1, 2), 6000), ((16, 8), 5000)])
def test_chunked_and_large_unit_paths(units_batch, n0):
    """Caches too long for LDS (6001 rows) or spread over several workgroups
    (few units), and the one-workgroup-per-unit path at 128 units; sampled units
    are compared one step from a fresh state, then a compression step."""
    batch, nkv = units_batch
    wl = W.WORKLOADS[3].scaled(batch=batch, n_layers=1, n_kv_heads=nkv, n_q_heads=4 * nkv,
                               n0=n0, budget=1500, steps=2)
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
    out = buf.decode_step(q, kn, vn)
    torch.cuda.synchronize()
    sample = sorted({0, U - 1, U // 2})
    pre = {u: H.download_unit(buf, u) for u in sample}
    L = buf.kv.len
    scores = torch.empty((U, L), dtype=torch.float32, device="cuda")
    kept = torch.empty((U, wl.budget), dtype=torch.int32, device="cuda")
    buf.score_evict(pol, wl.budget, scores, kept)
    torch.cuda.synchronize()
    outn, sc, kp = H.to_np(out), H.to_np(scores), H.to_np(kept)
    for u in sample:
        st = H.oracle_student(wl, u)
        att = ounit.decode_step(st, *H.step_inputs_np(wl, 0, u))
        _check_decode(wl, outn[u], pre[u], st, att, u)
        s_or = ounit.scores(st, pnp, wl.hidden)
        _check_evict(wl, wl.budget, pre[u], sc[u], kp[u], H.download_unit(buf, u), s_or, u)


def test_teacher_plain_attention_and_budget_covering_cache():
    """feat = NULL gives plain attention over the whole cache; a student whose
    budget covers the cache keeps every row bit-identical and attends exactly
    like that teacher."""
    wl = W.WORKLOADS[2].scaled(n_kv_heads=2, n_q_heads=8, n0=900, budget=5000, steps=3)
    U = wl.units
    tb = _buffers(wl, features=False)
    sb = _buffers(wl)
    for b in (tb, sb):
        sg.init_cache(wl, b.k, b.v, U, b.cap)
    tb.kv.len = wl.n0
    sb.feat_init(wl.n0, 0)
    params, pol = _policy(wl)
    q, kn, vn = _step_tensors(wl)
    tes = [H.oracle_teacher(wl, u) for u in range(U)]
    for t in range(wl.steps):
        sg.queries(wl, t, q)
        sg.new_rows(wl, t, kn, vn, U)
        ot = tb.decode_step(q, kn, vn, features=False)
        os_ = sb.decode_step(q, kn, vn)
        k_before = sb.k.clone()
        sb.score_evict(pol, wl.budget)
        torch.cuda.synchronize()
        assert torch.equal(ot, os_)
        assert torch.equal(sb.k, k_before) and sb.kv.len == tb.kv.len
        otn = H.to_np(ot)
        for u in range(U):
            att = ounit.teacher_step(tes[u], *H.step_inputs_np(wl, t, u))
            assert H.rel_err_rows(otn[u], att.o) <= H.OUT_TOL


def _tiny_state_after_one_step(n0=300):
    wl = W.WORKLOADS[2].scaled(n_kv_heads=2, n_q_heads=8, n0=n0, budget=100, steps=1)
    buf = _buffers(wl)
    sg.init_cache(wl, buf.k, buf.v, wl.units, buf.cap)
    buf.feat_init(wl.n0, 0)
    q, kn, vn = _step_tensors(wl)
    sg.queries(wl, 0, q)
    sg.new_rows(wl, 0, kn, vn, wl.units)
    buf.decode_step(q, kn, vn)
    torch.cuda.synchronize()
    return wl, buf


def _policy_from(values, hidden=(1,)):
    p = torch.tensor(values, dtype=torch.float32, device="cuda")
    return p, make_policy(p, hidden)


@pytest.mark.parametrize("case", ["all_equal", "neg_zero", "nan", "keep_newest", "keep_oldest",
                                  "budget_one", "budget_covers"])
def test_adversarial_selection(case):
    wl, buf = _tiny_state_after_one_step()
    U, L = wl.units, buf.kv.len
    budget = {"budget_one": 1, "budget_covers": L}.get(case, 100)
    # 4 -> 1 -> 1 MLP: params W1[1][4], b1[1], w_out[1], b_out
    vals = {"all_equal": [0, 0, 0, 0, 0, 1, 0.5], "neg_zero": [0, 0, 0, 0, 0, -1, -0.0],
            "nan": [0, 0, 0, 0, 0, 1, float("nan")], "keep_newest": [0, 0, 0, 1, 0, 1, 0],
            "keep_oldest": [0, 0, 0, -1, 2, 1, 0], "budget_one": [1, 0, 0, 0, 0, 1, 0],
            "budget_covers": [1, 0, 0, 0, 0, 1, 0]}[case]
    p, pol = _policy_from(vals)
    pre = [H.download_unit(buf, u) for u in range(U)]
    scores = torch.empty((U, L), dtype=torch.float32, device="cuda")
    kept = torch.empty((U, min(budget, L)), dtype=torch.int32, device="cuda")
    buf.score_evict(pol, budget, scores, kept)
    torch.cuda.synchronize()
    sc, kp = H.to_np(scores), H.to_np(kept)
    for u in range(U):
        post = H.download_unit(buf, u)
        layout = H.oracle_slot_map(sc[u], pre[u]["pos"], budget)
        assert np.array_equal(kp[u], layout), case
        for name in ("k", "v", "pos", "alpha", "num", "den", "vnorm"):
            assert np.array_equal(post[name], pre[u][name][layout]), (case, name)
        if case in ("all_equal", "neg_zero", "nan", "keep_oldest"):
            assert sorted(post["pos"]) == list(range(budget)), case      # earliest tokens kept
        if case == "keep_newest":
            assert sorted(post["pos"]) == list(range(L - budget, L))
        if case == "budget_covers":
            assert np.array_equal(post["k"], pre[u]["k"]) and buf.kv.len == L


def test_long_cache_selection_uses_workspace_keys():
    """A cache longer than the register-resident select (8192 rows) goes through
    the workspace-key path; compare a compression step with the oracle."""
    wl = W.WORKLOADS[4].scaled(batch=1, n_layers=1, n_kv_heads=2, n_q_heads=8, n0=12000,
                               budget=1200, steps=1)
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
    out = buf.decode_step(q, kn, vn)
    torch.cuda.synchronize()
    pre = [H.download_unit(buf, u) for u in range(U)]
    L = buf.kv.len
    scores = torch.empty((U, L), dtype=torch.float32, device="cuda")
    kept = torch.empty((U, wl.budget), dtype=torch.int32, device="cuda")
    buf.score_evict(pol, wl.budget, scores, kept)
    torch.cuda.synchronize()
    outn, sc, kp = H.to_np(out), H.to_np(scores), H.to_np(kept)
    for u in range(U):
        st = H.oracle_student(wl, u)
        att = ounit.decode_step(st, *H.step_inputs_np(wl, 0, u))
        _check_decode(wl, outn[u], pre[u], st, att, u)
        s_or = ounit.scores(st, pnp, wl.hidden)
        _check_evict(wl, wl.budget, pre[u], sc[u], kp[u], H.download_unit(buf, u), s_or, u)


@pytest.mark.parametrize("dtype,n0,head_dim", [("bf16", 1000, 128), ("bf16", 6000, 128),
                                               ("bf16", 900, 64), ("f32", 1000, 128),
                                               ("f32", 700, 64)])
def test_retire_recomputes_the_added_weights_bit_exactly(dtype, n0, head_dim):
    """Window w = 2, the same query every step, no appends: every step adds the
    same per-row contribution c, and from step 2 on retires the one added two
    steps earlier.  The window sums are then 2c after every step, bit for bit,
    only if the retire reproduces the added weights exactly (the recomputed
    logits, the stored max and 1/l, the same exp and the same head order)."""
    wl = W.WORKLOADS[2].scaled(n_kv_heads=2, n_q_heads=8, n0=n0, dtype=dtype, head_dim=head_dim,
                               ent_window=2, append=False, steps=5)
    U = wl.units
    buf = _buffers(wl, capacity=n0)
    buf.reserve_workspace(n0)
    sg.init_cache(wl, buf.k, buf.v, U, buf.cap)
    buf.feat_init(n0, 0)
    q = torch.empty((U, wl.group, head_dim), dtype=H.torch_dtype(wl), device="cuda")
    sg.queries(wl, 0, q)
    dens, nums = [], []
    for t in range(5):
        buf.decode_step(q)
        torch.cuda.synchronize()
        dens.append(buf.den[:, :n0].clone())
        nums.append(buf.num[:, :n0].clone())
    assert torch.all(dens[1] > 0)
    for t in (2, 3, 4):
        assert torch.equal(dens[t], dens[1]), t
        assert torch.equal(nums[t], nums[1]), t
    # and the first step's contribution is exactly half of the two-step window
    assert torch.equal(dens[0] * 2, dens[1])


@pytest.mark.parametrize("n0,budget", [(3000, 900), (6000, 1500)])
def test_fused_step_equals_decode_then_evict(n0, budget):
    """dc_decode_evict (one launch where the cache fits on chip; the chunked
    decode plus the separate eviction otherwise) leaves every buffer, output,
    score and slot map bit-identical to dc_decode_step + dc_score_evict."""
    wl = W.WORKLOADS[2].scaled(n_kv_heads=2, n_q_heads=8, n0=n0, budget=budget, steps=70)
    U = wl.units
    bufs = [_buffers(wl), _buffers(wl)]
    for b in bufs:
        b.reserve_workspace(wl.capacity)
        sg.init_cache(wl, b.k, b.v, U, b.cap)
        b.feat_init(wl.n0, 0)
    params, pol = _policy(wl)
    q, kn, vn = _step_tensors(wl)
    for t in range(wl.steps):
        sg.queries(wl, t, q)
        sg.new_rows(wl, t, kn, vn, U)
        L = bufs[0].kv.len + 1
        sc = [torch.empty((U, L), dtype=torch.float32, device="cuda") for _ in range(2)]
        kp = [torch.empty((U, min(L, budget)), dtype=torch.int32, device="cuda") for _ in range(2)]
        o0 = bufs[0].decode_step(q, kn, vn)
        bufs[0].score_evict(pol, budget, sc[0], kp[0])
        o1 = bufs[1].decode_evict(pol, budget, q, kn, vn, scores_out=sc[1], kept_out=kp[1])
        torch.cuda.synchronize()
        assert torch.equal(o0, o1), t
        assert torch.equal(sc[0], sc[1]) and torch.equal(kp[0], kp[1]), t
        assert bufs[0].kv.len == bufs[1].kv.len and bufs[0].feat.step == bufs[1].feat.step
        n = bufs[0].kv.len
        for name in ("k", "v", "alpha", "num", "den", "pos", "vnorm", "qring", "qstat"):
            a0, a1 = getattr(bufs[0], name), getattr(bufs[1], name)
            if name in ("qring", "qstat"):
                assert torch.equal(a0, a1), (t, name)
            else:
                assert torch.equal(a0[:, :n], a1[:, :n]), (t, name)


def test_shrink_after_compression_keeps_every_bit():
    """Moving the live rows into budget-sized buffers after the compression step
    changes no output, score, slot map or state bit of the following steps
    (through the window retire)."""
    wl = W.WORKLOADS[2].scaled(n_kv_heads=2, n_q_heads=8, n0=3000, budget=700, steps=70)
    U, budget = wl.units, wl.budget
    bufs = [_buffers(wl), _buffers(wl)]
    for b in bufs:
        sg.init_cache(wl, b.k, b.v, U, b.cap)
        b.feat_init(wl.n0, 0)
    params, pol = _policy(wl)
    q, kn, vn = _step_tensors(wl)
    for t in range(wl.steps):
        sg.queries(wl, t, q)
        sg.new_rows(wl, t, kn, vn, U)
        L = bufs[0].kv.len + 1
        sc = [torch.empty((U, L), dtype=torch.float32, device="cuda") for _ in range(2)]
        kp = [torch.empty((U, min(L, budget)), dtype=torch.int32, device="cuda") for _ in range(2)]
        outs = [b.decode_evict(pol, budget, q, kn, vn, scores_out=s, kept_out=k)
                for b, s, k in zip(bufs, sc, kp)]
        if t == 0:
            bufs[1].shrink(budget + 1)
            assert bufs[1].cap == budget + 1 and bufs[1].k.shape[1] == budget + 1
        torch.cuda.synchronize()
        assert torch.equal(outs[0], outs[1]), t
        assert torch.equal(sc[0], sc[1]) and torch.equal(kp[0], kp[1]), t
        n = bufs[0].kv.len
        for name in ("k", "v", "alpha", "num", "den", "pos", "vnorm", "qring", "qstat"):
            a0, a1 = getattr(bufs[0], name), getattr(bufs[1], name)
            if name in ("qring", "qstat"):
                assert torch.equal(a0, a1), (t, name)
            else:
                assert torch.equal(a0[:, :n], a1[:, :n]), (t, name)


def test_two_layer_policy_periodic_eviction():
    """The 4->64->64->1 policy (weights staged in LDS) on the long-context recipe
    with an eviction every 4th step: the fused decode+evict launch leaves every
    buffer bit-identical to decode then score/evict (register-resident path), and
    the scores match the oracle's MLP applied to the step's features."""
    from oracle import features as ofeat
    from oracle import policy as opol
    wl = W.WORKLOADS[4].scaled(batch=1, n_layers=1, n_kv_heads=2, n_q_heads=8, n0=3000,
                               budget=700, steps=70)
    U, budget = wl.units, wl.budget
    bufs = [_buffers(wl), _buffers(wl)]
    for b in bufs:
        sg.init_cache(wl, b.k, b.v, U, b.cap)
        b.feat_init(wl.n0, 0)
    params, pol = _policy(wl)
    pnp = H.to_np(params)
    q, kn, vn = _step_tensors(wl)
    for t in range(wl.steps):
        sg.queries(wl, t, q)
        sg.new_rows(wl, t, kn, vn, U)
        if t % 4 == 0:
            L = bufs[0].kv.len + 1
            sc = [torch.empty((U, L), dtype=torch.float32, device="cuda") for _ in range(2)]
            kp = [torch.empty((U, min(L, budget)), dtype=torch.int32, device="cuda") for _ in range(2)]
            o0 = bufs[0].decode_step(q, kn, vn)
            torch.cuda.synchronize()
            pre = [H.download_unit(bufs[0], u) for u in range(U)]
            T = bufs[0].feat.next_pos
            bufs[0].score_evict(pol, budget, sc[0], kp[0])
            o1 = bufs[1].decode_evict(pol, budget, q, kn, vn, scores_out=sc[1], kept_out=kp[1])
            torch.cuda.synchronize()
            assert torch.equal(sc[0], sc[1]) and torch.equal(kp[0], kp[1]), t
            scn = H.to_np(sc[0])
            for u in range(U):
                x = ofeat.feature_matrix(pre[u]["alpha"], pre[u]["v"], pre[u]["den"],
                                         pre[u]["num"], pre[u]["pos"], T)
                ok, worst = H.vec_ok(scn[u], opol.scores(pnp, x, wl.hidden))
                assert ok, (t, u, worst)
        else:
            o0 = bufs[0].decode_step(q, kn, vn)
            o1 = bufs[1].decode_step(q, kn, vn)
            torch.cuda.synchronize()
        assert torch.equal(o0, o1), t
        assert bufs[0].kv.len == bufs[1].kv.len
        n = bufs[0].kv.len
        for name in ("k", "v", "alpha", "num", "den", "pos", "vnorm", "qring", "qstat"):
            a0, a1 = getattr(bufs[0], name), getattr(bufs[1], name)
            if name in ("qring", "qstat"):
                assert torch.equal(a0, a1), (t, name)
            else:
                assert torch.equal(a0[:, :n], a1[:, :n]), (t, name)


def test_dynamic_budget_trajectory():
    """The budget of every step follows max(floor(0.25 T), 32) (App. D protocol):
    step 0 compresses 301 -> 75 rows, then the budget grows by one every four
    tokens.  Fused steps on the device against the oracle until a near-tie."""
    from paper_2608_08878_amd import binding as B
    wl = W.WORKLOADS[2].scaled(n_kv_heads=2, n_q_heads=8, n0=300, budget=75, steps=80)
    U = wl.units
    buf = _buffers(wl)
    sg.init_cache(wl, buf.k, buf.v, U, buf.cap)
    buf.feat_init(wl.n0, 0)
    params, pol = _policy(wl)
    pnp = H.to_np(params)
    sts = [H.oracle_student(wl, u) for u in range(U)]
    q, kn, vn = _step_tensors(wl)
    lens = []
    for t in range(wl.steps):
        sg.queries(wl, t, q)
        sg.new_rows(wl, t, kn, vn, U)
        budget = B.dc_dynamic_budget(0.25, buf.feat.next_pos + 1, 32)
        assert budget == osel.dynamic_budget(0.25, wl.n0 + t + 1, 32)
        buf.decode_evict(pol, budget, q, kn, vn)
        torch.cuda.synchronize()
        lens.append(buf.kv.len)
        diverged = False
        for u in range(U):
            ounit.decode_step(sts[u], *H.step_inputs_np(wl, t, u))
            s_or = ounit.scores(sts[u], pnp, wl.hidden)
            post = H.download_unit(buf, u)
            ok, amb, flips = H.selection_check(s_or, sts[u].pos, post["pos"], budget)
            assert ok, (t, u, amb, flips)
            ounit.evict(sts[u], s_or, budget)
            assert buf.kv.len == sts[u].L
            if flips == 0:      # both trajectories store the kept rows in the same slots
                assert np.array_equal(post["pos"], sts[u].pos), (t, u)
            diverged |= flips > 0
        if diverged:
            print("trajectories parted at a near-tie at step", t)
            break
    assert lens[0] == 75 and max(lens) <= 95


@pytest.mark.parametrize("n_q,n_kv,d", [(2, 2, 128), (4, 2, 128), (16, 2, 128), (8, 2, 64),
                                        (16, 2, 64)])
def test_fused_step_across_head_groups_and_dims(n_q, n_kv, d):
    """The single-launch step (dc_decode_evict) at G = 1, 2, 8 and head_dim 64,
    in lockstep with the oracle through the window retire: 70 steps, step 0
    compresses 701 -> 256 rows; every step starts from the oracle's state."""
    wl = W.WORKLOADS[2].scaled(n_kv_heads=n_kv, n_q_heads=n_q, head_dim=d, n0=700, budget=256,
                               steps=70)
    U = wl.units
    buf = _buffers(wl)
    params, pol = _policy(wl)
    pnp = H.to_np(params)
    sts = [H.oracle_student(wl, u) for u in range(U)]
    q, kn, vn = _step_tensors(wl)
    amb_total = 0
    for t in range(wl.steps):
        for u in range(U):
            H.upload_unit(buf, u, sts[u])
        H.set_host_fields(buf, sts[0])
        sg.queries(wl, t, q)
        sg.new_rows(wl, t, kn, vn, U)
        L = buf.kv.len + 1
        scores = torch.empty((U, L), dtype=torch.float32, device="cuda")
        kept = torch.empty((U, min(L, wl.budget)), dtype=torch.int32, device="cuda")
        out = buf.decode_evict(pol, wl.budget, q, kn, vn, scores_out=scores, kept_out=kept)
        torch.cuda.synchronize()
        outn, sc, kp = H.to_np(out), H.to_np(scores), H.to_np(kept)
        for u in range(U):
            att = ounit.decode_step(sts[u], *H.step_inputs_np(wl, t, u))
            assert H.rel_err_rows(outn[u], att.o) <= H.OUT_TOL, (t, u)
            s_or = ounit.scores(sts[u], pnp, wl.hidden)
            ok, worst = H.vec_ok(sc[u], s_or)        # uploaded rows are in the oracle's order
            assert ok, (t, u, "scores", worst)
            post = H.download_unit(buf, u)
            ok, amb, flips = H.selection_check(s_or, sts[u].pos, post["pos"], wl.budget)
            assert ok, (t, u, amb, flips)
            amb_total += amb
            pre_pos = sts[u].pos.copy()
            # exact: the oracle's selection and compaction on the GPU's own scores
            assert np.array_equal(kp[u], H.oracle_slot_map(sc[u], pre_pos, wl.budget)), (t, u)
            slot_map = ounit.evict(sts[u], s_or, wl.budget)
            if flips == 0:
                # the oracle's own step: same slot map, rows carrying its post-step features
                assert np.array_equal(kp[u], slot_map) and np.array_equal(post["pos"], sts[u].pos)
                Z, N = sts[u].hist.sums()
                for name, ref in (("alpha", sts[u].alpha), ("den", Z), ("num", N)):
                    ok, worst = H.vec_ok(post[name], ref)
                    assert ok, (t, u, name, worst)
    print("ambiguous selections excluded:", amb_total)


@pytest.mark.parametrize("dtype,head_dim,mode", [("bf16", 128, "one_launch"),
                                                 ("bf16", 128, "two_calls"),
                                                 ("f32", 64, "one_launch")])
def test_decode_from_an_empty_cache(dtype, head_dim, mode):
    """The first append onto an empty cache (one row: weight 1, entropy 0), then
    caches shorter than one 16-row tile while they grow to the budget of 6
    (no eviction: every row kept), then one eviction per step, past step 64
    where the entropy window starts to retire.  Device and oracle run their
    own trajectories and must agree until a selection lands in the near-tie band."""
    budget = 6
    wl = W.WORKLOADS[2].scaled(n_kv_heads=2, n_q_heads=8, n0=0, budget=budget, steps=80,
                               dtype=dtype, head_dim=head_dim)
    U = wl.units
    buf = _buffers(wl)
    buf.reserve_workspace(wl.capacity)
    buf.feat_init(0, 0)
    params, pol = _policy(wl)
    pnp = H.to_np(params)
    sts = [H.oracle_student(wl, u) for u in range(U)]
    assert all(st.L == 0 for st in sts)
    q, kn, vn = _step_tensors(wl)
    slot_pos = [np.zeros(0, np.int64) for _ in range(U)]    # device slot order before the step
    print(f"empty cache: {dtype} d={head_dim} {mode}", flush=True)
    for t in range(wl.steps):
        sg.queries(wl, t, q)
        sg.new_rows(wl, t, kn, vn, U)
        L = buf.kv.len + 1
        scores = torch.empty((U, L), dtype=torch.float32, device="cuda")
        kept = torch.empty((U, min(L, budget)), dtype=torch.int32, device="cuda")
        if mode == "one_launch":
            out = buf.decode_evict(pol, budget, q, kn, vn, scores_out=scores, kept_out=kept)
        else:
            out = buf.decode_step(q, kn, vn)
            buf.score_evict(pol, budget, scores, kept)
        torch.cuda.synchronize()
        assert buf.kv.len == min(L, budget)
        outn, sc, kp = H.to_np(out), H.to_np(scores), H.to_np(kept)
        diverged = False
        for u in range(U):
            st = sts[u]
            att = ounit.decode_step(st, *H.step_inputs_np(wl, t, u))
            assert H.rel_err_rows(outn[u], att.o) <= H.OUT_TOL, (t, u)
            if t == 0:
                assert np.allclose(att.o, st.V[0][None, :].repeat(wl.group, 0))   # one row: its value
            s_or = ounit.scores(st, pnp, wl.hidden)
            dev_pos = np.append(slot_pos[u], t)                 # the appended row takes the last slot
            assert np.array_equal(dev_pos, st.pos), (t, u)       # same compaction order so far
            o_dev, o_or = np.argsort(dev_pos), np.argsort(st.pos)
            assert np.array_equal(dev_pos[o_dev], st.pos[o_or]), (t, u)
            ok, worst = H.vec_ok(sc[u][o_dev], s_or[o_or])
            assert ok, (t, u, "scores", worst)
            post = H.download_unit(buf, u)
            # exact: the oracle's selection and compaction applied to the device's scores
            assert np.array_equal(kp[u], H.oracle_slot_map(sc[u], dev_pos, budget)), (t, u)
            assert np.array_equal(post["pos"], dev_pos[kp[u]]), (t, u)
            ok, amb, flips = H.selection_check(s_or, st.pos, post["pos"], budget)
            assert ok, (t, u, amb, flips)
            diverged |= flips > 0
            pre_pos = st.pos.copy()
            ounit.evict(st, s_or, budget)
            if flips == 0:
                Z, N = st.hist.sums()
                pb = H.by_position(post)
                o = np.argsort(st.pos)
                assert np.array_equal(pb["pos"], st.pos[o]), (t, u)
                for name, ref in (("k", st.K), ("v", st.V)):
                    assert H.rel_err_rows(pb[name], ref[o]) <= H.OUT_TOL, (t, u, name)
                for name, ref in (("alpha", st.alpha), ("den", Z), ("num", N),
                                  ("vnorm", np.sqrt((st.V ** 2).sum(1)))):
                    ok, worst = H.vec_ok(pb[name], ref[o])
                    assert ok, (t, u, name, worst)
            assert len(pre_pos) == L
            slot_pos[u] = post["pos"].astype(np.int64)
        if diverged:
            print("trajectories parted at a near-tie at step", t)
            return


@pytest.mark.parametrize("n_q,n_kv,d", [(2, 2, 128), (4, 2, 128), (8, 2, 128), (16, 2, 128),
                                        (2, 2, 64), (8, 2, 64), (16, 2, 64)])
def test_chunked_step_across_head_groups_and_dims(n_q, n_kv, d):
    """The chunked decode on two units of 5001 rows (ten chunks, the last one
    ragged; each chunk's K and V passes in one workgroup, the chunks combined at
    their common maximum) at G = 1, 2, 4, 8 and head_dim 64 and 128, with an
    entropy window of 2 so that the third step retires; then a compression
    step through the stand-alone selection, all against the oracle."""
    wl = W.WORKLOADS[2].scaled(n_kv_heads=n_kv, n_q_heads=n_q, head_dim=d, n0=5000, budget=1200,
                               steps=3, ent_window=2)
    U = wl.units
    buf = _buffers(wl)
    buf.reserve_workspace(wl.capacity)
    sg.init_cache(wl, buf.k, buf.v, U, buf.cap)
    buf.feat_init(wl.n0, 0)
    params, pol = _policy(wl)
    pnp = H.to_np(params)
    sts = [H.oracle_student(wl, u) for u in range(U)]
    q, kn, vn = _step_tensors(wl)
    print(f"chunked G={wl.group} d={d}", flush=True)
    for t in range(wl.steps):
        sg.queries(wl, t, q)
        sg.new_rows(wl, t, kn, vn, U)
        out = buf.decode_step(q, kn, vn)
        torch.cuda.synchronize()
        outn = H.to_np(out)
        for u in range(U):
            att = ounit.decode_step(sts[u], *H.step_inputs_np(wl, t, u))
            _check_decode(wl, outn[u], H.download_unit(buf, u), sts[u], att, (t, u))
    L = buf.kv.len
    assert L == 5003
    pre = [H.download_unit(buf, u) for u in range(U)]
    scores = torch.empty((U, L), dtype=torch.float32, device="cuda")
    kept = torch.empty((U, wl.budget), dtype=torch.int32, device="cuda")
    buf.score_evict(pol, wl.budget, scores, kept)
    torch.cuda.synchronize()
    sc, kp = H.to_np(scores), H.to_np(kept)
    for u in range(U):
        s_or = ounit.scores(sts[u], pnp, wl.hidden)
        _check_evict(wl, wl.budget, pre[u], sc[u], kp[u], H.download_unit(buf, u), s_or, ("c", u))
