"""GPU parity of per-unit budgets on ragged caches (the head-level hybrid of
the appendix: some heads keep their full cache, the others a budget; Sec. 3.2
per-unit top-B): every unit keeps its own row count on the device, decode runs
the chunked kernels per unit, and each unit's selection follows its budget.
Free-running device and oracle trajectories until a selection lands in the
near-tie band."""
import numpy as np
import pytest
import torch

from oracle import sampling as osmp
from oracle import unit as ounit
from paper_2608_08878_amd import binding as B
from paper_2608_08878_amd.buffers import DecodeBuffers
from synth import gpu as sg
from synth import workloads as W

from . import harness as H
from .test_gpu_sampling import _logz_tol, _sampled_check
from .test_gpu_step import _check_decode, _policy, _step_tensors

pytestmark = pytest.mark.gpu


def _download(buf, u, L):
    d = {"k": H.to_np(buf.k[u, :L]).astype(np.float64), "v": H.to_np(buf.v[u, :L]).astype(np.float64),
         "pos": H.to_np(buf.pos[u, :L]).astype(np.int64), "alpha": H.to_np(buf.alpha[u, :L]),
         "num": H.to_np(buf.num[u, :L]), "den": H.to_np(buf.den[u, :L]),
         "vnorm": H.to_np(buf.vnorm[u, :L])}
    return d


def _ragged_run(budgets, steps, n0=700, gumbel=None, tau=1.0, hidden=None):
    kw = {"hidden": tuple(hidden)} if hidden else {}
    wl = W.WORKLOADS[2].scaled(n_kv_heads=len(budgets), n_q_heads=4 * len(budgets), n0=n0,
                               budget=max(budgets), steps=steps, **kw)
    U = wl.units
    buf = DecodeBuffers(wl.batch, wl.n_layers, wl.n_q_heads, wl.n_kv_heads, wl.head_dim,
                        wl.capacity, wl.dtype, wl.ent_window, 0.0, True, ragged=True)
    buf.reserve_workspace(wl.capacity)
    sg.init_cache(wl, buf.k, buf.v, U, buf.cap)
    buf.feat_init(n0, 0)
    params, pol = _policy(wl)
    pnp = H.to_np(params)
    bud = torch.tensor(budgets, dtype=torch.int32, device="cuda")
    maxb = max(budgets)
    sts = [H.oracle_student(wl, u) for u in range(U)]
    q, kn, vn = _step_tensors(wl)
    for t in range(steps):
        sg.queries(wl, t, q)
        sg.new_rows(wl, t, kn, vn, U)
        out = buf.decode_step(q, kn, vn)
        torch.cuda.synchronize()
        lens = H.to_np(buf.unit_len).astype(int)
        outn = H.to_np(out)
        pre = [_download(buf, u, lens[u]) for u in range(U)]
        Lb = buf.kv.len
        scores = torch.empty((U, Lb), dtype=torch.float32, device="cuda")
        kept = torch.empty((U, min(maxb, Lb)), dtype=torch.int32, device="cuda")
        logp = torch.empty(U, dtype=torch.float64, device="cuda") if gumbel else None
        g = B.make_gumbel(tau, gumbel, t) if gumbel else None
        buf.score_evict_units(pol, bud, maxb, g, scores, kept, logp)
        torch.cuda.synchronize()
        sc, kp = H.to_np(scores), H.to_np(kept)
        post_lens = H.to_np(buf.unit_len).astype(int)
        lp = logp.cpu().numpy() if gumbel else None
        diverged = False
        for u in range(U):
            att = ounit.decode_step(sts[u], *H.step_inputs_np(wl, t, u))
            assert lens[u] == sts[u].L, (t, u, lens[u], sts[u].L)
            # until a near-tie parts them, device and oracle store the rows in the same slots
            _check_decode(wl, outn[u], pre[u], sts[u], att, (t, u))
            s_or = ounit.scores(sts[u], pnp, wl.hidden)
            ok, worst = H.vec_ok(sc[u, :lens[u]], s_or)
            assert ok, (t, u, worst)
            Bu = budgets[u]
            nk = min(Bu, lens[u])
            assert post_lens[u] == nk, (t, u)
            assert np.all(kp[u, nk:] == -1) and np.all(kp[u, :nk] >= 0), (t, u)
            post = _download(buf, u, nk)
            # the oracle's compaction for this unit's own budget (deterministic: its
            # selection on the GPU's own scores; sampled: the kept set checked below)
            if gumbel:
                layout = H.slot_map_of(kp[u, :nk], lens[u])
            else:
                layout = H.oracle_slot_map(sc[u, :lens[u]], pre[u]["pos"], nk)
            assert np.array_equal(kp[u, :nk], layout), (t, u)
            for name in ("k", "v", "pos", "alpha", "num", "den", "vnorm"):
                assert np.array_equal(post[name], pre[u][name][layout]), (t, u, name)
            if gumbel:
                ok, kept_o, amb, flips = _sampled_check(s_or, sts[u].pos, post["pos"], Bu, tau,
                                                        gumbel, u, t)
                assert ok, (t, u, amb, flips)
                if flips == 0:
                    ref = osmp.log_prob(s_or, kept_o, Bu, tau)
                    ds = float(np.abs(sc[u, :lens[u]].astype(np.float64) - s_or).max()) / tau
                    tol = _logz_tol(lens[u], Bu) + 2 * nk * ds + 1e-9 * abs(ref)
                    assert abs(lp[u] - ref) <= tol, (t, u, lp[u], ref)
                keep_rows = np.sort(kept_o)
                flips_u = flips
            else:
                ok, amb, flips_u = H.selection_check(s_or, sts[u].pos, post["pos"], Bu)
                assert ok, (t, u, amb, flips_u)
                keep_rows = None
            if keep_rows is not None:
                ounit.evict(sts[u], np.where(np.isin(np.arange(sts[u].L), keep_rows), 1.0, 0.0), Bu)
            else:
                ounit.evict(sts[u], s_or, Bu)
            diverged |= flips_u > 0
        assert buf.kv.len == min(maxb, Lb)
        if diverged:
            print("trajectories parted at a near-tie at step", t)
            return t
    return steps


def test_per_unit_budgets_and_a_full_cache_head():
    # unit 1 never evicts (the hybrid's full-cache head); the others keep 200, 150, 320
    assert _ragged_run([200, 10 ** 6, 150, 320], steps=6) >= 1


def test_equal_budgets_reduce_to_the_fixed_budget():
    assert _ragged_run([180, 180, 180], steps=5) >= 1


def test_per_unit_budgets_sampled_with_log_prob():
    assert _ragged_run([120, 700, 90], steps=4, gumbel=55, tau=0.8) >= 1


def test_two_layer_policy_on_ragged_caches():
    # the matrix-core scoring pass with per-unit lengths and budgets (widths
    # padded to 64, then to 128)
    assert _ragged_run([200, 10 ** 6, 150], steps=4, hidden=(64, 64)) >= 1
    assert _ragged_run([260, 90], steps=3, hidden=(96, 40)) >= 1


def test_two_layer_policy_sampled_on_ragged_caches():
    assert _ragged_run([120, 700, 90], steps=3, gumbel=77, tau=0.7, hidden=(64, 64)) >= 1


@pytest.mark.parametrize("hidden", [None, (64, 64)])
def test_units_that_keep_every_row_are_not_scored_without_scores_out(hidden):
    """Without scores_out, a unit whose budget covers its rows is not scored (its
    selection reads no key).  Two buffers run the same ragged steps, one asking
    for scores and one not: every state buffer, length and slot map must agree
    bit for bit, while the covering units keep every row in place."""
    budgets = [5000, 300, 5000, 120]                    # units 0 and 2 keep their full cache
    kw = {"hidden": tuple(hidden)} if hidden else {}
    wl = W.WORKLOADS[2].scaled(n_kv_heads=len(budgets), n_q_heads=4 * len(budgets), n0=700,
                               budget=max(budgets), steps=4, **kw)
    U = wl.units
    bufs = []
    for _ in range(2):
        b = DecodeBuffers(wl.batch, wl.n_layers, wl.n_q_heads, wl.n_kv_heads, wl.head_dim,
                          wl.capacity, wl.dtype, wl.ent_window, 0.0, True, ragged=True)
        b.reserve_workspace(wl.capacity)
        sg.init_cache(wl, b.k, b.v, U, b.cap)
        b.feat_init(wl.n0, 0)
        bufs.append(b)
    _, pol = _policy(wl)
    bud = torch.tensor(budgets, dtype=torch.int32, device="cuda")
    q, kn, vn = _step_tensors(wl)
    for t in range(wl.steps):
        sg.queries(wl, t, q)
        sg.new_rows(wl, t, kn, vn, U)
        kept = []
        for i, b in enumerate(bufs):
            b.decode_step(q, kn, vn)
            Lb = b.kv.len
            k = torch.full((U, min(max(budgets), Lb)), -7, dtype=torch.int32, device="cuda")
            sc = torch.empty((U, Lb), dtype=torch.float32, device="cuda") if i == 0 else None
            b.score_evict_units(pol, bud, max(budgets), None, sc, k, None)
            kept.append(k)
        torch.cuda.synchronize()
        assert np.array_equal(H.to_np(kept[0]), H.to_np(kept[1])), t
        lens = [H.to_np(b.unit_len).astype(int) for b in bufs]
        assert np.array_equal(lens[0], lens[1]), t
        for u in range(U):
            a, c = _download(bufs[0], u, lens[0][u]), _download(bufs[1], u, lens[1][u])
            for name in a:
                assert np.array_equal(a[name], c[name]), (t, u, name)
            if budgets[u] >= wl.n0 + t + 1:              # covering: its rows before the selection
                assert np.array_equal(a["pos"], np.arange(wl.n0 + t + 1)), (t, u)
                assert np.array_equal(H.to_np(kept[1][u])[:lens[0][u]], np.arange(lens[0][u]))


def _fused_ragged_run(pattern, steps, n0, batch=32):
    """dc_decode_evict_units (one call per step) on free-running device and oracle
    trajectories, on enough units for the single-launch route (unit u keeps the
    budget of KV head u mod len(pattern)); the oracle follows unit 0, the last
    unit and six seeded random units: attention output, scores, the slot map
    (exactly, under the oracle's selection and compaction of the GPU's scores),
    lengths and the post-step state, until a selection lands in the near-tie band."""
    wl = W.WORKLOADS[2].scaled(batch=batch, n_kv_heads=len(pattern), n_q_heads=4 * len(pattern),
                               n0=n0, budget=max(pattern), steps=steps)
    U = wl.units
    assert U >= 128
    budgets = [pattern[u % len(pattern)] for u in range(U)]
    buf = DecodeBuffers(wl.batch, wl.n_layers, wl.n_q_heads, wl.n_kv_heads, wl.head_dim,
                        wl.capacity, wl.dtype, wl.ent_window, 0.0, True, ragged=True)
    buf.reserve_workspace(wl.capacity)
    sg.init_cache(wl, buf.k, buf.v, U, buf.cap)
    buf.feat_init(n0, 0)
    params, pol = _policy(wl)
    pnp = H.to_np(params)
    bud = torch.tensor(budgets, dtype=torch.int32, device="cuda")
    maxb = max(budgets)
    rng = np.random.default_rng(wl.seed)
    sample = sorted({0, U - 1, *rng.choice(np.arange(1, U - 1), 6, replace=False).tolist()})
    sts = {u: H.oracle_student(wl, u) for u in sample}
    q, kn, vn = _step_tensors(wl)
    for t in range(steps):
        sg.queries(wl, t, q)
        sg.new_rows(wl, t, kn, vn, U)
        Lb = buf.kv.len + 1
        scores = torch.full((U, Lb), float("nan"), dtype=torch.float32, device="cuda")
        kept = torch.full((U, min(maxb, Lb)), -7, dtype=torch.int32, device="cuda")
        if t % 16 == 0:
            print(f"one-call ragged step {t}: bound {Lb} rows", flush=True)
        out = buf.decode_evict_units(pol, bud, maxb, q, kn, vn, scores_out=scores, kept_out=kept)
        torch.cuda.synchronize()
        outn, sc, kp = H.to_np(out), H.to_np(scores), H.to_np(kept)
        lens = H.to_np(buf.unit_len).astype(int)
        diverged = False
        for u in sample:
            st = sts[u]
            att = ounit.decode_step(st, *H.step_inputs_np(wl, t, u))
            Lu = st.L
            assert H.rel_err_rows(outn[u], att.o) <= H.OUT_TOL, (t, u)
            s_or = ounit.scores(st, pnp, wl.hidden)
            ok, worst = H.vec_ok(sc[u, :Lu], s_or)       # same slots as the oracle so far
            assert ok, (t, u, "scores", worst)
            Bu = budgets[u]
            nk = min(Bu, Lu)
            assert lens[u] == nk, (t, u, lens[u], nk)
            # exact: the oracle's selection and compaction on the GPU's own scores
            assert np.array_equal(kp[u, :nk], H.oracle_slot_map(sc[u, :Lu], st.pos, Bu)), (t, u)
            assert np.all(kp[u, nk:] == -1), (t, u)
            post = _download(buf, u, nk)
            ok, amb, flips = H.selection_check(s_or, st.pos, post["pos"], Bu)
            assert ok, (t, u, amb, flips)
            ounit.evict(st, s_or, Bu)
            if flips == 0:
                assert np.array_equal(post["pos"], st.pos), (t, u)
                Z, N = st.hist.sums()
                for name, ref in (("alpha", st.alpha), ("den", Z), ("num", N)):
                    ok, worst = H.vec_ok(post[name], ref)
                    assert ok, (t, u, name, worst)
            diverged |= flips > 0
        assert buf.kv.len == min(maxb, Lb)
        assert np.all(lens == np.minimum(budgets, n0 + t + 1)), t
        if diverged:
            print("trajectories parted at a near-tie at step", t)
            return t
    return steps


def test_one_call_ragged_step_all_units_on_chip():
    # the full-cache units grow from 701 rows and stay within the single-launch bound
    assert _fused_ragged_run([200, 10 ** 6, 150, 320], steps=70, n0=700) >= 1


def test_one_call_ragged_step_with_long_full_cache_units():
    # 4601 rows exceed the single-launch bound (4479 rows at head_dim 128, G = 4): step 0
    # compresses every unit through the chunked decode and the stand-alone selection;
    # then the budgeted units run in one launch and the full-cache units on the chunked path
    assert _fused_ragged_run([200, 10 ** 6, 150, 10 ** 6], steps=70, n0=4600) >= 1


def test_one_call_ragged_step_equals_the_uniform_single_launch_step():
    """Equal lengths and budgets: the ragged single-launch variant does exactly
    what the uniform one does, bit for bit (outputs, scores, slot maps, every
    state buffer), through the window's retire."""
    wl = W.WORKLOADS[2].scaled(batch=64, n_kv_heads=2, n_q_heads=8, n0=700, budget=256, steps=70)
    U, budget = wl.units, wl.budget
    assert U >= 128
    uni = DecodeBuffers(wl.batch, wl.n_layers, wl.n_q_heads, wl.n_kv_heads, wl.head_dim,
                        wl.capacity, wl.dtype, wl.ent_window, 0.0, True)
    rag = DecodeBuffers(wl.batch, wl.n_layers, wl.n_q_heads, wl.n_kv_heads, wl.head_dim,
                        wl.capacity, wl.dtype, wl.ent_window, 0.0, True, ragged=True)
    for b in (uni, rag):
        b.reserve_workspace(wl.capacity)
        sg.init_cache(wl, b.k, b.v, U, b.cap)
        b.feat_init(wl.n0, 0)
    _, pol = _policy(wl)
    bud = torch.full((U,), budget, dtype=torch.int32, device="cuda")
    q, kn, vn = _step_tensors(wl)
    for t in range(wl.steps):
        sg.queries(wl, t, q)
        sg.new_rows(wl, t, kn, vn, U)
        L = uni.kv.len + 1
        sc = [torch.empty((U, L), dtype=torch.float32, device="cuda") for _ in range(2)]
        kp = [torch.empty((U, min(L, budget)), dtype=torch.int32, device="cuda") for _ in range(2)]
        o0 = uni.decode_evict(pol, budget, q, kn, vn, scores_out=sc[0], kept_out=kp[0])
        o1 = rag.decode_evict_units(pol, bud, budget, q, kn, vn, scores_out=sc[1], kept_out=kp[1])
        torch.cuda.synchronize()
        assert torch.equal(o0, o1), t
        assert torch.equal(sc[0], sc[1]) and torch.equal(kp[0], kp[1]), t
        n = uni.kv.len
        assert rag.kv.len == n and torch.all(rag.unit_len == n), t
        for name in ("k", "v", "alpha", "num", "den", "pos", "vnorm", "qring", "qstat"):
            a0, a1 = getattr(uni, name), getattr(rag, name)
            if name in ("qring", "qstat"):
                assert torch.equal(a0, a1), (t, name)
            else:
                assert torch.equal(a0[:, :n], a1[:, :n]), (t, name)
