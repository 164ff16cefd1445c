"""Benchmark: DistillCache budgeted decode step on one MI355X.

Workload (default): the Mistral-7B-shaped 32-layer KV stack — batch 16, 32
layers, 32 query / 8 KV heads, head_dim 128, bf16, synthetic context 16384,
budget 4096 (25 %), per-KV-head top-k.  One *step* is the whole hot path over
every (batch, layer, KV head) unit: append the new K/V row, GQA decode
attention, feature accumulation (alpha, windowed entropy, ||v||, position),
policy-MLP scoring of every cached token, top-4096 keep and in-place
compaction.  The workload's 128 steps run first, each timed on its own: the
compression step 16385 -> 4096, steps 1..63 while the entropy window fills,
steps 64..127 with the window full; their average and the two kinds of steady
step are reported separately.  The headline value times further steady steps
(4097 -> 4096 per unit), all with the window full, so each also retires the
queries of step t - 64.

Prints one JSON line.  Inputs are resident in HBM before timing starts.
"""
from __future__ import annotations

import argparse
import json
import os
import re

import numpy as np
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode steps/s + KV GB/s (% of 8 TB/s HBM) for attention+evict at 16k ctx, 25% budget"
HBM_PEAK_GBPS = 8000.0


def step_alg_bytes(U, L, G, D, elt, retire, moved):
    """Algorithmic HBM bytes of one fused decode step over U units of L rows
    (after the append): every cached K/V row read once (L - 1 rows; the new row
    arrives in k_new/v_new, read once and written to the cache once); per row the
    feature state read and written (alpha f32 and num/den f64: 40 B) plus pos and
    ||v|| read (8 B); the queries read and outputs written; the retiring ring
    queries read and this step's queries written to the ring (1 KB each), the
    per-query statistics; compaction moves read and write the K/V row and its
    28 bytes of state."""
    row = 2 * D * elt
    qbytes = G * D * elt
    per_unit = (L - 1) * row + 2 * row + L * 48
    per_unit += 2 * qbytes + (qbytes if retire else 0) + qbytes + 2 * G * 3 * 4
    return U * per_unit + moved * 2 * (row + 28)


def evict_alg_bytes(U, L, moved, D, elt):
    """score/select/compact: features read (alpha, vnorm f32, num/den f64, pos i32:
    28 B/row), moved rows read+written (K/V + 28 B of state each)."""
    return U * L * 28 + moved * 2 * (2 * D * elt + 28)


def kv_bytes(U, L, D, elt, moved, append=1):
    """KV bytes of a step: K/V read by attention, the appended row written, and the
    K/V part of the compaction moves (read + write)."""
    row = 2 * D * elt
    return U * ((L - append) * row + append * 2 * row) + moved * 2 * row


STEP_KERNEL_SOURCES = ("dc_step.hip", "dc_select.hpp", "dc_device.hpp", "dc_kernels.hpp")
TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "step_unit_kernel_c3_hbm_counters.md")


def step_kernel_source_hash():
    import hashlib
    h = hashlib.sha256()
    for f in STEP_KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2608_08878_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic():
    """HBM bytes per launch of the fused step kernel from the committed
    FETCH_SIZE/WRITE_SIZE counter runs (copy-kernel calibrated), or None when the
    kernel sources changed after the counters were taken."""
    try:
        text = open(TRAFFIC_PROFILE).read()
    except OSError:
        return None
    tb = re.search(r"traffic_bytes_per_launch: (\d+)", text)
    hs = re.search(r"kernel source sha256\[:16\]: ([0-9a-f]+)", text)
    if not tb or not hs or hs.group(1) != step_kernel_source_hash():
        return None
    return int(tb.group(1))


def _oracle_units_worker(task):
    """Worker process of the CPU baseline: bring each unit to a full entropy
    window (steps 0..w-1, untimed) and time `steps` further steps of the oracle
    (append, attention, features, score, top-B, compaction), one BLAS thread."""
    cid, units, steps = task
    from threadpoolctl import threadpool_limits

    from oracle import attention as oatt
    from oracle import unit as ounit
    from synth import workloads as W

    wl = W.WORKLOADS[cid]
    params = W.policy_params(wl)
    scale = oatt.default_scale(wl.head_dim)
    fill = max(wl.ent_window, 1)
    timed = 0.0
    with threadpool_limits(1):
        for u in units:
            pos = np.arange(wl.n0)
            st = ounit.new_student(W.key_rows(wl, u, pos), W.value_rows(wl, u, pos), pos,
                                   G=wl.group, scale=scale, window=wl.ent_window, next_pos=wl.n0)
            inputs = []
            for t in range(fill + steps):
                p = [wl.n0 + t]
                inputs.append((W.queries(wl, t, u), W.key_rows(wl, u, p)[0],
                               W.value_rows(wl, u, p)[0]))
            for t in range(fill):
                ounit.decode_step(st, *inputs[t])
                ounit.score_evict(st, params, wl.hidden, wl.budget)
            t0 = time.perf_counter()
            for t in range(fill, fill + steps):
                ounit.decode_step(st, *inputs[t])
                ounit.score_evict(st, params, wl.hidden, wl.budget)
            timed += time.perf_counter() - t0
    return timed, len(units) * steps


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def run_oracle_baseline(wl, n_units, steps, workers):
    """Time the CPU oracle on a bounded sample of units in `workers` processes
    (one thread each); returns (unit-steps per second of the whole pool, total
    timed CPU seconds).  Units are independent, so the pool's rate scales to
    the workload by its unit count."""
    import multiprocessing

    units = [(k * 2654435761) % wl.units for k in range(n_units)]
    chunks = [units[w::workers] for w in range(workers) if units[w::workers]]
    ctx = multiprocessing.get_context("spawn")      # fresh interpreters, no GPU state
    with ctx.Pool(len(chunks)) as pool:
        res = pool.map(_oracle_units_worker, [(wl.cid, c, steps) for c in chunks])
    wall = max(r[0] for r in res)                   # the pool finishes with its slowest worker
    return sum(r[1] for r in res) / wall, sum(r[0] for r in res)


def _events(n):
    import torch
    return [torch.cuda.Event(enable_timing=True) for _ in range(n)]


def _load_compression_kernels(wl, cap, pol, dev, sample=None):
    """A kernel's first launch also loads its code (milliseconds).  Run the
    compression step once on a one-unit cache of the same length, so that the
    reported step 0 is the GPU's work on the workload."""
    import torch
    from paper_2608_08878_amd.buffers import DecodeBuffers
    from paper_2608_08878_amd import binding as B
    G, D = wl.group, wl.head_dim
    td = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    one = DecodeBuffers(1, 1, G, 1, D, cap, wl.dtype, wl.ent_window)
    one.reserve_workspace(cap)
    one.feat_init(wl.n0, 0)
    q = torch.zeros((1, G, D), dtype=td, device=dev)
    kn = torch.zeros((1, D), dtype=td, device=dev)
    if sample is None:
        one.decode_evict(pol, wl.budget, q, kn, kn.clone())
    else:
        L = wl.n0 + 1
        sc = torch.empty((1, L), dtype=torch.float32, device=dev)
        kp = torch.empty((1, wl.budget), dtype=torch.int32, device=dev)
        lp = torch.empty(1, dtype=torch.float64, device=dev)
        one.decode_sample_evict(pol, wl.budget, B.make_gumbel(1.0, sample, 0), q, kn, kn.clone(),
                                None, sc, kp, lp)
    torch.cuda.synchronize()
    del one


def bench_single_step(args, wl, dev, log):
    """Workload 1: one step (attention, features, score, top-B, compaction) over a
    512-row fp32 cache, no append.  Each repetition starts from the same state
    (restored by device copies, untimed)."""
    import torch
    from paper_2608_08878_amd.buffers import DecodeBuffers, make_policy
    from synth import gpu as sg
    from synth import workloads as W

    U, G, D = wl.units, wl.group, wl.head_dim
    buf = DecodeBuffers(wl.batch, wl.n_layers, wl.n_q_heads, wl.n_kv_heads, D, wl.n0, wl.dtype,
                        wl.ent_window)
    sg.init_cache(wl, buf.k, buf.v, U, wl.n0)
    k0, v0 = buf.k.clone(), buf.v.clone()
    params = torch.empty(wl.n_params, dtype=torch.float32, device=dev)
    sg.fill_normal(params, wl, W.S_POLICY, 0, 0.1)
    pol = make_policy(params, wl.hidden)
    q = torch.empty((U, G, D), dtype=torch.float32, device=dev)
    sg.queries(wl, 0, q)
    out = torch.empty_like(q)
    times = []
    for r in range(args.warmup + args.steps):
        buf.k.copy_(k0)
        buf.v.copy_(v0)
        buf.feat_init(wl.n0, 0)
        torch.cuda.synchronize()
        a, b = _events(2)
        a.record()
        buf.decode_evict(pol, wl.budget, q, None, None, out)
        b.record()
        torch.cuda.synchronize()
        if r >= args.warmup:
            times.append(a.elapsed_time(b))
    ms = float(sorted(times)[len(times) // 2])
    kvb = U * wl.n0 * 2 * D * 4
    return {"value": round(1e3 / ms, 3), "unit": "decode steps/s", "ms_per_step": round(ms, 4),
            "kv_gbps": round(kvb / (ms * 1e-3) / 1e9, 2),
            "note": "median of single-step repetitions from a restored state; launch-bound (8 KB of K/V per unit)"}


def bench_periodic_evict(args, wl, dev, log):
    """Workload 4: 32k context, budget 3277, 4->64->64->1 policy, eviction every 64
    steps.  After the compression step the live rows move into buffers of
    capacity B + 64; one cycle is 63 decode steps with feature updates plus one
    step with eviction (3341 -> 3277 rows)."""
    import torch
    from paper_2608_08878_amd.buffers import DecodeBuffers, make_policy
    from synth import gpu as sg
    from synth import workloads as W

    U, G, D, E = wl.units, wl.group, wl.head_dim, wl.evict_every
    cap = wl.n0 + 1
    buf = DecodeBuffers(wl.batch, wl.n_layers, wl.n_q_heads, wl.n_kv_heads, D, cap, wl.dtype,
                        wl.ent_window)
    buf.reserve_workspace(cap)
    sg.init_cache(wl, buf.k, buf.v, U, cap)
    buf.feat_init(wl.n0, 0)
    params = torch.empty(wl.n_params, dtype=torch.float32, device=dev)
    sg.fill_normal(params, wl, W.S_POLICY, 0, 0.1)
    pol = make_policy(params, wl.hidden)
    cycles = max(1, args.steps // E)
    nsteps = 1 + E * (1 + cycles)                  # step 0, one warm-up cycle, timed cycles
    q = torch.empty((nsteps, U, G, D), dtype=torch.bfloat16, device=dev)
    kn = torch.empty((nsteps, U, D), dtype=torch.bfloat16, device=dev)
    vn = torch.empty_like(kn)
    for t in range(nsteps):
        sg.queries(wl, t, q[t])
        sg.new_rows(wl, t, kn[t], vn[t], U)
    out = torch.empty((U, G, D), dtype=torch.bfloat16, device=dev)
    _load_compression_kernels(wl, cap, pol, dev)
    torch.cuda.synchronize()
    a, b = _events(2)
    a.record()
    buf.decode_evict(pol, wl.budget, q[0], kn[0], vn[0], out)
    b.record()
    torch.cuda.synchronize()
    first_ms = a.elapsed_time(b)
    log(f"step 0 (L={cap} -> {wl.budget}): {first_ms:.3f} ms")
    if not args.no_shrink:
        buf.shrink(wl.budget + E)
    dec_ms, ev_ms, cyc_ms = [], [], []
    t = 1
    for c in range(1 + cycles):
        ev = _events(2 * E)
        for j in range(E):
            ev[2 * j].record()
            if (t % E) == 0:
                buf.decode_evict(pol, wl.budget, q[t], kn[t], vn[t], out)
            else:
                buf.decode_step(q[t], kn[t], vn[t], out)
            ev[2 * j + 1].record()
            t += 1
        torch.cuda.synchronize()
        if c >= 1:
            per = [ev[2 * j].elapsed_time(ev[2 * j + 1]) for j in range(E)]
            cyc_ms.append(ev[0].elapsed_time(ev[-1]))
            ev_ms += [p for j, p in enumerate(per) if ((t - E + j) % E) == 0]
            dec_ms += [p for j, p in enumerate(per) if ((t - E + j) % E) != 0]
    cycle = float(np.mean(cyc_ms))
    ms = cycle / E
    Lmean = wl.budget + (E + 1) / 2.0
    kvb = U * Lmean * 2 * D * 2
    return {"value": round(1e3 / ms, 3), "unit": "decode steps/s", "ms_per_step": round(ms, 4),
            "kv_gbps": round(kvb / (ms * 1e-3) / 1e9, 1),
            "kv_frac_of_8TBps": round(kvb / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
            "decode_step_ms": round(float(np.mean(dec_ms)), 4),
            "evict_step_ms": round(float(np.mean(ev_ms)), 4),
            "first_step_ms": round(first_ms, 3), "steady_capacity": buf.cap,
            "note": f"mean over {cycles} cycles of {E} steps (63 decode steps + 1 eviction step)"}


def bench_teacher_student_kl(args, wl, dev, log):
    """Workload 5: per step the teacher's plain attention over the never-pruned
    cache (8193.. rows), the student's decode + evict (2049 -> 2048 rows) and the
    KL reward of 8 rows over the 32768 x 4096 lm head."""
    import torch
    from paper_2608_08878_amd import binding as B
    from paper_2608_08878_amd.buffers import DecodeBuffers, make_policy, stream_handle
    from synth import gpu as sg
    from synth import workloads as W

    U, G, D = wl.units, wl.group, wl.head_dim
    nsteps = 1 + args.warmup + args.steps
    stu = DecodeBuffers(wl.batch, wl.n_layers, wl.n_q_heads, wl.n_kv_heads, D, wl.n0 + 1, wl.dtype,
                        wl.ent_window)
    tea = DecodeBuffers(wl.batch, wl.n_layers, wl.n_q_heads, wl.n_kv_heads, D, wl.n0 + nsteps,
                        wl.dtype, wl.ent_window, features=False)
    stu.reserve_workspace(wl.n0 + 1)
    sg.init_cache(wl, stu.k, stu.v, U, stu.cap)
    stu.feat_init(wl.n0, 0)
    sg.init_cache(wl, tea.k, tea.v, U, tea.cap, n0=wl.n0)
    tea.kv.len = wl.n0
    params = torch.empty(wl.n_params, dtype=torch.float32, device=dev)
    sg.fill_normal(params, wl, W.S_POLICY, 0, 0.1)
    pol = make_policy(params, wl.hidden)
    rows, hid, voc = wl.batch, wl.kl_hidden, wl.kl_vocab
    w = torch.empty((voc, hid), dtype=torch.bfloat16, device=dev)
    sg.fill_normal(w, wl, W.S_WLM, 0, 0.02)
    sh = stream_handle()
    # the lm head is laid out once, as a model's weights are at load time, in
    # the tile layout the per-step reward streams fastest (same results)
    kl_fn = B.dc_kl_reward
    pack_ms = None
    if not args.kl_row_major:
        wp = torch.empty_like(w)
        ev = _events(2)
        ev[0].record()
        B.dc_kl_pack_lm_head(hid, voc, w, wp, sh)
        ev[1].record()
        torch.cuda.synchronize()
        pack_ms = ev[0].elapsed_time(ev[1])
        w, kl_fn = wp, B.dc_kl_reward_packed
    hf = torch.empty((nsteps, rows, hid), dtype=torch.bfloat16, device=dev)
    hc = torch.empty_like(hf)
    for t in range(nsteps):
        sg.fill_normal(hf[t], wl, W.S_HFULL, t, 1.0)
        sg.fill_noisy(hc[t], hf[t], wl, t, 0.01)
    kl = torch.empty(rows, dtype=torch.float32, device=dev)
    ws = torch.empty(B.dc_workspace_bytes(stu.dims, 0, rows, voc), dtype=torch.uint8, device=dev)
    q = torch.empty((U, G, D), dtype=torch.bfloat16, device=dev)
    kn = torch.empty((U, D), dtype=torch.bfloat16, device=dev)
    vn = torch.empty_like(kn)
    o_t, o_s = torch.empty_like(q), torch.empty_like(q)
    parts = {"teacher": [], "student": [], "kl": [], "step": []}
    first_ms = None
    train = args.train_select
    if train:
        # training-mode student: Gumbel-perturbed top-B and log pi of the kept set
        sc_flat = torch.empty(U * (wl.n0 + 1), dtype=torch.float32, device=dev)
        kept = torch.empty((U, wl.budget), dtype=torch.int32, device=dev)
        logp = torch.empty(U, dtype=torch.float64, device=dev)
    # load step 0's kernels (student compression, teacher, KL) before timing it
    _load_compression_kernels(wl, wl.n0 + 1, pol, dev, sample=wl.seed if train else None)
    nt = 128                   # enough units for the teacher's one-workgroup-per-unit path
    one_t = DecodeBuffers(nt, 1, G, 1, D, wl.n0 + 2, wl.dtype, wl.ent_window, features=False)
    one_t.kv.len = wl.n0
    one_t.decode_step(q[:nt], kn[:nt], vn[:nt], features=False)
    kl_fn(rows, hid, voc, hf[0], hc[0], w, kl, ws, ws.numel(), sh)
    torch.cuda.synchronize()
    del one_t
    for t in range(nsteps):
        sg.queries(wl, t, q)
        sg.new_rows(wl, t, kn, vn, U)
        ev = _events(4)
        ev[0].record()
        tea.decode_step(q, kn, vn, o_t, features=False)
        ev[1].record()
        if train:
            L = stu.kv.len + 1
            stu.decode_sample_evict(pol, wl.budget, B.make_gumbel(1.0, wl.seed, t), q, kn, vn,
                                    o_s, sc_flat[:U * L].view(U, L), kept, logp)
        else:
            stu.decode_evict(pol, wl.budget, q, kn, vn, o_s)
        ev[2].record()
        kl_fn(rows, hid, voc, hf[t], hc[t], w, kl, ws, ws.numel(), sh)
        ev[3].record()
        torch.cuda.synchronize()
        if t == 0:
            first_ms = ev[0].elapsed_time(ev[3])
            if not args.no_shrink:
                stu.shrink(wl.budget + 1)
        elif t > args.warmup:
            parts["teacher"].append(ev[0].elapsed_time(ev[1]))
            parts["student"].append(ev[1].elapsed_time(ev[2]))
            parts["kl"].append(ev[2].elapsed_time(ev[3]))
            parts["step"].append(ev[0].elapsed_time(ev[3]))
    m = {k: float(np.mean(v)) for k, v in parts.items()}
    extra = {"kl_lm_head_layout": "row-major" if args.kl_row_major else "packed 64x64 tiles",
             "kl_pack_ms": None if pack_ms is None else round(pack_ms, 4)}
    # the same rewards deferred to the end of the rollout: one call over all
    # steps x batch rows reads the lm head once
    Td = nsteps
    wsd = torch.empty(B.dc_workspace_bytes(stu.dims, 0, Td * rows, voc), dtype=torch.uint8, device=dev)
    kld = torch.empty(Td * rows, dtype=torch.float32, device=dev)
    hfv, hcv = hf.view(Td * rows, hid), hc.view(Td * rows, hid)
    kl_fn(Td * rows, hid, voc, hfv, hcv, w, kld, wsd, wsd.numel(), sh)
    torch.cuda.synchronize()
    ev = _events(2)
    ev[0].record()
    for _ in range(3):
        kl_fn(Td * rows, hid, voc, hfv, hcv, w, kld, wsd, wsd.numel(), sh)
    ev[1].record()
    torch.cuda.synchronize()
    kd_ms = ev[0].elapsed_time(ev[1]) / 3
    flops = 2.0 * 2 * Td * rows * hid * voc
    extra.update({"kl_deferred_rows": Td * rows, "kl_deferred_ms": round(kd_ms, 4),
                  "kl_deferred_ms_per_step": round(kd_ms / Td, 4),
                  "kl_deferred_tflops": round(flops / (kd_ms * 1e-3) / 1e12, 1)})
    log(f"deferred KL over {Td} steps x {rows} rows: {kd_ms:.3f} ms "
        f"({kd_ms / Td:.4f} ms per step vs {m['kl']:.4f} per-step calls)")
    if train:
        extra.update({"student_select": "gumbel top-B + log pi (training mode, one fused "
                                        "launch + the log-partition)"})
        extra.update(time_log_partition(wl, U, dev, log))
    Lt = wl.n0 + 1 + args.warmup + args.steps / 2.0
    kvb = U * (Lt + wl.budget + 1) * 2 * D * 2 + voc * hid * 2
    return {"value": round(1e3 / m["step"], 3), "unit": "decode steps/s",
            "ms_per_step": round(m["step"], 4),
            "kv_gbps": round(kvb / (m["step"] * 1e-3) / 1e9, 1),
            "kv_frac_of_8TBps": round(kvb / (m["step"] * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
            "teacher_ms": round(m["teacher"], 4), "student_ms": round(m["student"], 4),
            "kl_ms": round(m["kl"], 4), "first_step_ms": round(first_ms, 3),
            "kl_gbps": round(voc * hid * 2 / (m["kl"] * 1e-3) / 1e9, 1),
            "note": "teacher K/V read + student K/V read + lm head per step; steps timed "
                    "one by one (events per part)", **extra}


def bench_paper_policy(args, wl, dev, log):
    """The paper's full state and policy on a decode workload: five features
    (sigma_i included) and a 5 -> 128 -> 128 -> 1 MLP with LayerNorm after each
    hidden layer (App. D), every step.  The step runs as decode (writing sigma)
    plus the stand-alone scoring pass and selection; the parts are timed apart."""
    import torch
    from paper_2608_08878_amd.buffers import DecodeBuffers, make_policy
    from synth import gpu as sg
    from synth import workloads as W

    U, G, D = wl.units, wl.group, wl.head_dim
    hidden, n_in = (128, 128), 5
    cap = max(wl.n0 + 1, wl.budget + 1)
    buf = DecodeBuffers(wl.batch, wl.n_layers, wl.n_q_heads, wl.n_kv_heads, D, cap, wl.dtype,
                        wl.ent_window, sigma=True)
    buf.reserve_workspace(cap)
    sg.init_cache(wl, buf.k, buf.v, U, cap)
    buf.feat_init(wl.n0, 0)
    # packed blob: per layer W, b, gain, bias; then w_out, b_out.  N(0, 0.1), gains 1 + N(0, 0.1)
    sizes, prev = [], n_in
    for h in hidden:
        sizes += [h * prev, h, h, h]
        prev = h
    n = sum(sizes) + prev + 1
    params = torch.empty(n, dtype=torch.float32, device=dev)
    sg.fill_normal(params, wl, W.S_POLICY, 1, 0.1)
    off = 0
    for li in range(len(hidden)):
        off += sizes[4 * li] + sizes[4 * li + 1]
        params[off:off + sizes[4 * li + 2]] += 1.0
        off += sizes[4 * li + 2] + sizes[4 * li + 3]
    pol = make_policy(params, hidden, n_in=n_in, layer_norm=True)
    nsteps = 1 + args.warmup + args.steps
    td = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    q = torch.empty((U, G, D), dtype=td, device=dev)
    kn = torch.empty((U, D), dtype=td, device=dev)
    vn = torch.empty_like(kn)
    out = torch.empty_like(q)
    parts = {"decode": [], "score_select": [], "step": []}
    first_ms = None
    for t in range(nsteps):
        sg.queries(wl, t, q)
        sg.new_rows(wl, t, kn, vn, U)
        ev = _events(3)
        ev[0].record()
        buf.decode_step(q, kn, vn, out)
        ev[1].record()
        buf.score_evict(pol, wl.budget)
        ev[2].record()
        torch.cuda.synchronize()
        if t == 0:
            first_ms = ev[0].elapsed_time(ev[2])
            if not args.no_shrink:
                buf.shrink(wl.budget + 1)
        elif t > args.warmup:
            parts["decode"].append(ev[0].elapsed_time(ev[1]))
            parts["score_select"].append(ev[1].elapsed_time(ev[2]))
            parts["step"].append(ev[0].elapsed_time(ev[2]))
    m = {k: float(np.mean(v)) for k, v in parts.items()}
    L = wl.budget + 1
    flop_row = 2 * (n_in * hidden[0] + hidden[0] * hidden[1] + hidden[1])
    return {"value": round(1e3 / m["step"], 3), "unit": "decode steps/s",
            "ms_per_step": round(m["step"], 4), "decode_ms": round(m["decode"], 4),
            "score_select_ms": round(m["score_select"], 4), "first_step_ms": round(first_ms, 3),
            "policy": "5->128->128->1 ReLU MLP with LayerNorm, features [alpha, |v|, sigma, H, pos]",
            "mlp_tflops": round(U * L * flop_row / (m["score_select"] * 1e-3) / 1e12, 2),
            # float32-accurate work (the scoring runs on the bf16 matrix cores with
            # a three-part operand split) against the float32 peak
            "mlp_frac_of_f32_peak": round(U * L * flop_row / (m["score_select"] * 1e-3) / 157.3e12, 4),
            "note": "paper-faithful state and policy; decode + separate scoring pass, timed apart"}


def bench_global_alpha(args, wl, dev, log):
    """The paper's alpha on a decode workload: every step leaves each row's
    most recent mass (alpha_recent), the cross-unit average over all heads and
    layers of each sequence replaces it, then the workload's policy scores
    and the selection evicts.  Decode, the average and scoring + selection are
    timed apart."""
    import torch
    from paper_2608_08878_amd.buffers import DecodeBuffers, make_policy
    from synth import gpu as sg
    from synth import workloads as W

    U, G, D = wl.units, wl.group, wl.head_dim
    cap = max(wl.n0 + 1, wl.budget + 1)
    buf = DecodeBuffers(wl.batch, wl.n_layers, wl.n_q_heads, wl.n_kv_heads, D, cap, wl.dtype,
                        wl.ent_window, alpha_recent=True)
    buf.reserve_workspace(cap)
    sg.init_cache(wl, buf.k, buf.v, U, cap)
    buf.feat_init(wl.n0, 0)
    params = torch.empty(wl.n_params, dtype=torch.float32, device=dev)
    sg.fill_normal(params, wl, W.S_POLICY, 0, 0.1)
    pol = make_policy(params, wl.hidden)
    nsteps = 1 + args.warmup + args.steps
    td = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    q = torch.empty((U, G, D), dtype=td, device=dev)
    kn = torch.empty((U, D), dtype=td, device=dev)
    vn = torch.empty_like(kn)
    out = torch.empty_like(q)
    parts = {"decode": [], "global_alpha": [], "score_select": [], "step": []}
    first_ms = None
    for t in range(nsteps):
        sg.queries(wl, t, q)
        sg.new_rows(wl, t, kn, vn, U)
        ev = _events(4)
        ev[0].record()
        buf.decode_step(q, kn, vn, out)
        ev[1].record()
        buf.global_alpha()
        ev[2].record()
        buf.score_evict(pol, wl.budget)
        ev[3].record()
        torch.cuda.synchronize()
        if t == 0:
            first_ms = ev[0].elapsed_time(ev[3])
            if not args.no_shrink:
                buf.shrink(wl.budget + 1)
        elif t > args.warmup:
            parts["decode"].append(ev[0].elapsed_time(ev[1]))
            parts["global_alpha"].append(ev[1].elapsed_time(ev[2]))
            parts["score_select"].append(ev[2].elapsed_time(ev[3]))
            parts["step"].append(ev[0].elapsed_time(ev[3]))
    m = {k: float(np.mean(v)) for k, v in parts.items()}
    L = wl.budget + 1
    # the average reads alpha and pos and writes alpha (12 B per row), plus the sums
    ga_bytes = U * L * 12 + wl.batch * (wl.n0 + nsteps) * 8 * 2
    return {"value": round(1e3 / m["step"], 3), "unit": "decode steps/s",
            "ms_per_step": round(m["step"], 4), "decode_ms": round(m["decode"], 4),
            "global_alpha_ms": round(m["global_alpha"], 4),
            "global_alpha_gbps": round(ga_bytes / (m["global_alpha"] * 1e-3) / 1e9, 1),
            "score_select_ms": round(m["score_select"], 4), "first_step_ms": round(first_ms, 3),
            "note": "alpha = the most recent step's mass averaged over all heads and layers of "
                    "each sequence; decode + average + scoring pass, timed apart"}


def bench_hybrid(args, wl, dev, log):
    """The appendix's head-level hybrid on a decode workload: a fraction of the
    KV heads keeps its full cache, the others keep the workload's budget
    (per-unit budgets on a ragged cache), every step.  The step is one
    dc_decode_evict_units call: the budgeted units (their rows fit on chip) run
    decode, scoring, selection and compaction in one launch, the full-cache
    units take the chunked decode.  The two-call route it replaces (chunked
    decode of every unit, then the per-unit selection) is timed on a second
    cache for comparison."""
    import torch
    from paper_2608_08878_amd.buffers import DecodeBuffers, make_policy
    from synth import gpu as sg
    from synth import workloads as W

    U, G, D = wl.units, wl.group, wl.head_dim
    nsteps = 1 + args.warmup + args.steps
    cap = wl.n0 + nsteps
    params = torch.empty(wl.n_params, dtype=torch.float32, device=dev)
    sg.fill_normal(params, wl, W.S_POLICY, 0, 0.1)
    pol = make_policy(params, wl.hidden)
    # every k-th KV head of a layer keeps its full cache (k = 1 / fraction)
    every = max(1, round(1.0 / args.hybrid))
    full = np.array([(u % wl.n_kv_heads) % every == 0 for u in range(U)])
    big = cap + 1
    budgets = torch.tensor(np.where(full, big, wl.budget), dtype=torch.int32, device=dev)
    td = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    q = torch.empty((U, G, D), dtype=td, device=dev)
    kn = torch.empty((U, D), dtype=td, device=dev)
    vn = torch.empty_like(kn)
    out = torch.empty_like(q)
    res = {}
    for route in ("one_call", "two_call"):
        buf = DecodeBuffers(wl.batch, wl.n_layers, wl.n_q_heads, wl.n_kv_heads, D, cap, wl.dtype,
                            wl.ent_window, ragged=True)
        buf.reserve_workspace(cap)
        sg.init_cache(wl, buf.k, buf.v, U, cap)
        buf.feat_init(wl.n0, 0)
        times = []
        first_ms = None
        for t in range(nsteps):
            sg.queries(wl, t, q)
            sg.new_rows(wl, t, kn, vn, U)
            ev = _events(2)
            ev[0].record()
            if route == "one_call":
                buf.decode_evict_units(pol, budgets, big, q, kn, vn, out)
            else:
                buf.decode_step(q, kn, vn, out)
                buf.score_evict_units(pol, budgets, big)
            ev[1].record()
            torch.cuda.synchronize()
            if t == 0:
                first_ms = ev[0].elapsed_time(ev[1])
            elif t > args.warmup:
                times.append(ev[0].elapsed_time(ev[1]))
        lens = buf.unit_len.cpu().numpy().astype(np.int64)
        res[route] = (float(np.mean(times)), first_ms, lens)
        log(f"hybrid {route}: {res[route][0]:.4f} ms/step, step 0 {first_ms:.3f} ms")
        del buf
        torch.cuda.empty_cache()
    ms, first_ms, lens = res["one_call"]
    assert np.array_equal(lens, res["two_call"][2])
    kvb = int(lens.sum()) * 2 * D * 2
    return {"value": round(1e3 / ms, 3), "unit": "decode steps/s",
            "ms_per_step": round(ms, 4), "two_call_ms_per_step": round(res["two_call"][0], 4),
            "first_step_ms": round(first_ms, 3),
            "full_cache_units": int(full.sum()), "rows_full": int(lens[full].max()),
            "rows_budgeted": int(lens[~full].max()),
            "kv_gbps": round(kvb / (ms * 1e-3) / 1e9, 1),
            "kv_frac_of_8TBps": round(kvb / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
            "note": f"head-level hybrid: 1 of every {every} KV heads keeps its full cache; one "
                    "dc_decode_evict_units call per step (budgeted units in one launch, "
                    "full-cache units on the chunked decode)"}


LOGZ_OPS_PER_UPDATE = 7     # VALU instructions of one recursion update (see the design notes)
VALU_PEAK_TOPS = 256 * 4 * 16 * 2.4e9 / 1e12   # lane-instructions/s without packed math
FP32_VECTOR_PEAK_TFLOPS = 157.3                 # MI355X fp32 vector peak (an FMA counts 2)


def time_log_partition(wl, U, dev, log, reps=5):
    """dc_subset_log_prob alone at the compression step (L = n0 + 1 -> budget) and
    at the one-eviction step (budget + 1 -> budget), inputs resident."""
    import torch
    from paper_2608_08878_amd import binding as B
    from paper_2608_08878_amd.buffers import stream_handle
    out = {}
    for tag, L in (("compress", wl.n0 + 1), ("evict1", wl.budget + 1)):
        Bk = wl.budget
        K = min(Bk, L - Bk)
        g = torch.Generator(device=dev).manual_seed(5)
        s = torch.randn((U, L), generator=g, device=dev) * 3.0
        kept = torch.arange(Bk, dtype=torch.int32, device=dev).repeat(U, 1)
        lz = torch.empty(U, dtype=torch.float64, device=dev)
        lp = torch.empty(U, dtype=torch.float64, device=dev)
        need = B.dc_subset_log_prob_workspace_bytes(U, L, Bk)
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
        sh = stream_handle()
        B.dc_subset_log_prob(U, L, Bk, 1.0, s, kept, lz, lp, ws, need, sh)
        torch.cuda.synchronize()
        ev = _events(2)
        ev[0].record()
        for _ in range(reps):
            B.dc_subset_log_prob(U, L, Bk, 1.0, s, kept, lz, lp, ws, need, sh)
        ev[1].record()
        torch.cuda.synchronize()
        ms = ev[0].elapsed_time(ev[1]) / reps
        upd = U * L * max(K, 1)
        out[f"logz_{tag}_ms"] = round(ms, 4)
        out[f"logz_{tag}_shape"] = f"units={U} L={L} B={Bk} K={K}"
        if K > 8:
            # the method's work: L K updates E_j += x_i E_(j-1) of the subset recursion
            # (App. C, over K = min(B, L - B) entries), one fused multiply-add each
            tflops = 2.0 * upd / (ms * 1e-3) / 1e12
            out[f"logz_{tag}_tflops"] = round(tflops, 2)
            out[f"logz_{tag}_fma_frac"] = round(tflops / FP32_VECTOR_PEAK_TFLOPS, 4)
            # issue efficiency of the implementation (7 VALU instructions per update)
            tops = upd * LOGZ_OPS_PER_UPDATE / (ms * 1e-3) / 1e12
            out[f"logz_{tag}_issue_frac"] = round(tops / VALU_PEAK_TOPS, 4)
        log(f"log-partition {tag}: {ms:.4f} ms ({U} units, L={L}, K={K})")
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=128)
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--config", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-shrink", action="store_true",
                    help="keep the steady steps in the capacity-16385 buffers of step 0")
    ap.add_argument("--policy", choices=["workload", "paper"], default="workload",
                    help="paper: five features (sigma included) and a 5->128->128->1 LayerNorm "
                         "MLP every step (workloads 2 and 3)")
    ap.add_argument("--hybrid", type=float, default=0.0,
                    help="fraction of KV heads that keep their full cache (head-level hybrid; "
                         "per-unit budgets on a ragged cache), workloads 2 and 3")
    ap.add_argument("--global-alpha", action="store_true",
                    help="alpha as the most recent step's mass averaged over all heads and "
                         "layers of each sequence (decode, the average, then scoring), "
                         "workloads 2 and 3")
    ap.add_argument("--train-select", action="store_true",
                    help="workload 5: the student keeps a Gumbel-sampled top-B and computes "
                         "log pi (training mode) instead of the deterministic selection")
    ap.add_argument("--kl-row-major", action="store_true",
                    help="workload 5: read the lm head row-major instead of in the packed "
                         "tile layout")
    ap.add_argument("--cpu-units", type=int, default=128)
    ap.add_argument("--cpu-steps", type=int, default=64)
    ap.add_argument("--calib-copy-mib", type=int, default=1024,
                    help="size of the plain copy kernel run first (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU (--gpus 1): the decode step shards by independent "
              "(batch, layer, KV head) units with no exchange between GPUs, and the "
              "multi-GPU launcher is not implemented.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2608_08878_amd.buffers import DecodeBuffers, make_policy
    from synth import gpu as sg
    from synth import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda")
    wl = W.WORKLOADS[args.config]
    U, G, D, elt = wl.units, wl.group, wl.head_dim, 2 if wl.dtype == "bf16" else 4
    log = lambda *a: print(*a, file=sys.stderr, flush=True)

    # plain copy kernel of known size (HBM counter calibration under rocprofv3 --pmc),
    # then timed: the measured copy bandwidth (bytes read + written per second)
    copy_gbps = None
    if args.calib_copy_mib > 0:
        a = torch.empty(args.calib_copy_mib << 20, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        c0, c1 = _events(2)
        c0.record()
        for _ in range(5):
            b.copy_(a)
        c1.record()
        torch.cuda.synchronize()
        copy_gbps = 5 * 2 * a.numel() / (c0.elapsed_time(c1) * 1e-3) / 1e9
        log(f"device copy: {copy_gbps:.0f} GB/s (read + write)")
        del a, b

    if args.config in (1, 4, 5) or args.policy == "paper" or args.hybrid > 0 or args.global_alpha:
        fn = {1: bench_single_step, 4: bench_periodic_evict, 5: bench_teacher_student_kl}.get(args.config)
        if args.policy == "paper":
            fn = bench_paper_policy
        if args.hybrid > 0:
            fn = bench_hybrid
        if args.global_alpha:
            fn = bench_global_alpha
        res = fn(args, wl, dev, log)
        result = {"metric": f"decode steps/s, workload {args.config}", "n_gpus": 1,
                  "steps": args.steps, "warmup": args.warmup, "higher_is_better": True,
                  "scaling": "weak", "vs_baseline": None, "dtype": wl.dtype,
                  "data": "synthetic (seeded Philox)",
                  "config": {"workload": wl.name, "batch": wl.batch, "layers": wl.n_layers,
                             "q_heads": wl.n_q_heads, "kv_heads": wl.n_kv_heads,
                             "head_dim": D, "context": wl.n0, "budget": wl.budget,
                             "units": U, "policy": "4->%s->1 ReLU MLP" % "->".join(map(str, wl.hidden))}}
        if "policy" in res:
            result["config"]["policy"] = res.pop("policy")
        result.update(res)
        print(json.dumps(result), flush=True)
        return

    cap = max(wl.n0 + 1, wl.budget + 1)
    buf = DecodeBuffers(wl.batch, wl.n_layers, wl.n_q_heads, wl.n_kv_heads, D, cap, wl.dtype,
                        wl.ent_window)
    buf.reserve_workspace(cap)
    t0 = time.time()
    sg.init_cache(wl, buf.k, buf.v, U, cap)
    buf.feat_init(wl.n0, 0)
    params = torch.empty(wl.n_params, dtype=torch.float32, device=dev)
    sg.fill_normal(params, wl, W.S_POLICY, 0, 0.1)
    pol = make_policy(params, wl.hidden)
    # The workload's own steps run first (step 0 compresses, steps 1..w-1 fill the
    # entropy window, from step w on every step also retires step t - w), then
    # `warmup` untimed and `steps` timed steps: every timed step is a window-full
    # steady step, whatever --steps and --warmup are.
    fill = max(wl.ent_window, 1)
    n_wl = max(wl.steps, fill)
    nsteps = n_wl + args.warmup + args.steps + 1         # + one untimed step with the slot map
    td = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    Q = torch.empty((nsteps, U, G, D), dtype=td, device=dev)
    KN = torch.empty((nsteps, U, D), dtype=td, device=dev)
    VN = torch.empty_like(KN)
    for t in range(nsteps):
        sg.queries(wl, t, Q[t])
        sg.new_rows(wl, t, KN[t], VN[t], U)
    out = torch.empty((U, G, D), dtype=td, device=dev)
    torch.cuda.synchronize()
    log(f"setup {time.time() - t0:.1f}s: {U} units, cache {buf.k.numel() * elt * 2 / 1e9:.1f} GB")

    # step 0: compression n0+1 -> budget
    _load_compression_kernels(wl, cap, pol, dev)
    e0, e1 = _events(2)
    e0.record()
    buf.decode_evict(pol, wl.budget, Q[0], KN[0], VN[0], out)
    e1.record()
    torch.cuda.synchronize()
    first_ms = e0.elapsed_time(e1)
    log(f"step 0 (L={wl.n0 + 1} -> {wl.budget}): {first_ms:.3f} ms")
    if not args.no_shrink:
        # after compression only budget + 1 rows per unit are live: move them into
        # budget-sized buffers (one-time, between steps 0 and 1)
        buf.shrink(wl.budget + 1)
        log(f"caches moved to capacity {buf.cap}")

    # the rest of the workload's steps, each between its own events
    ev = [_events(2) for _ in range(n_wl)]
    for t in range(1, n_wl):
        ev[t][0].record()
        buf.decode_evict(pol, wl.budget, Q[t], KN[t], VN[t], out)
        ev[t][1].record()
    torch.cuda.synchronize()
    wl_ms = [first_ms] + [ev[t][0].elapsed_time(ev[t][1]) for t in range(1, n_wl)]
    pre_ms = float(np.mean(wl_ms[1:fill])) if fill > 1 else float("nan")
    full_ms = float(np.mean(wl_ms[fill:])) if n_wl > fill else float("nan")
    wl_avg_ms = float(np.sum(wl_ms[:wl.steps])) / wl.steps
    log(f"workload steps 1..{fill - 1} (window filling): {pre_ms:.4f} ms/step; steps "
        f"{fill}..{n_wl - 1} (window full): {full_ms:.4f} ms/step; {wl.steps}-step average "
        f"incl. step 0: {wl_avg_ms:.4f} ms")

    for t in range(n_wl, n_wl + args.warmup):
        buf.decode_evict(pol, wl.budget, Q[t], KN[t], VN[t], out)
    torch.cuda.synchronize()
    assert buf.feat.step >= fill, "timed steps must all retire a window step"

    L_steady = buf.kv.len + 1
    ev = [_events(2) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for i in range(args.steps):
        t = n_wl + args.warmup + i
        a, b = ev[i]
        a.record()
        buf.decode_evict(pol, wl.budget, Q[t], KN[t], VN[t], out)
        b.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    step_ms = float(np.mean([a.elapsed_time(b) for a, b in ev]))
    ms_per_step = wall * 1e3 / args.steps
    log(f"steady (window full): {ms_per_step:.3f} ms/step wall; fused step kernel "
        f"{step_ms:.3f} ms (events)")

    # moved rows per steady step (one untimed extra step with the slot map)
    kept = torch.empty((U, wl.budget), dtype=torch.int32, device=dev)
    t = nsteps - 1
    buf.decode_evict(pol, wl.budget, Q[t], KN[t], VN[t], out, kept_out=kept)
    torch.cuda.synchronize()
    moved = int((kept != torch.arange(wl.budget, device=dev, dtype=torch.int32)[None, :]).sum())

    step_bytes = step_alg_bytes(U, L_steady, G, D, elt, True, moved)
    kvb = kv_bytes(U, L_steady, D, elt, moved)
    steps_per_s = 1e3 / ms_per_step
    step_gbps = step_bytes / (step_ms * 1e-3) / 1e9
    kv_gbps = kvb / (ms_per_step * 1e-3) / 1e9
    result = {
        "metric": METRIC,
        "value": round(steps_per_s, 3),
        "unit": "decode steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic (seeded Philox; Mistral-7B-shaped K/V with log-normal key norms)",
        "config": {"workload": wl.name, "batch": wl.batch, "layers": wl.n_layers,
                   "q_heads": wl.n_q_heads, "kv_heads": wl.n_kv_heads, "head_dim": D,
                   "context": wl.n0, "budget": wl.budget, "units": U,
                   "steady_len": L_steady, "steady_capacity": buf.cap,
                   "timed_steps": f"{n_wl + args.warmup}..{n_wl + args.warmup + args.steps - 1} "
                                  f"(entropy window full: every step retires step t - {fill})",
                   "policy": "4->%s->1 ReLU MLP" % "->".join(map(str, wl.hidden))},
        "kv_gbps": round(kv_gbps, 1),
        "kv_frac_of_8TBps": round(kv_gbps / HBM_PEAK_GBPS, 4),
        "kv_bytes_per_step": kvb,
        "moved_rows_per_step": moved,
        "step_kernel_ms": round(step_ms, 4),
        "hip_graph": False,       # one launch per steady step, issued directly
        "first_step_ms": round(first_ms, 3),
        "prewindow_step_ms": round(pre_ms, 4),
        "workload_window_full_step_ms": round(full_ms, 4),
        f"workload_{wl.steps}_step_avg_ms": round(wl_avg_ms, 4),
        f"workload_{wl.steps}_step_avg_steps_per_s": round(1e3 / wl_avg_ms, 3),
        "roofline": {"bound": "hbm", "kernel": "step_unit_kernel (attention + features + score + select + compact)",
                     "achieved": round(step_gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(step_gbps / HBM_PEAK_GBPS, 4),
                     "traffic": measured_traffic() if wl.name == W.WORKLOADS[3].name else None,
                     "alg_bytes_per_launch": step_bytes},
    }
    if copy_gbps:
        result["copy_gbps"] = round(copy_gbps, 1)
        result["kv_frac_of_copy"] = round(kv_gbps / copy_gbps, 4)
        result["roofline"]["frac_of_measured_copy"] = round(step_gbps / copy_gbps, 4)
    if not args.no_cpu_baseline:
        del buf, Q, KN, VN
        torch.cuda.empty_cache()
        workers = min(16, len(os.sched_getaffinity(0)))
        t_cpu = time.time()
        rate, cpu_s = run_oracle_baseline(wl, args.cpu_units, args.cpu_steps, workers)
        log(f"cpu oracle: {args.cpu_units} units x {args.cpu_steps} steps on {workers} workers, "
            f"{time.time() - t_cpu:.1f}s wall")
        result["cpu_baseline"] = {
            "value": rate / U, "unit": "decode steps/s", "cores": workers, "kind": "oracle",
            "cpu": cpu_model(),
            "sample": f"{args.cpu_units} of {U} units x {args.cpu_steps} window-full steady "
                      f"steps each ({cpu_s:.1f} CPU-s timed), {workers} worker processes x 1 "
                      f"BLAS thread; extrapolated from {args.cpu_units} units by the unit count; "
                      f"numpy float64"}
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
