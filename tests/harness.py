"""Shared helpers of the GPU parity tests: build oracle states from the input
generator, move unit states between the oracle and the device buffers, and the
comparison rules (kept sets bit-exact with the near-tie band; 2e-2 on bf16
attention outputs; 1e-3 on float32 features, scores and KL)."""
from __future__ import annotations

import math

import numpy as np
import torch

from oracle import attention as oatt
from oracle import compact as ocomp
from oracle import select as osel
from oracle import unit as ounit
from synth import philox as px
from synth import workloads as W

TIE_BAND = 1e-6          # |s - tau| <= band: selection ambiguous, excluded and counted
OUT_TOL = 2e-2           # bf16 attention output, max-abs relative per (unit, head)
FP_TOL = 1e-3            # float32 features, scores, KL


def dev():
    return torch.device("cuda")


def torch_dtype(wl):
    return torch.float32 if wl.dtype == "f32" else torch.bfloat16


def scale_of(wl):
    return oatt.default_scale(wl.head_dim)


def oracle_student(wl: W.Workload, u: int, n0: int | None = None, window: int | None = None):
    n0 = wl.n0 if n0 is None else n0
    pos = np.arange(n0)
    return ounit.new_student(W.key_rows(wl, u, pos), W.value_rows(wl, u, pos), pos, G=wl.group,
                             scale=scale_of(wl), window=wl.ent_window if window is None else window,
                             next_pos=n0)


def oracle_teacher(wl: W.Workload, u: int, n0: int | None = None):
    n0 = wl.n0 if n0 is None else n0
    pos = np.arange(n0)
    return ounit.new_teacher(W.key_rows(wl, u, pos), W.value_rows(wl, u, pos), pos,
                             scale=scale_of(wl), next_pos=n0)


def step_inputs_np(wl: W.Workload, step: int, u: int):
    q = W.queries(wl, step, u)
    if not wl.append:
        return q, None, None
    p = [wl.n0 + step]
    return q, W.key_rows(wl, u, p)[0], W.value_rows(wl, u, p)[0]


def to_np(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy() if t.dtype == torch.bfloat16 else t.detach().cpu().numpy()


def download_unit(buf, u: int) -> dict:
    """Rows [0, len) of unit u as numpy arrays (slot order)."""
    L = buf.kv.len
    d = {"k": to_np(buf.k[u, :L]).astype(np.float64), "v": to_np(buf.v[u, :L]).astype(np.float64)}
    if buf.feat is not None:
        d.update(pos=to_np(buf.pos[u, :L]).astype(np.int64), alpha=to_np(buf.alpha[u, :L]),
                 num=to_np(buf.num[u, :L]), den=to_np(buf.den[u, :L]),
                 vnorm=to_np(buf.vnorm[u, :L]))
    return d


def upload_unit(buf, u: int, st: ounit.StudentState) -> None:
    """Write an oracle state into unit u's device buffers (slots 0..L-1 in the
    oracle's row order; the ring gets the oracle's step records)."""
    L = st.L
    td = buf.k.dtype
    buf.k[u, :L] = torch.from_numpy(st.K.astype(np.float32)).to(td).to(buf.k.device)
    buf.v[u, :L] = torch.from_numpy(st.V.astype(np.float32)).to(td).to(buf.k.device)
    buf.pos[u, :L] = torch.from_numpy(st.pos.astype(np.int32)).to(buf.k.device)
    buf.alpha[u, :L] = torch.from_numpy(st.alpha.astype(np.float32)).to(buf.k.device)
    Z, N = st.hist.sums()
    buf.num[u, :L] = torch.from_numpy(N).to(buf.k.device)
    buf.den[u, :L] = torch.from_numpy(Z).to(buf.k.device)
    buf.vnorm[u, :L] = torch.from_numpy(np.sqrt((st.V ** 2).sum(1)).astype(np.float32)).to(buf.k.device)
    if buf.window > 0 and st.records:
        # the ring slots of the last w steps (slots of older steps are never read)
        ring = np.zeros(tuple(buf.qring.shape[1:]), np.float32)
        stat = np.zeros(tuple(buf.qstat.shape[1:]), np.float32)
        for step, rec in st.records.items():
            slot = step % buf.window
            ring[slot] = rec.q
            stat[slot] = np.stack([rec.m, 1.0 / rec.l, rec.H], axis=1)
        buf.qring[u] = torch.from_numpy(ring).to(td).to(buf.k.device)
        buf.qstat[u] = torch.from_numpy(stat).to(buf.k.device)


def set_host_fields(buf, st: ounit.StudentState) -> None:
    buf.kv.len = st.L
    buf.feat.step = st.step
    buf.feat.next_pos = st.next_pos
    for step, rec in st.records.items():
        buf.feat.ring_pmax[step % buf.window] = rec.pmax


# ------------------------------------------------------------------ comparisons

def rel_err_rows(got, ref) -> float:
    """max over rows of max|got - ref| / max|ref| (per head)."""
    got = np.asarray(got, np.float64).reshape(-1, np.shape(got)[-1])
    ref = np.asarray(ref, np.float64).reshape(-1, np.shape(ref)[-1])
    den = np.maximum(np.abs(ref).max(axis=1), 1e-30)
    return float((np.abs(got - ref).max(axis=1) / den).max())


def vec_ok(got, ref, tol=FP_TOL, floor_frac=1e-3) -> tuple[bool, float]:
    """|g - o| <= tol * max(|o|, floor_frac max|o|) elementwise; returns (ok, worst ratio)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    floor = floor_frac * max(np.abs(ref).max(), 1e-30)
    lim = tol * np.maximum(np.abs(ref), floor)
    ratio = np.abs(got - ref) / lim
    return bool(np.all(ratio <= 1.0)), float(ratio.max() if ratio.size else 0.0)


def by_position(d: dict) -> dict:
    order = np.argsort(d["pos"])
    return {k: v[order] for k, v in d.items()}


def selection_check(scores_oracle, pos, kept_pos_gpu, budget):
    """End-to-end kept-set comparison with the near-tie band.  Returns
    (ok, n_ambiguous, n_flips_in_band)."""
    s = np.asarray(scores_oracle, np.float64)
    L = len(s)
    if budget >= L:
        return set(kept_pos_gpu) == set(pos.tolist()), 0, 0
    order = osel.ranking(s, pos)
    tau = s[order[budget - 1]]
    amb = np.abs(s - tau) <= TIE_BAND
    kept_o = np.zeros(L, bool)
    kept_o[order[:budget]] = True
    kept_g = np.isin(pos, np.asarray(list(kept_pos_gpu)))
    mism = kept_o != kept_g
    return bool(not np.any(mism & ~amb)), int(amb.sum()), int((mism & amb).sum())


def oracle_slot_map(scores_gpu, pos, budget):
    """The oracle's selection applied to the GPU's own float32 scores, stored in
    the oracle's compaction order: the slot map that kept_out must equal."""
    kept = osel.top_budget(np.asarray(scores_gpu, np.float64), pos, budget)
    return ocomp.hole_fill(kept, len(pos))


def slot_map_of(kept_rows, n_rows):
    """The oracle's compaction order for a kept set decided elsewhere (sampled
    selection, whose kept set is checked on its own)."""
    return ocomp.hole_fill(kept_rows, n_rows)
