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
