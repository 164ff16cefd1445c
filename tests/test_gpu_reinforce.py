"""GPU parity of the rollout reward math (Sec. 3.2) and of the deferred,
many-row KL reward (Sec. 3.1.4): the HIP path through the C ABI against the
oracle.  Float64 arithmetic on both sides: 1e-12 relative, scaled by the
magnitude of the sums involved."""
import numpy as np
import pytest
import torch

from oracle import kl as okl
from oracle import reinforce as orf
from paper_2608_08878_amd import binding as B
from synth import gpu as sg
from synth import philox as px
from synth import workloads as W

from . import harness as H
from .test_gpu_kl import _kl_gpu, _kl_ok, _lm_head_np

pytestmark = pytest.mark.gpu

STREAM_R, STREAM_LP = 43, 44


def _inputs(T, K, step):
    seed = W.WORKLOADS[5].seed
    idx = np.arange(T * K, dtype=np.uint64)
    R = px.to_f32(-np.abs(px.normal(seed, STREAM_R, step, idx)) * 0.05).reshape(T, K)
    lp = (-50.0 - 10.0 * np.abs(px.normal(seed, STREAM_LP, step, idx))).reshape(T, K)
    return R, lp


def _run(T, K, R, lp, cfg, ema0):
    d = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a)).to(dt).cuda()
    r, l = d(R, torch.float32), d(lp, torch.float64)
    ema = torch.tensor([ema0], dtype=torch.float64, device="cuda")
    outs = [torch.empty((T, K), dtype=torch.float64, device="cuda") for _ in range(4)]
    stats = torch.empty(3, dtype=torch.float64, device="cuda")
    B.dc_reinforce_terms(T, K, cfg, r, l, ema, *outs, stats, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    return [o.cpu().numpy() for o in outs], stats.cpu().numpy(), float(ema.item())


def _close(got, ref, scale):
    return bool(np.all(np.abs(np.asarray(got) - np.asarray(ref)) <= 1e-12 * (np.abs(ref) + scale)))


@pytest.mark.parametrize("T,K,gamma,beta,d", [(1, 1, 0.99, 0.01, 0.9), (64, 8, 0.99, 0.01, 0.9),
                                             (37, 1, 0.5, 0.0, 0.0), (200, 5, 1.0, 0.2, 0.99),
                                             (5, 300, 0.0, 0.01, 0.5), (300, 2, 0.99, 0.01, 0.9)])
def test_reinforce_terms_match_oracle(T, K, gamma, beta, d):
    R, lp = _inputs(T, K, T * 1000 + K)
    cfg = B.dc_reinforce_cfg(gamma, beta, d)
    ema0 = -0.7
    (G, b, A, w), stats, ema = _run(T, K, R, lp, cfg, ema0)
    ref = orf.reinforce_terms(R, lp, gamma, beta, ema0, d)
    sG = np.abs(ref["returns"]).max() + 1e-30
    assert _close(G, ref["returns"], sG)
    assert _close(b, ref["baseline"], sG)
    assert _close(A, ref["advantage"], sG)
    assert _close(w, ref["weight"], (sG + abs(beta)) / (T * K))
    scale = np.abs(lp).max() * (sG + abs(beta))
    assert _close([stats[0]], [ref["loss"]], scale)
    assert _close([stats[1]], [ref["entropy"]], np.abs(lp).max())
    assert _close([stats[2]], [ref["returns"].mean()], sG)
    assert _close([ema], [ref["ema"]], sG + abs(ema0))


def test_reinforce_long_rollout_properties():
    """4096 steps: gamma = 1 gives suffix sums (library cumsum), and the RLOO
    advantages of every step sum to zero."""
    T, K = 4096, 3
    R, lp = _inputs(T, K, 7)
    (G, b, A, w), stats, ema = _run(T, K, R, lp, B.dc_reinforce_cfg(1.0, 0.01, 0.9), 0.0)
    suffix = np.flip(np.cumsum(np.flip(R.astype(np.float64), 0), 0), 0)
    assert np.all(np.abs(G - suffix) <= 1e-12 * (np.abs(suffix).max() + 1))
    assert np.all(np.abs(A.sum(1)) <= 1e-12 * np.abs(G).max() * K)


def test_deferred_kl_of_a_rollout():
    """512 rows (64 steps x batch 8) in one call against the oracle on sampled
    steps, and each step's rows bit-identical to the per-step call."""
    wl = W.WORKLOADS[5]
    b, hid, voc, T = wl.batch, wl.kl_hidden, wl.kl_vocab, 64
    w = torch.empty((voc, hid), dtype=torch.bfloat16, device="cuda")
    sg.fill_normal(w, wl, W.S_WLM, 0, 0.02)
    hf = torch.empty((T, b, hid), dtype=torch.bfloat16, device="cuda")
    hc = torch.empty_like(hf)
    for t in range(T):
        sg.fill_normal(hf[t], wl, W.S_HFULL, t, 1.0)
        sg.fill_noisy(hc[t], hf[t], wl, t, 0.01)
    got = _kl_gpu(T * b, hid, voc, hf.view(T * b, hid), hc.view(T * b, hid), w).reshape(T, b)
    Wn = _lm_head_np()
    for t in (0, 17, 63):
        ref = okl.kl_reward(W.hidden_states(wl, t, "full"), W.hidden_states(wl, t, "noisy"), Wn)
        assert _kl_ok(got[t], ref), (t, got[t], ref)
        one = _kl_gpu(b, hid, voc, hf[t], hc[t], w)
        assert np.array_equal(one, got[t]), t
    assert np.all(got >= 0)


@pytest.mark.parametrize("rows", [65, 100, 1000])
def test_kl_ragged_row_counts(rows):
    hid, voc = 256, 2048
    g = torch.Generator(device="cpu").manual_seed(rows)
    hf = torch.randn(rows, hid, generator=g).to(torch.bfloat16)
    hc = (hf.float() + 0.3 * torch.randn(rows, hid, generator=g)).to(torch.bfloat16)
    w = (0.1 * torch.randn(voc, hid, generator=g)).to(torch.bfloat16)
    got = _kl_gpu(rows, hid, voc, hf.cuda(), hc.cuda(), w.cuda())
    ref = okl.kl_reward(hf.float().numpy(), hc.float().numpy(), w.float().numpy())
    assert _kl_ok(got, ref)
