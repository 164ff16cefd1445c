"""GPU parity of the KL reward (MFMA lm-head GEMM + fused log-softmax/KL)."""
import functools

import numpy as np
import pytest
import torch

from oracle import kl as okl
from paper_2608_08878_amd import binding as B
from synth import gpu as sg
from synth import workloads as W

from . import harness as H

pytestmark = pytest.mark.gpu


def _kl_gpu(rows, hidden, vocab, hf, hc, w):
    ws = torch.empty(B.dc_workspace_bytes(B.dc_dims(), 0, rows, vocab), dtype=torch.uint8, device="cuda")
    out = torch.empty(rows, dtype=torch.float32, device="cuda")
    B.dc_kl_reward(rows, hidden, vocab, hf, hc, w, out, ws, ws.numel(),
                   torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    return H.to_np(out)


def _kl_ok(got, ref):
    return bool(np.all(np.abs(got - ref) <= 1e-3 * np.abs(ref) + 1e-6))


@functools.lru_cache(maxsize=1)
def _lm_head_np():
    return W.lm_head(W.WORKLOADS[5])


@pytest.mark.parametrize("which", ["comp", "noisy", "equal"])
def test_kl_reward_full_size(which):
    """8 rows, hidden 4096, vocab 32768 (lm head 4096 x 32768 bf16, N(0, 0.02))."""
    wl = W.WORKLOADS[5]
    rows, hid, voc = wl.batch, wl.kl_hidden, wl.kl_vocab
    w = torch.empty((voc, hid), dtype=torch.bfloat16, device="cuda")
    sg.fill_normal(w, wl, W.S_WLM, 0, 0.02)
    hf = torch.empty((rows, hid), dtype=torch.bfloat16, device="cuda")
    sg.fill_normal(hf, wl, W.S_HFULL, 0, 1.0)
    hc = torch.empty_like(hf)
    if which == "equal":
        hc.copy_(hf)
    elif which == "comp":
        sg.fill_normal(hc, wl, W.S_HCOMP, 0, 1.0)
    else:
        sg.fill_noisy(hc, hf, wl, 0, 0.01)
    got = _kl_gpu(rows, hid, voc, hf, hc, w)
    Wn = _lm_head_np()
    assert np.array_equal(H.to_np(w), Wn)
    ref = okl.kl_reward(W.hidden_states(wl, 0, "full"), W.hidden_states(wl, 0, which), Wn)
    if which == "equal":
        assert np.all(got == 0.0)
    assert _kl_ok(got, ref), (got, ref)
    assert np.all(got >= 0)


@pytest.mark.parametrize("rows,hid,voc", [(1, 128, 64), (13, 256, 1024), (64, 512, 4096)])
def test_kl_reward_shapes(rows, hid, voc):
    g = torch.Generator(device="cpu").manual_seed(rows * 7 + hid)
    hf = torch.randn(rows, hid, generator=g).to(torch.bfloat16)
    hc = (hf.float() + 0.3 * torch.randn(rows, hid, generator=g)).to(torch.bfloat16)
    w = (0.1 * torch.randn(voc, hid, generator=g)).to(torch.bfloat16)
    got = _kl_gpu(rows, hid, voc, hf.cuda(), hc.cuda(), w.cuda())
    ref = okl.kl_reward(hf.float().numpy(), hc.float().numpy(), w.float().numpy())
    assert _kl_ok(got, ref), (got, ref)
