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


# up to 64 rows take the per-step kernel (workgroups of 8, 16, 32 or 64 rows),
# 65-128 the blocked GEMM, more the large-tile GEMM (partial row blocks,
# vocabularies that end inside a 256-column block, a 128k-token vocabulary:
# 2048 tiles per row in the merge)
@pytest.mark.parametrize("rows,hid,voc", [(1, 128, 64), (13, 256, 1024), (15, 128, 4160),
                                          (16, 128, 256), (17, 256, 4160), (32, 128, 640),
                                          (33, 128, 4160), (64, 512, 4096), (65, 128, 640),
                                          (100, 256, 4160), (128, 128, 640), (129, 256, 4160),
                                          (523, 128, 640), (4, 128, 131072)])
def test_kl_reward_shapes(rows, hid, voc):
    g = torch.Generator(device="cpu").manual_seed(rows * 7 + hid)
    hf = torch.randn(rows, hid, generator=g).to(torch.bfloat16)
    hc = (hf.float() + 0.3 * torch.randn(rows, hid, generator=g)).to(torch.bfloat16)
    w = (0.1 * torch.randn(voc, hid, generator=g)).to(torch.bfloat16)
    got = _kl_gpu(rows, hid, voc, hf.cuda(), hc.cuda(), w.cuda())
    ref = okl.kl_reward(hf.float().numpy(), hc.float().numpy(), w.float().numpy())
    assert _kl_ok(got, ref), (got, ref)


def test_kl_reward_deferred_rollout_full_size():
    """A rollout's rewards deferred to one call: 256 rows (32 steps x batch 8)
    at hidden 4096, vocab 32768 through the blocked GEMM; sampled rows (first
    and last of row blocks) against the oracle, one unpruned step exactly 0."""
    wl = W.WORKLOADS[5]
    hid, voc = wl.kl_hidden, wl.kl_vocab
    rows = 256
    w = torch.empty((voc, hid), dtype=torch.bfloat16, device="cuda")
    sg.fill_normal(w, wl, W.S_WLM, 0, 0.02)
    g = torch.Generator(device="cpu").manual_seed(2608)
    hf = torch.randn(rows, hid, generator=g).to(torch.bfloat16)
    hc = (hf.float() + 0.05 * torch.randn(rows, hid, generator=g)).to(torch.bfloat16)
    hc[7] = hf[7]
    got = _kl_gpu(rows, hid, voc, hf.cuda(), hc.cuda(), w)
    idx = [0, 7, 63, 64, 127, 128, 200, 255]
    ref = okl.kl_reward(hf.float().numpy()[idx], hc.float().numpy()[idx], _lm_head_np())
    assert got[7] == 0.0
    assert _kl_ok(got[idx], ref), (got[idx], ref)
    assert np.all(got >= 0)


def test_kl_reward_does_not_depend_on_the_rows_per_call():
    """The per-step kernel (up to 64 rows, 8, 16, 32 or 64 rows per workgroup) and
    both GEMM shapes (65..128 rows, 129 and more) give every row the same
    bits."""
    wl = W.WORKLOADS[5]
    hid, voc = wl.kl_hidden, wl.kl_vocab
    w = torch.empty((voc, hid), dtype=torch.bfloat16, device="cuda")
    sg.fill_normal(w, wl, W.S_WLM, 0, 0.02)
    g = torch.Generator(device="cpu").manual_seed(55)
    hf = torch.randn(300, hid, generator=g).to(torch.bfloat16).cuda()
    hc = (hf.float().cpu() + 0.05 * torch.randn(300, hid, generator=g)).to(torch.bfloat16).cuda()
    wide = _kl_gpu(300, hid, voc, hf, hc, w)
    narrow = _kl_gpu(100, hid, voc, hf[:100], hc[:100], w)
    step = _kl_gpu(8, hid, voc, hf[96:104].contiguous(), hc[96:104].contiguous(), w)
    step16 = _kl_gpu(13, hid, voc, hf[40:53].contiguous(), hc[40:53].contiguous(), w)
    step32 = _kl_gpu(29, hid, voc, hf[200:229].contiguous(), hc[200:229].contiguous(), w)
    step64 = _kl_gpu(50, hid, voc, hf[250:300].contiguous(), hc[250:300].contiguous(), w)
    assert np.array_equal(wide[:100], narrow)
    assert np.array_equal(wide[96:104], step)
    assert np.array_equal(wide[40:53], step16)
    assert np.array_equal(wide[200:229], step32)
    assert np.array_equal(wide[250:300], step64)


def test_kl_reward_at_the_maximum_row_count():
    """DC_KL_MAX_ROWS rows in one call (256 row blocks of the GEMM); sampled rows
    against the oracle, including the last."""
    rows, hid, voc = B.KL_MAX_ROWS, 256, 1024
    g = torch.Generator(device="cpu").manual_seed(16384)
    hf = torch.randn(rows, hid, generator=g).to(torch.bfloat16)
    hc = (hf.float() + 0.2 * torch.randn(rows, hid, generator=g)).to(torch.bfloat16)
    w = (0.1 * torch.randn(voc, hid, generator=g)).to(torch.bfloat16)
    got = _kl_gpu(rows, hid, voc, hf.cuda(), hc.cuda(), w.cuda())
    idx = [0, 1, 63, 64, 8191, 12345, rows - 65, rows - 1]
    ref = okl.kl_reward(hf.float().numpy()[idx], hc.float().numpy()[idx], w.float().numpy())
    assert _kl_ok(got[idx], ref), (got[idx], ref)
    assert np.all(got >= 0) and np.all(np.isfinite(got))
