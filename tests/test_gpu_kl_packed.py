"""GPU checks of the packed lm-head layout (dc_kl_pack_lm_head) and of the KL
reward read through it (dc_kl_reward_packed): the layout against its
definition (64 x 64 blocks, tile-major, then stage), and the reward against the
row-major call bit for bit and against the oracle."""
import numpy as np
import pytest
import torch

from oracle import kl as okl
from paper_2608_08878_amd import binding as B
from synth import gpu as sg
from synth import workloads as W

from . import harness as H

pytestmark = pytest.mark.gpu


def _stream():
    return torch.cuda.current_stream().cuda_stream


def _pack(w):
    voc, hid = w.shape
    out = torch.empty_like(w)
    B.dc_kl_pack_lm_head(hid, voc, w, out, _stream())
    torch.cuda.synchronize()
    return out


def _blocked(w):
    """The layout's definition: block (t, k) = rows 64 t.., hidden 64 k.., row-major."""
    voc, hid = w.shape
    return w.view(voc // 64, 64, hid // 64, 64).permute(0, 2, 1, 3).contiguous().view(voc, hid)


def _kl(fn, rows, hid, voc, hf, hc, w):
    ws = torch.empty(B.dc_workspace_bytes(B.dc_dims(), 0, rows, voc), dtype=torch.uint8, device="cuda")
    out = torch.empty(rows, dtype=torch.float32, device="cuda")
    fn(rows, hid, voc, hf, hc, w, out, ws, ws.numel(), _stream())
    torch.cuda.synchronize()
    return H.to_np(out)


def _full_size_head():
    wl = W.WORKLOADS[5]
    w = torch.empty((wl.kl_vocab, wl.kl_hidden), dtype=torch.bfloat16, device="cuda")
    sg.fill_normal(w, wl, W.S_WLM, 0, 0.02)
    return w


@pytest.mark.parametrize("voc,hid", [(64, 128), (192, 384), (4160, 256), (32768, 4096)])
def test_pack_layout_matches_its_definition(voc, hid):
    if voc == 32768:
        w = _full_size_head()
    else:
        g = torch.Generator(device="cpu").manual_seed(voc + hid)
        w = torch.randn(voc, hid, generator=g).to(torch.bfloat16).cuda()
    p = _pack(w)
    assert torch.equal(p.view(torch.int16), _blocked(w).view(torch.int16))
    # the source is left as it was
    if voc != 32768:
        assert torch.equal(w.cpu(), torch.randn(voc, hid, generator=torch.Generator(device="cpu")
                                                .manual_seed(voc + hid)).to(torch.bfloat16))


# every kernel the reward dispatches to (per-step up to 64 rows in workgroups
# of 8, 16, 32 or 64, the two GEMM shapes from 65 and from 129 rows) on both
# sides of each boundary, vocabularies ending inside a GEMM block
@pytest.mark.parametrize("rows,hid,voc", [(1, 128, 64), (8, 256, 1024), (9, 128, 640),
                                          (16, 128, 4160), (17, 128, 256), (32, 256, 4160),
                                          (64, 128, 640), (65, 128, 4160), (128, 128, 640),
                                          (129, 128, 4160), (523, 128, 640)])
def test_packed_reward_is_bit_identical_and_matches_the_oracle(rows, hid, voc):
    g = torch.Generator(device="cpu").manual_seed(rows * 11 + voc)
    hf = torch.randn(rows, hid, generator=g).to(torch.bfloat16)
    hc = (hf.float() + 0.3 * torch.randn(rows, hid, generator=g)).to(torch.bfloat16)
    w = (0.1 * torch.randn(voc, hid, generator=g)).to(torch.bfloat16).cuda()
    hfd, hcd = hf.cuda(), hc.cuda()
    plain = _kl(B.dc_kl_reward, rows, hid, voc, hfd, hcd, w)
    packed = _kl(B.dc_kl_reward_packed, rows, hid, voc, hfd, hcd, _pack(w))
    assert np.array_equal(plain.view(np.uint32), packed.view(np.uint32))
    ref = okl.kl_reward(hf.float().numpy(), hc.float().numpy(), w.float().cpu().numpy())
    assert np.all(np.abs(packed - ref) <= 1e-3 * np.abs(ref) + 1e-6), (packed, ref)


@pytest.mark.parametrize("rows", [8, 32, 64, 100, 300])
def test_packed_reward_full_size(rows):
    """hidden 4096, vocab 32768: the per-step call (8 rows; 32 and 64 rows, four
    and eight 8-row blocks per workgroup), the blocked GEMM (100 rows) and the large-tile GEMM
    (300 rows, a partial last row block),
    bit-identical to the row-major weight; sampled rows against the oracle;
    an unpruned row exactly 0."""
    wl = W.WORKLOADS[5]
    hid, voc = wl.kl_hidden, wl.kl_vocab
    w = _full_size_head()
    g = torch.Generator(device="cpu").manual_seed(4096 + rows)
    hf = torch.randn(rows, hid, generator=g).to(torch.bfloat16)
    hc = (hf.float() + 0.05 * torch.randn(rows, hid, generator=g)).to(torch.bfloat16)
    hc[3] = hf[3]
    hfd, hcd = hf.cuda(), hc.cuda()
    plain = _kl(B.dc_kl_reward, rows, hid, voc, hfd, hcd, w)
    packed = _kl(B.dc_kl_reward_packed, rows, hid, voc, hfd, hcd, _pack(w))
    assert np.array_equal(plain.view(np.uint32), packed.view(np.uint32))
    assert packed[3] == 0.0
    idx = {8: [0, 3, 7], 32: [0, 3, 15, 16, 31], 64: [0, 3, 31, 32, 63], 100: [0, 3, 63, 64, 99],
           300: [0, 3, 127, 128, 255, 256, 299]}[rows]
    ref = okl.kl_reward(hf.float().numpy()[idx], hc.float().numpy()[idx], w.float().cpu().numpy())
    assert np.all(np.abs(packed[idx] - ref) <= 1e-3 * np.abs(ref) + 1e-6), (packed[idx], ref)


def test_packed_reward_at_the_maximum_row_count():
    """DC_KL_MAX_ROWS rows (the blocked GEMM's largest grid) through the packed
    layout: bit-identical to the row-major call, sampled rows against the oracle."""
    rows, hid, voc = B.KL_MAX_ROWS, 256, 1024
    g = torch.Generator(device="cpu").manual_seed(16385)
    hf = torch.randn(rows, hid, generator=g).to(torch.bfloat16)
    hc = (hf.float() + 0.2 * torch.randn(rows, hid, generator=g)).to(torch.bfloat16)
    w = (0.1 * torch.randn(voc, hid, generator=g)).to(torch.bfloat16).cuda()
    hfd, hcd = hf.cuda(), hc.cuda()
    plain = _kl(B.dc_kl_reward, rows, hid, voc, hfd, hcd, w)
    packed = _kl(B.dc_kl_reward_packed, rows, hid, voc, hfd, hcd, _pack(w))
    assert np.array_equal(plain.view(np.uint32), packed.view(np.uint32))
    idx = [0, 127, 128, 9999, rows - 1]
    ref = okl.kl_reward(hf.float().numpy()[idx], hc.float().numpy()[idx], w.float().cpu().numpy())
    assert np.all(np.abs(packed[idx] - ref) <= 1e-3 * np.abs(ref) + 1e-6), (packed[idx], ref)
