"""GPU check of the allocation-free KL entry point (dc_kl_reward_static): the
same rewards, bit for bit, as dc_kl_reward with a caller workspace, and within
the KL tolerance of the oracle, on two calls in a row that share the fixed
scratch, the second with a smaller input."""
import numpy as np
import pytest
import torch

from oracle import kl as okl
from paper_2608_08878_amd import binding as B

from . import harness as H

pytestmark = pytest.mark.gpu


def _inputs(rows, hid, voc, seed):
    g = torch.Generator(device="cpu").manual_seed(seed)
    hf = torch.randn(rows, hid, generator=g).to(torch.bfloat16)
    hc = (hf.float() + 0.3 * torch.randn(rows, hid, generator=g)).to(torch.bfloat16)
    w = (0.02 * torch.randn(voc, hid, generator=g)).to(torch.bfloat16)
    return hf.cuda(), hc.cuda(), w.cuda()


def _with_workspace(rows, hid, voc, hf, hc, w):
    ws = torch.empty(B.KL_STATIC_MAX_PAIRS * 16, dtype=torch.uint8, device="cuda")
    kl = torch.empty(rows, dtype=torch.float32, device="cuda")
    B.dc_kl_reward(rows, hid, voc, hf, hc, w, kl, ws, ws.numel(),
                   torch.cuda.current_stream().cuda_stream)
    return kl


def test_static_kl_matches_the_workspace_entry_point_on_two_calls():
    stream = torch.cuda.current_stream().cuda_stream
    # first call: 1024 rows of the 32768-entry vocabulary fill the scratch exactly
    # (blocked GEMM path); second call: 8 rows (per-step path) over a smaller vocabulary
    for rows, hid, voc, seed in ((1024, 4096, 32768, 1), (8, 1024, 8192, 2)):
        print(f"static KL: rows={rows} hidden={hid} vocab={voc}", flush=True)
        hf, hc, w = _inputs(rows, hid, voc, seed)
        kl_s = torch.full((rows,), float("nan"), dtype=torch.float32, device="cuda")
        B.dc_kl_reward_static(rows, hid, voc, hf, hc, w, kl_s, stream)
        kl_w = _with_workspace(rows, hid, voc, hf, hc, w)
        torch.cuda.synchronize()
        assert torch.equal(kl_s, kl_w), (rows, voc)
        # the oracle on sampled rows (binary64)
        sample = sorted({0, rows - 1, *np.random.default_rng(seed).choice(rows, 6).tolist()})
        idx = torch.tensor(sample, device="cuda")
        ref = okl.kl_reward(H.to_np(hf[idx]).astype(np.float64), H.to_np(hc[idx]).astype(np.float64),
                            H.to_np(w).astype(np.float64))
        got = H.to_np(kl_s)[sample]
        assert np.all(np.abs(got - ref) <= H.FP_TOL * np.abs(ref) + 1e-6), (rows, got, ref)
    # identical hidden states give exactly zero from the static scratch as well
    hf, _, w = _inputs(8, 1024, 8192, 3)
    kl0 = torch.full((8,), float("nan"), dtype=torch.float32, device="cuda")
    B.dc_kl_reward_static(8, 1024, 8192, hf, hf, w, kl0, stream)
    torch.cuda.synchronize()
    assert torch.all(kl0 == 0)


def test_static_kl_rejects_a_call_past_its_scratch_and_leaves_the_output():
    hf, hc, w = _inputs(8, 128, 64, 4)
    kl = torch.full((8,), 7.0, dtype=torch.float32, device="cuda")
    with pytest.raises(B.DCError) as e:
        B.dc_kl_reward_static(1025, 4096, 32768, hf, hc, w, kl)
    assert e.value.status == 9
    torch.cuda.synchronize()
    assert torch.all(kl == 7.0)


def test_static_kl_under_graph_capture_replays_bit_identically():
    """The allocation-free entry point inside a captured HIP graph: three
    replays, new hidden states copied in eagerly before each, every replay's
    rewards bit-identical to an eager dc_kl_reward call on the same inputs."""
    rows, hid, voc = 8, 1024, 8192
    hf, hc, w = _inputs(rows, hid, voc, 10)
    kl_g = torch.empty(rows, dtype=torch.float32, device="cuda")
    # the first call looks the scratch address up (outside the capture)
    B.dc_kl_reward_static(rows, hid, voc, hf, hc, w, kl_g, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        B.dc_kl_reward_static(rows, hid, voc, hf, hc, w, kl_g,
                              torch.cuda.current_stream().cuda_stream)
    for rep in range(3):
        print(f"graph replay {rep}", flush=True)
        nf, nc, _ = _inputs(rows, hid, voc, 20 + rep)
        hf.copy_(nf)
        hc.copy_(nc)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        kl_w = _with_workspace(rows, hid, voc, hf, hc, w)
        torch.cuda.synchronize()
        assert torch.equal(kl_g, kl_w), rep
        assert torch.all(kl_g > 0)
