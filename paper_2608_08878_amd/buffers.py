"""Device buffers for the C-ABI structs, allocated with torch (device memory and
streams only; no computation happens here)."""
from __future__ import annotations

import ctypes

import torch

from . import binding as B

TORCH_DTYPE = {"f32": torch.float32, "bf16": torch.bfloat16}
DC_DTYPE = {"f32": B.DC_F32, "bf16": B.DC_BF16}


def stream_handle(stream=None):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


class DecodeBuffers:
    """K/V cache and (optionally) feature state for `units` caches of `capacity` rows."""

    def __init__(self, batch, n_layers, n_q_heads, n_kv_heads, head_dim, capacity, dtype="bf16",
                 ent_window=64, scale=0.0, features=True, device="cuda", sigma=False,
                 ragged=False, alpha_recent=False):
        self.G = n_q_heads // n_kv_heads
        self.U = batch * n_layers * n_kv_heads
        self.D = head_dim
        self.cap = capacity
        self.dtype = dtype
        self.window = ent_window
        td = TORCH_DTYPE[dtype]
        self.dims = B.dc_dims(batch, n_layers, n_q_heads, n_kv_heads, head_dim, capacity,
                              DC_DTYPE[dtype], ent_window, scale)
        self.k = torch.zeros((self.U, capacity, head_dim), dtype=td, device=device)
        self.v = torch.zeros((self.U, capacity, head_dim), dtype=td, device=device)
        self.kv = B.dc_kv(self.k.data_ptr(), self.v.data_ptr(), 0)
        self.unit_len = None
        if ragged:
            # per-unit lengths on the device (units may keep different row counts)
            self.unit_len = torch.zeros(self.U, dtype=torch.int32, device=device)
            self.kv.unit_len = self.unit_len.data_ptr()
        self.feat = None
        if features:
            self.alpha = torch.zeros((self.U, capacity), dtype=torch.float32, device=device)
            self.num = torch.zeros((self.U, capacity), dtype=torch.float64, device=device)
            self.den = torch.zeros((self.U, capacity), dtype=torch.float64, device=device)
            self.pos = torch.zeros((self.U, capacity), dtype=torch.int32, device=device)
            self.vnorm = torch.zeros((self.U, capacity), dtype=torch.float32, device=device)
            w = max(ent_window, 1)
            self.qring = torch.zeros((self.U, w, self.G, head_dim), dtype=td, device=device)
            self.qstat = torch.zeros((self.U, w, self.G, 3), dtype=torch.float32, device=device)
            self.feat = B.dc_feat(self.alpha.data_ptr(), self.num.data_ptr(), self.den.data_ptr(),
                                  self.pos.data_ptr(), self.vnorm.data_ptr(),
                                  self.qring.data_ptr(), self.qstat.data_ptr(), 0, 0)
            self.feat.alpha_recent = int(alpha_recent)
            self.ga_ws = None
            self.sigma = None
            if sigma:
                # the fifth feature (needed by five-input policies)
                self.sigma = torch.zeros((self.U, capacity), dtype=torch.float32, device=device)
                self.feat.sigma = self.sigma.data_ptr()
        self.ws = None
        self.ws_bytes = 0
        if features:
            self.reserve_workspace(capacity)

    @property
    def len(self) -> int:
        return self.kv.len

    def shrink(self, capacity: int):
        """Move the valid rows of every unit into buffers of a smaller capacity (device
        copies; the old buffers are released).  After a compression step only
        budget + 1 rows per unit are ever live, and the steady steps stream fewer
        distinct pages when each unit's rows sit closer together."""
        n = self.kv.len
        if capacity < n + 1:
            raise ValueError(f"capacity {capacity} cannot hold {n} rows plus an append")
        td = self.k.dtype
        dev = self.k.device

        def moved(t):
            out = torch.zeros((t.shape[0], capacity) + tuple(t.shape[2:]), dtype=t.dtype, device=dev)
            out[:, :n] = t[:, :n]
            return out

        self.k = moved(self.k)
        self.v = moved(self.v)
        self.kv.k, self.kv.v = self.k.data_ptr(), self.v.data_ptr()
        if self.feat is not None:
            self.alpha, self.num, self.den = moved(self.alpha), moved(self.num), moved(self.den)
            self.pos, self.vnorm = moved(self.pos), moved(self.vnorm)
            if self.sigma is not None:
                self.sigma = moved(self.sigma)
                self.feat.sigma = self.sigma.data_ptr()
            self.feat.alpha, self.feat.ent_num = self.alpha.data_ptr(), self.num.data_ptr()
            self.feat.ent_den, self.feat.pos = self.den.data_ptr(), self.pos.data_ptr()
            self.feat.vnorm = self.vnorm.data_ptr()
        self.cap = capacity
        self.dims.capacity = capacity
        assert self.k.dtype == td
        torch.cuda.synchronize(dev)

    def reserve_workspace(self, max_len: int, kl_rows: int = 0, kl_vocab: int = 0):
        need = B.dc_workspace_bytes(self.dims, max_len, kl_rows, kl_vocab)
        if need > self.ws_bytes:
            self.ws = torch.empty(need, dtype=torch.uint8, device=self.k.device)
            self.ws_bytes = need
        return self.ws

    def feat_init(self, length: int, first_pos: int = 0, stream=None):
        self.kv.len = length
        if self.unit_len is not None:
            self.unit_len.fill_(length)
        B.dc_feat_init(self.dims, self.kv, self.feat, first_pos, stream_handle(stream))

    def decode_step(self, q, k_new=None, v_new=None, out=None, stream=None, features=True):
        if out is None:
            out = torch.empty_like(q)
        B.dc_decode_step(self.dims, self.kv, self.feat if features else None, q, k_new, v_new,
                         out, self.ws, self.ws_bytes, stream_handle(stream))
        return out

    def decode_evict(self, policy, budget, q, k_new=None, v_new=None, out=None, scores_out=None,
                     kept_out=None, stream=None):
        if out is None:
            out = torch.empty_like(q)
        B.dc_decode_evict(self.dims, self.kv, self.feat, policy, budget, q, k_new, v_new, out,
                          scores_out, kept_out, self.ws, self.ws_bytes, stream_handle(stream))
        return out

    def global_alpha(self, stream=None):
        """Replace every row's recent alpha by its average over the sequence's
        units (all layers and KV heads) at the row's position."""
        need = B.dc_global_alpha_workspace_bytes(self.dims, self.feat.next_pos)
        if self.ga_ws is None or self.ga_ws.numel() < need:
            self.ga_ws = torch.empty(need, dtype=torch.uint8, device=self.k.device)
        B.dc_global_alpha(self.dims, self.kv, self.feat, self.ga_ws, self.ga_ws.numel(),
                          stream_handle(stream))

    def score_evict(self, policy, budget, scores_out=None, kept_out=None, stream=None):
        B.dc_score_evict(self.dims, self.kv, self.feat, policy, budget, scores_out, kept_out,
                         self.ws, self.ws_bytes, stream_handle(stream))


    def decode_sample_evict(self, policy, budget, gumbel, q, k_new=None, v_new=None, out=None,
                            scores_out=None, kept_out=None, logp_out=None, stream=None):
        if out is None:
            out = torch.empty_like(q)
        B.dc_decode_sample_evict(self.dims, self.kv, self.feat, policy, budget, gumbel, q, k_new,
                                 v_new, out, scores_out, kept_out, logp_out, self.ws, self.ws_bytes,
                                 stream_handle(stream))
        return out

    def decode_evict_units(self, policy, budgets, max_budget, q, k_new, v_new, out=None,
                           scores_out=None, kept_out=None, stream=None):
        """One decode step of a ragged cache with per-unit budgets (decode, then the
        deterministic per-unit selection); units that fit on chip run it in one launch."""
        if out is None:
            out = torch.empty_like(q)
        B.dc_decode_evict_units(self.dims, self.kv, self.feat, policy, budgets, max_budget, q,
                                k_new, v_new, out, scores_out, kept_out, self.ws, self.ws_bytes,
                                stream_handle(stream))
        return out

    def score_evict_units(self, policy, budgets, max_budget, gumbel=None, scores_out=None,
                          kept_out=None, logp_out=None, stream=None):
        B.dc_score_evict_units(self.dims, self.kv, self.feat, policy, budgets, max_budget, gumbel,
                               scores_out, kept_out, logp_out, self.ws, self.ws_bytes,
                               stream_handle(stream))

    def sample_evict(self, policy, budget, gumbel, scores_out=None, kept_out=None, logp_out=None,
                     stream=None):
        B.dc_sample_evict(self.dims, self.kv, self.feat, policy, budget, gumbel, scores_out,
                          kept_out, logp_out, self.ws, self.ws_bytes, stream_handle(stream))


def subset_log_prob(scores: torch.Tensor, budget: int, tau: float = 1.0, kept=None, logz=True,
                    stream=None):
    """log Z and (with `kept`) log pi for every row of `scores` ([units][len] float32
    on the device).  Returns (logz, logp) float64 tensors (logp None without kept)."""
    units, length = scores.shape
    dev = scores.device
    lz = torch.empty(units, dtype=torch.float64, device=dev) if logz else None
    lp = torch.empty(units, dtype=torch.float64, device=dev) if kept is not None else None
    need = B.dc_subset_log_prob_workspace_bytes(units, length, budget)
    ws = torch.empty(need, dtype=torch.uint8, device=dev) if need else None
    B.dc_subset_log_prob(units, length, budget, tau, scores, kept, lz, lp, ws, need,
                         stream_handle(stream))
    return lz, lp


def make_policy(params: torch.Tensor, hidden, n_in: int = 4, layer_norm: bool = False) -> B.dc_policy:
    hidden = tuple(hidden)
    h = (ctypes.c_int32 * 2)(hidden[0], hidden[1] if len(hidden) > 1 else 0)
    return B.dc_policy(n_in, len(hidden), h, params.data_ptr(), int(layer_norm))
