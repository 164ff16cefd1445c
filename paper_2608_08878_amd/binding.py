"""ctypes binding of libdistillcache.so: the C-ABI structs and entry points
under the same names (argument marshalling only; all work runs in the HIP
kernels).  Tensors are passed as device pointers (``Tensor.data_ptr()``)."""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdistillcache.so")

MAX_WINDOW = 64
DC_F32, DC_BF16 = 0, 1
STATUS = {0: "DC_OK", 1: "DC_ERR_NULL", 2: "DC_ERR_SHAPE", 3: "DC_ERR_UNSUPPORTED",
          4: "DC_ERR_CAPACITY", 5: "DC_ERR_BUDGET", 6: "DC_ERR_WORKSPACE", 7: "DC_ERR_HIP",
          8: "DC_ERR_VALUE", 9: "DC_ERR_SCRATCH"}


class dc_dims(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("n_layers", ctypes.c_int32),
                ("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("capacity", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("ent_window", ctypes.c_int32),
                ("scale", ctypes.c_float)]


class dc_kv(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("len", ctypes.c_int32),
                ("unit_len", ctypes.c_void_p)]


class dc_feat(ctypes.Structure):
    _fields_ = [("alpha", ctypes.c_void_p), ("ent_num", ctypes.c_void_p),
                ("ent_den", ctypes.c_void_p), ("pos", ctypes.c_void_p),
                ("vnorm", ctypes.c_void_p), ("qring", ctypes.c_void_p),
                ("qstat", ctypes.c_void_p), ("step", ctypes.c_int32),
                ("next_pos", ctypes.c_int32), ("ring_pmax", ctypes.c_int32 * MAX_WINDOW),
                ("sigma", ctypes.c_void_p), ("alpha_recent", ctypes.c_int32)]


class dc_policy(ctypes.Structure):
    _fields_ = [("n_in", ctypes.c_int32), ("n_hidden_layers", ctypes.c_int32),
                ("hidden", ctypes.c_int32 * 2), ("params", ctypes.c_void_p),
                ("layer_norm", ctypes.c_int32)]


class dc_gumbel(ctypes.Structure):
    _fields_ = [("tau", ctypes.c_float), ("seed", ctypes.c_uint32 * 2), ("draw", ctypes.c_uint32)]


def make_gumbel(tau: float, seed: int, draw: int) -> dc_gumbel:
    s = (ctypes.c_uint32 * 2)(seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF)
    return dc_gumbel(tau, s, draw & 0xFFFFFFFF)


class dc_reinforce_cfg(ctypes.Structure):
    _fields_ = [("gamma", ctypes.c_double), ("beta", ctypes.c_double), ("ema_decay", ctypes.c_double)]


KL_MAX_ROWS = 16384
KL_STATIC_MAX_PAIRS = 524288     # rows * (vocab / 64) of one dc_kl_reward_static call

EXPORTS = ("dc_workspace_bytes", "dc_feat_init", "dc_decode_step", "dc_score_evict",
           "dc_decode_evict", "dc_sample_evict", "dc_decode_sample_evict", "dc_score_evict_units",
           "dc_decode_evict_units",
           "dc_subset_log_prob",
           "dc_subset_log_prob_workspace_bytes", "dc_kl_reward", "dc_kl_pack_lm_head",
           "dc_kl_reward_packed", "dc_kl_reward_static",
           "dc_reinforce_terms",
           "dc_dynamic_budget", "dc_global_alpha", "dc_global_alpha_workspace_bytes",
           "dc_status_str")

_lib = None


def lib() -> ctypes.CDLL:
    """Load the HIP library; raises if it has not been built (there is no fallback)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with "
                              "python -m paper_2608_08878_amd.build (or __graft_entry__.build())")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        L.dc_workspace_bytes.argtypes = [ctypes.POINTER(dc_dims), i32, i32, i32]
        L.dc_workspace_bytes.restype = sz
        L.dc_feat_init.argtypes = [ctypes.POINTER(dc_dims), ctypes.POINTER(dc_kv),
                                   ctypes.POINTER(dc_feat), i32, vp]
        L.dc_feat_init.restype = ctypes.c_int
        L.dc_decode_step.argtypes = [ctypes.POINTER(dc_dims), ctypes.POINTER(dc_kv),
                                     ctypes.POINTER(dc_feat), vp, vp, vp, vp, vp, sz, vp]
        L.dc_decode_step.restype = ctypes.c_int
        L.dc_score_evict.argtypes = [ctypes.POINTER(dc_dims), ctypes.POINTER(dc_kv),
                                     ctypes.POINTER(dc_feat), ctypes.POINTER(dc_policy), i32,
                                     vp, vp, vp, sz, vp]
        L.dc_score_evict.restype = ctypes.c_int
        L.dc_decode_evict.argtypes = [ctypes.POINTER(dc_dims), ctypes.POINTER(dc_kv),
                                      ctypes.POINTER(dc_feat), ctypes.POINTER(dc_policy), i32,
                                      vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.dc_decode_evict.restype = ctypes.c_int
        L.dc_sample_evict.argtypes = [ctypes.POINTER(dc_dims), ctypes.POINTER(dc_kv),
                                      ctypes.POINTER(dc_feat), ctypes.POINTER(dc_policy), i32,
                                      ctypes.POINTER(dc_gumbel), vp, vp, vp, vp, sz, vp]
        L.dc_sample_evict.restype = ctypes.c_int
        L.dc_decode_sample_evict.argtypes = [ctypes.POINTER(dc_dims), ctypes.POINTER(dc_kv),
                                             ctypes.POINTER(dc_feat), ctypes.POINTER(dc_policy), i32,
                                             ctypes.POINTER(dc_gumbel), vp, vp, vp, vp, vp, vp, vp,
                                             vp, sz, vp]
        L.dc_decode_sample_evict.restype = ctypes.c_int
        L.dc_score_evict_units.argtypes = [ctypes.POINTER(dc_dims), ctypes.POINTER(dc_kv),
                                           ctypes.POINTER(dc_feat), ctypes.POINTER(dc_policy), vp,
                                           i32, ctypes.POINTER(dc_gumbel), vp, vp, vp, vp, sz, vp]
        L.dc_score_evict_units.restype = ctypes.c_int
        L.dc_decode_evict_units.argtypes = [ctypes.POINTER(dc_dims), ctypes.POINTER(dc_kv),
                                            ctypes.POINTER(dc_feat), ctypes.POINTER(dc_policy),
                                            vp, i32, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.dc_decode_evict_units.restype = ctypes.c_int
        L.dc_subset_log_prob.argtypes = [i32, i32, i32, ctypes.c_float, vp, vp, vp, vp, vp, sz, vp]
        L.dc_subset_log_prob.restype = ctypes.c_int
        L.dc_subset_log_prob_workspace_bytes.argtypes = [i32, i32, i32]
        L.dc_subset_log_prob_workspace_bytes.restype = sz
        L.dc_kl_reward.argtypes = [i32, i32, i32, vp, vp, vp, vp, vp, sz, vp]
        L.dc_kl_reward.restype = ctypes.c_int
        L.dc_kl_pack_lm_head.argtypes = [i32, i32, vp, vp, vp]
        L.dc_kl_pack_lm_head.restype = ctypes.c_int
        L.dc_kl_reward_packed.argtypes = [i32, i32, i32, vp, vp, vp, vp, vp, sz, vp]
        L.dc_kl_reward_packed.restype = ctypes.c_int
        L.dc_kl_reward_static.argtypes = [i32, i32, i32, vp, vp, vp, vp, vp]
        L.dc_kl_reward_static.restype = ctypes.c_int
        L.dc_reinforce_terms.argtypes = [i32, i32, ctypes.POINTER(dc_reinforce_cfg), vp, vp, vp,
                                         vp, vp, vp, vp, vp, vp]
        L.dc_reinforce_terms.restype = ctypes.c_int
        L.dc_global_alpha.argtypes = [ctypes.POINTER(dc_dims), ctypes.POINTER(dc_kv),
                                      ctypes.POINTER(dc_feat), vp, sz, vp]
        L.dc_global_alpha.restype = ctypes.c_int
        L.dc_global_alpha_workspace_bytes.argtypes = [ctypes.POINTER(dc_dims), i32]
        L.dc_global_alpha_workspace_bytes.restype = sz
        L.dc_dynamic_budget.argtypes = [ctypes.c_float, i32, i32]
        L.dc_dynamic_budget.restype = i32
        L.dc_status_str.argtypes = [ctypes.c_int]
        L.dc_status_str.restype = ctypes.c_char_p
        _lib = L
    return _lib


class DCError(RuntimeError):
    def __init__(self, status: int):
        self.status = status
        super().__init__(dc_status_str(status))


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _check(st: int) -> None:
    if st != 0:
        raise DCError(st)


def _ref(x):
    return None if x is None else ctypes.byref(x)


def dc_status_str(status: int) -> str:
    return lib().dc_status_str(status).decode()


def dc_workspace_bytes(dims: dc_dims, max_len: int, kl_rows: int = 0, kl_vocab: int = 0) -> int:
    return int(lib().dc_workspace_bytes(ctypes.byref(dims), max_len, kl_rows, kl_vocab))


def dc_feat_init(dims, kv, feat, first_pos: int, stream=None) -> None:
    _check(lib().dc_feat_init(ctypes.byref(dims), ctypes.byref(kv), ctypes.byref(feat),
                              first_pos, stream))


def dc_decode_step(dims, kv, feat, q, k_new, v_new, out, ws=None, ws_bytes: int = 0,
                   stream=None) -> None:
    _check(lib().dc_decode_step(ctypes.byref(dims), ctypes.byref(kv), _ref(feat), _ptr(q),
                                _ptr(k_new), _ptr(v_new), _ptr(out), _ptr(ws), ws_bytes, stream))


def dc_score_evict(dims, kv, feat, policy, budget: int, scores_out=None, kept_out=None,
                   ws=None, ws_bytes: int = 0, stream=None) -> None:
    _check(lib().dc_score_evict(ctypes.byref(dims), ctypes.byref(kv), _ref(feat),
                                _ref(policy), budget, _ptr(scores_out), _ptr(kept_out),
                                _ptr(ws), ws_bytes, stream))


def dc_decode_evict(dims, kv, feat, policy, budget: int, q, k_new, v_new, out, scores_out=None,
                    kept_out=None, ws=None, ws_bytes: int = 0, stream=None) -> None:
    _check(lib().dc_decode_evict(ctypes.byref(dims), ctypes.byref(kv), _ref(feat), _ref(policy),
                                 budget, _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(out),
                                 _ptr(scores_out), _ptr(kept_out), _ptr(ws), ws_bytes, stream))


def dc_global_alpha(dims, kv, feat, ws=None, ws_bytes: int = 0, stream=None) -> None:
    _check(lib().dc_global_alpha(ctypes.byref(dims), ctypes.byref(kv), ctypes.byref(feat),
                                 _ptr(ws), ws_bytes, stream))


def dc_global_alpha_workspace_bytes(dims, positions: int) -> int:
    return int(lib().dc_global_alpha_workspace_bytes(ctypes.byref(dims), positions))


def dc_kl_reward(rows: int, hidden: int, vocab: int, h_full, h_comp, w_lm, kl_out, ws=None,
                 ws_bytes: int = 0, stream=None) -> None:
    _check(lib().dc_kl_reward(rows, hidden, vocab, _ptr(h_full), _ptr(h_comp), _ptr(w_lm),
                              _ptr(kl_out), _ptr(ws), ws_bytes, stream))


def dc_kl_pack_lm_head(hidden: int, vocab: int, w_lm, w_packed, stream=None) -> None:
    _check(lib().dc_kl_pack_lm_head(hidden, vocab, _ptr(w_lm), _ptr(w_packed), stream))


def dc_kl_reward_packed(rows: int, hidden: int, vocab: int, h_full, h_comp, w_packed, kl_out,
                        ws=None, ws_bytes: int = 0, stream=None) -> None:
    _check(lib().dc_kl_reward_packed(rows, hidden, vocab, _ptr(h_full), _ptr(h_comp),
                                     _ptr(w_packed), _ptr(kl_out), _ptr(ws), ws_bytes, stream))


def dc_kl_reward_static(rows: int, hidden: int, vocab: int, h_full, h_comp, w_lm, kl_out,
                        stream=None) -> None:
    _check(lib().dc_kl_reward_static(rows, hidden, vocab, _ptr(h_full), _ptr(h_comp),
                                     _ptr(w_lm), _ptr(kl_out), stream))


def dc_sample_evict(dims, kv, feat, policy, budget: int, gumbel, scores_out=None, kept_out=None,
                    logp_out=None, ws=None, ws_bytes: int = 0, stream=None) -> None:
    _check(lib().dc_sample_evict(ctypes.byref(dims), ctypes.byref(kv), _ref(feat), _ref(policy),
                                 budget, _ref(gumbel), _ptr(scores_out), _ptr(kept_out),
                                 _ptr(logp_out), _ptr(ws), ws_bytes, stream))


def dc_subset_log_prob(units: int, length: int, budget: int, tau: float, scores, kept=None,
                       logz_out=None, logp_out=None, ws=None, ws_bytes: int = 0,
                       stream=None) -> None:
    _check(lib().dc_subset_log_prob(units, length, budget, tau, _ptr(scores), _ptr(kept),
                                    _ptr(logz_out), _ptr(logp_out), _ptr(ws), ws_bytes, stream))


def dc_subset_log_prob_workspace_bytes(units: int, length: int, budget: int) -> int:
    return int(lib().dc_subset_log_prob_workspace_bytes(units, length, budget))


def dc_reinforce_terms(steps: int, rollouts: int, cfg, rewards, logp, ema, returns_out,
                       baseline_out=None, adv_out=None, weight_out=None, stats_out=None,
                       stream=None) -> None:
    _check(lib().dc_reinforce_terms(steps, rollouts, ctypes.byref(cfg), _ptr(rewards), _ptr(logp),
                                    _ptr(ema), _ptr(returns_out), _ptr(baseline_out),
                                    _ptr(adv_out), _ptr(weight_out), _ptr(stats_out), stream))


def dc_dynamic_budget(ratio: float, seq_len: int, b_min: int = 32) -> int:
    return int(lib().dc_dynamic_budget(ratio, seq_len, b_min))


def dc_decode_sample_evict(dims, kv, feat, policy, budget: int, gumbel, q, k_new, v_new, out,
                           scores_out=None, kept_out=None, logp_out=None, ws=None,
                           ws_bytes: int = 0, stream=None) -> None:
    _check(lib().dc_decode_sample_evict(ctypes.byref(dims), ctypes.byref(kv), _ref(feat),
                                        _ref(policy), budget, _ref(gumbel), _ptr(q), _ptr(k_new),
                                        _ptr(v_new), _ptr(out), _ptr(scores_out), _ptr(kept_out),
                                        _ptr(logp_out), _ptr(ws), ws_bytes, stream))


def dc_decode_evict_units(dims, kv, feat, policy, budgets, max_budget: int, q, k_new, v_new, out,
                          scores_out=None, kept_out=None, ws=None, ws_bytes: int = 0,
                          stream=None) -> None:
    _check(lib().dc_decode_evict_units(ctypes.byref(dims), ctypes.byref(kv), ctypes.byref(feat),
                                       ctypes.byref(policy), _ptr(budgets), max_budget, _ptr(q),
                                       _ptr(k_new), _ptr(v_new), _ptr(out), _ptr(scores_out),
                                       _ptr(kept_out), _ptr(ws), ws_bytes, stream))


def dc_score_evict_units(dims, kv, feat, policy, budgets, max_budget: int, gumbel=None,
                         scores_out=None, kept_out=None, logp_out=None, ws=None, ws_bytes: int = 0,
                         stream=None) -> None:
    _check(lib().dc_score_evict_units(ctypes.byref(dims), ctypes.byref(kv), _ref(feat), _ref(policy),
                                      _ptr(budgets), max_budget, _ref(gumbel), _ptr(scores_out),
                                      _ptr(kept_out), _ptr(logp_out), _ptr(ws), ws_bytes, stream))
