"""C-ABI checks that need no GPU: the library loads, exports every entry point
the header declares, and rejects invalid calls on the host before any launch
(status codes and untouched host fields)."""
import ctypes
import os
import re

import pytest

from paper_2608_08878_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "distillcache.h")
FAKE = 0x10000          # a non-NULL pointer that validation failures never dereference

pytestmark = pytest.mark.skipif(not os.path.exists(B.LIB_PATH), reason="library not built")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(dc_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_function():
    names = declared_functions()
    assert set(names) == set(B.EXPORTS), names
    lib = ctypes.CDLL(B.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


def _dims(**kw):
    d = dict(batch=1, n_layers=2, n_q_heads=8, n_kv_heads=2, head_dim=128, capacity=100,
             dtype=B.DC_BF16, ent_window=64, scale=0.0)
    d.update(kw)
    return B.dc_dims(*[d[f] for f, _ in B.dc_dims._fields_])


def _feat(**kw):
    f = B.dc_feat(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 5, 50)
    for k, v in kw.items():
        setattr(f, k, v)
    return f


def _decode(dims, kv, feat, q=FAKE, kn=FAKE, vn=FAKE, out=FAKE, ws=None, wsb=0):
    L = B.lib()
    return L.dc_decode_step(ctypes.byref(dims), ctypes.byref(kv),
                            ctypes.byref(feat) if feat is not None else None, q, kn, vn, out, ws,
                            wsb, None)


def test_status_strings():
    for code, name in B.STATUS.items():
        assert B.dc_status_str(code).startswith(name)
    assert "unknown" in B.dc_status_str(99)


@pytest.mark.parametrize("kw,status", [
    (dict(head_dim=96), 3), (dict(n_q_heads=6, n_kv_heads=4), 2), (dict(n_q_heads=48, n_kv_heads=2), 3),
    (dict(dtype=7), 3), (dict(ent_window=65), 2), (dict(ent_window=-1), 2), (dict(batch=0), 2),
    (dict(scale=-1.0), 2), (dict(scale=float("nan")), 2), (dict(capacity=0), 2)])
def test_decode_rejects_bad_dims(kw, status):
    kv = B.dc_kv(FAKE, FAKE, 10)
    feat = _feat()
    assert _decode(_dims(**kw), kv, feat) == status
    assert kv.len == 10 and feat.step == 5 and feat.next_pos == 50


def test_decode_rejects_bad_state():
    d = _dims()
    assert _decode(d, B.dc_kv(None, FAKE, 10), _feat()) == 1
    assert _decode(d, B.dc_kv(FAKE, FAKE, 10), _feat(), q=None) == 1
    assert _decode(d, B.dc_kv(FAKE, FAKE, 10), _feat(), kn=None) == 1          # k_new without v_new
    assert _decode(d, B.dc_kv(FAKE, FAKE, 10), _feat(alpha=None)) == 1
    assert _decode(d, B.dc_kv(FAKE, FAKE, 10), _feat(qring=None)) == 1         # window needs the ring
    assert _decode(d, B.dc_kv(FAKE, FAKE, 101), _feat()) == 2                  # len > capacity
    assert _decode(d, B.dc_kv(FAKE, FAKE, 100), _feat()) == 4                  # append beyond capacity
    assert _decode(d, B.dc_kv(FAKE, FAKE, 0), _feat(), kn=None, vn=None) == 2  # empty, no append
    big = _dims(capacity=50000)
    kv = B.dc_kv(FAKE, FAKE, 40000)                                            # chunked path needs scratch
    assert _decode(big, kv, _feat(), ws=None) == 6
    assert _decode(big, kv, _feat(), ws=FAKE, wsb=10) == 6
    assert kv.len == 40000


def test_score_evict_rejects_bad_arguments():
    L = B.lib()
    d = _dims()
    params = ctypes.c_void_p(FAKE)

    def call(budget=10, kv=None, feat=None, pol=None, ws=None, wsb=0):
        kv = kv or B.dc_kv(FAKE, FAKE, 50)
        feat = feat or _feat()
        pol = pol or B.dc_policy(4, 1, (ctypes.c_int32 * 2)(32, 0), FAKE)
        return L.dc_score_evict(ctypes.byref(d), ctypes.byref(kv), ctypes.byref(feat),
                                ctypes.byref(pol), budget, None, None, ws, wsb, None)

    assert call(budget=0) == 5
    assert call(budget=-3) == 5
    assert call(pol=B.dc_policy(6, 1, (ctypes.c_int32 * 2)(32, 0), FAKE)) == 3
    assert call(pol=B.dc_policy(3, 1, (ctypes.c_int32 * 2)(32, 0), FAKE)) == 3
    # five inputs need the sigma state
    assert call(pol=B.dc_policy(5, 1, (ctypes.c_int32 * 2)(32, 0), FAKE)) == 1
    assert call(pol=B.dc_policy(4, 3, (ctypes.c_int32 * 2)(32, 32), FAKE)) == 3
    assert call(pol=B.dc_policy(4, 2, (ctypes.c_int32 * 2)(129, 32), FAKE)) == 3
    assert call(pol=B.dc_policy(4, 2, (ctypes.c_int32 * 2)(32, 129), FAKE)) == 3
    assert call(pol=B.dc_policy(4, 1, (ctypes.c_int32 * 2)(32, 0), FAKE, 2)) == 3
    assert call(pol=B.dc_policy(4, 1, (ctypes.c_int32 * 2)(0, 0), FAKE)) == 3
    # extended policies (LayerNorm, five inputs, a 65..128-wide first of two layers)
    # score through row keys in the workspace at every length
    assert call(pol=B.dc_policy(4, 2, (ctypes.c_int32 * 2)(65, 32), FAKE)) == 6
    assert call(pol=B.dc_policy(4, 1, (ctypes.c_int32 * 2)(32, 0), FAKE, 1)) == 6
    assert call(pol=B.dc_policy(5, 2, (ctypes.c_int32 * 2)(128, 128), FAKE, 1),
                feat=_feat(sigma=FAKE)) == 6
    assert call(pol=B.dc_policy(4, 1, (ctypes.c_int32 * 2)(32, 0), None)) == 1
    assert call(kv=B.dc_kv(FAKE, FAKE, 0)) == 2
    assert call(feat=_feat(vnorm=None)) == 1
    big = _dims(capacity=60000)
    kv = B.dc_kv(FAKE, FAKE, 41000)
    assert L.dc_score_evict(ctypes.byref(big), ctypes.byref(kv), ctypes.byref(_feat()),
                            ctypes.byref(B.dc_policy(4, 1, (ctypes.c_int32 * 2)(32, 0), FAKE)),
                            10, None, None, None, 0, None) == 3              # beyond 40960 rows
    kv = B.dc_kv(FAKE, FAKE, 9000)                                            # long cache: key scratch
    assert L.dc_score_evict(ctypes.byref(big), ctypes.byref(kv), ctypes.byref(_feat()),
                            ctypes.byref(B.dc_policy(4, 1, (ctypes.c_int32 * 2)(32, 0), FAKE)),
                            10, None, None, None, 0, None) == 6
    assert kv.len == 9000


def test_kl_reward_rejects_bad_arguments():
    L = B.lib()
    assert L.dc_kl_reward(8, 4096, 32768, None, FAKE, FAKE, FAKE, FAKE, 1 << 30, None) == 1
    assert L.dc_kl_reward(0, 4096, 32768, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 30, None) == 2
    assert L.dc_kl_reward(B.KL_MAX_ROWS + 1, 4096, 32768, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 40, None) == 3
    assert L.dc_kl_reward(8, 4000, 32768, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 30, None) == 3
    assert L.dc_kl_reward(8, 4096, 32700, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 30, None) == 3
    assert L.dc_kl_reward(8, 4096, 32768, FAKE, FAKE, FAKE, FAKE, FAKE, 16, None) == 6


def test_kl_pack_and_packed_reward_reject_bad_arguments():
    L = B.lib()
    n = 4096 * 32768 * 2
    assert L.dc_kl_pack_lm_head(4096, 32768, None, FAKE, None) == 1
    assert L.dc_kl_pack_lm_head(4096, 32768, FAKE, None, None) == 1
    assert L.dc_kl_pack_lm_head(0, 32768, FAKE, FAKE + 2 * n, None) == 2
    assert L.dc_kl_pack_lm_head(4000, 32768, FAKE, FAKE + 2 * n, None) == 3
    assert L.dc_kl_pack_lm_head(4096, 32700, FAKE, FAKE + 2 * n, None) == 3
    # in place, or overlapping by one element either way
    assert L.dc_kl_pack_lm_head(4096, 32768, FAKE, FAKE, None) == 3
    assert L.dc_kl_pack_lm_head(4096, 32768, FAKE, FAKE + n - 2, None) == 3
    assert L.dc_kl_pack_lm_head(4096, 32768, FAKE + n - 2, FAKE, None) == 3
    assert L.dc_kl_reward_packed(8, 4096, 32768, None, FAKE, FAKE, FAKE, FAKE, 1 << 30, None) == 1
    assert L.dc_kl_reward_packed(0, 4096, 32768, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 30, None) == 2
    assert L.dc_kl_reward_packed(8, 4000, 32768, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 30, None) == 3
    assert L.dc_kl_reward_packed(B.KL_MAX_ROWS + 1, 4096, 64, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 40,
                                 None) == 3
    assert L.dc_kl_reward_packed(8, 4096, 32768, FAKE, FAKE, FAKE, FAKE, FAKE, 16, None) == 6


def test_kl_reward_static_rejects_bad_arguments_before_any_device_work():
    L = B.lib()
    assert L.dc_kl_reward_static(8, 4096, 32768, None, FAKE, FAKE, FAKE, None) == 1
    assert L.dc_kl_reward_static(8, 4096, 32768, FAKE, FAKE, FAKE, None, None) == 1
    assert L.dc_kl_reward_static(0, 4096, 32768, FAKE, FAKE, FAKE, FAKE, None) == 2
    assert L.dc_kl_reward_static(8, 4000, 32768, FAKE, FAKE, FAKE, FAKE, None) == 3
    assert L.dc_kl_reward_static(B.KL_MAX_ROWS + 1, 4096, 64, FAKE, FAKE, FAKE, FAKE, None) == 3
    # one pair past the fixed scratch (rows * vocab / 64 > 524288): DC_ERR_SCRATCH
    assert L.dc_kl_reward_static(1025, 4096, 32768, FAKE, FAKE, FAKE, FAKE, None) == 9
    assert L.dc_kl_reward_static(1, 128, 64 * (B.KL_STATIC_MAX_PAIRS + 1), FAKE, FAKE, FAKE,
                                 FAKE, None) == 9
    assert "scratch" in B.dc_status_str(9)


def test_workspace_sizes():
    d = _dims(batch=16, n_layers=32, n_q_heads=32, n_kv_heads=8, capacity=16385)
    assert B.dc_workspace_bytes(d, 0, 0, 0) == 0
    big = B.dc_workspace_bytes(d, 16385, 0, 0)
    assert big >= 4096 * 16385 * 7 * 4            # per-row logits, retired sums, norms
    assert B.dc_workspace_bytes(d, 4097, 0, 0) < big
    assert B.dc_workspace_bytes(d, 0, 8, 32768) >= 8 * 512 * 16
    assert B.dc_workspace_bytes(_dims(head_dim=96), 100, 0, 0) == 0


@pytest.mark.parametrize("kv_heads,dtype", [(1, "bf16"), (2, "bf16"), (8, "bf16"), (64, "bf16"),
                                            (127, "bf16"), (128, "bf16"), (2, "f32")])
def test_workspace_never_shrinks_as_the_length_grows(kv_heads, dtype):
    """A workspace sized for max_len serves every shorter cache.  Few bf16 units
    cut their rows into chunks that grow with the length, so the number of
    chunks alone is not monotone in the length; the bound must be."""
    d = _dims(batch=1, n_layers=1, n_q_heads=4 * kv_heads, n_kv_heads=kv_heads, capacity=40960,
              dtype=B.DC_BF16 if dtype == "bf16" else B.DC_F32)
    lengths = sorted(set(list(range(1, 9000, 97)) + [4096, 4097, 4098, 8192, 8193, 16384, 16385,
                                                      16513, 32768, 32769, 40960]))
    sizes = [B.dc_workspace_bytes(d, L, 0, 0) for L in lengths]
    assert all(a <= b for a, b in zip(sizes, sizes[1:])), [
        (L, a, b) for L, a, b in zip(lengths[1:], sizes, sizes[1:]) if a > b][:3]


def _logprob(units=4, length=100, budget=10, tau=1.0, scores=FAKE, kept=FAKE, logz=FAKE,
             logp=FAKE, ws=None, wsb=0):
    return B.lib().dc_subset_log_prob(units, length, budget, tau, scores, kept, logz, logp, ws,
                                      wsb, None)


@pytest.mark.parametrize("kw,status", [
    (dict(scores=None), 1), (dict(kept=None), 1), (dict(units=0), 2), (dict(length=0), 2),
    (dict(budget=0), 5), (dict(tau=0.0), 8), (dict(tau=-1.0), 8), (dict(tau=float("nan")), 8),
    (dict(tau=float("inf")), 8), (dict(length=40961), 3), (dict(units=(1 << 24) + 1), 3),
    # K = min(B, L - B) = 5000 > 4096 needs the band workspace
    (dict(length=10000, budget=5000), 6), (dict(length=10000, budget=5000, ws=FAKE, wsb=16), 6)])
def test_subset_log_prob_rejects_bad_arguments(kw, status):
    assert _logprob(**kw) == status


def test_subset_log_prob_workspace_sizes():
    W = B.dc_subset_log_prob_workspace_bytes
    assert W(4, 8192, 4096) == 0                 # K = 4096 fits one band
    assert W(4, 10000, 5000) == 4 * 10000 * 8    # K = 5000: one float and one int per row
    assert W(4, 10000, 9000) == 0                # K = 1000 through the complement
    assert W(0, 100, 10) == 0 and W(4, 0, 10) == 0 and W(4, 100, 0) == 0
    assert W(1, 40961, 20000) == 0


def test_sample_evict_rejects_bad_arguments():
    L = B.lib()
    pol = B.dc_policy(4, 1, (ctypes.c_int32 * 2)(32, 0), FAKE)
    for tau, want in [(0.0, 8), (float("nan"), 8), (-2.0, 8), (float("inf"), 8)]:
        kv = B.dc_kv(FAKE, FAKE, 10)
        feat = _feat()
        g = B.make_gumbel(tau, 1, 0)
        st = L.dc_sample_evict(ctypes.byref(_dims()), ctypes.byref(kv), ctypes.byref(feat),
                               ctypes.byref(pol), 5, ctypes.byref(g), FAKE, FAKE, FAKE, None, 0, None)
        assert st == want and kv.len == 10
    kv = B.dc_kv(FAKE, FAKE, 10)
    g = B.make_gumbel(1.0, 1, 0)
    # no gumbel struct; logp_out without scores_out / kept_out
    assert L.dc_sample_evict(ctypes.byref(_dims()), ctypes.byref(kv), ctypes.byref(_feat()),
                             ctypes.byref(pol), 5, None, FAKE, FAKE, FAKE, None, 0, None) == 1
    assert L.dc_sample_evict(ctypes.byref(_dims()), ctypes.byref(kv), ctypes.byref(_feat()),
                             ctypes.byref(pol), 5, ctypes.byref(g), None, FAKE, FAKE, None, 0, None) == 1
    assert L.dc_sample_evict(ctypes.byref(_dims()), ctypes.byref(kv), ctypes.byref(_feat()),
                             ctypes.byref(pol), 5, ctypes.byref(g), FAKE, None, FAKE, None, 0, None) == 1
    assert L.dc_sample_evict(ctypes.byref(_dims()), ctypes.byref(kv), ctypes.byref(_feat()),
                             ctypes.byref(pol), 0, ctypes.byref(g), FAKE, FAKE, FAKE, None, 0, None) == 5
    assert kv.len == 10


def test_reinforce_terms_rejects_bad_arguments():
    L = B.lib()
    ok = B.dc_reinforce_cfg(0.99, 0.01, 0.9)

    def call(steps=64, rollouts=8, cfg=ok, r=FAKE, lp=FAKE, ema=FAKE, ret=FAKE):
        return L.dc_reinforce_terms(steps, rollouts, None if cfg is None else ctypes.byref(cfg), r,
                                    lp, ema, ret, None, None, None, None, None)

    assert call(cfg=None) == 1 and call(r=None) == 1 and call(lp=None) == 1
    assert call(ema=None) == 1 and call(ret=None) == 1
    assert call(steps=0) == 2 and call(rollouts=0) == 2
    assert call(steps=1 << 14, rollouts=1 << 13) == 3
    for cfg in (B.dc_reinforce_cfg(1.5, 0.01, 0.9), B.dc_reinforce_cfg(-0.1, 0.01, 0.9),
                B.dc_reinforce_cfg(float("nan"), 0.01, 0.9), B.dc_reinforce_cfg(0.99, float("inf"), 0.9),
                B.dc_reinforce_cfg(0.99, 0.01, 1.0), B.dc_reinforce_cfg(0.99, 0.01, -0.5)):
        assert call(cfg=cfg) == 8


def test_dynamic_budget_matches_the_oracle():
    from oracle import select as osel
    for r in (0.25, 0.125, 0.5, 0.1, 1.0, 0.3333):
        for T in (0, 1, 31, 127, 128, 129, 1025, 4097, 8193, 16385, 40960, 123457):
            assert B.dc_dynamic_budget(r, T, 32) == osel.dynamic_budget(r, T, 32), (r, T)
    assert B.dc_dynamic_budget(0.0, 100, 32) == -1
    assert B.dc_dynamic_budget(1.5, 100, 32) == -1
    assert B.dc_dynamic_budget(float("nan"), 100, 32) == -1
    assert B.dc_dynamic_budget(0.25, -1, 32) == -1
    assert B.dc_dynamic_budget(0.25, 100, 0) == -1


def test_score_evict_units_rejects_bad_arguments():
    L = B.lib()
    pol = B.dc_policy(4, 1, (ctypes.c_int32 * 2)(32, 0), FAKE)
    g = B.make_gumbel(1.0, 1, 0)

    def call(kv=None, budgets=FAKE, maxb=64, gum=None, sc=FAKE, kp=FAKE, lp=None, ws=None, wsb=0,
             dims=None):
        kv = kv or B.dc_kv(FAKE, FAKE, 50, FAKE)
        return L.dc_score_evict_units(ctypes.byref(dims or _dims()), ctypes.byref(kv),
                                      ctypes.byref(_feat()), ctypes.byref(pol), budgets, maxb,
                                      None if gum is None else ctypes.byref(gum), sc, kp, lp, ws, wsb,
                                      None)

    assert call(budgets=None) == 1
    assert call(kv=B.dc_kv(FAKE, FAKE, 50, None)) == 1          # per-unit lengths are required
    assert call(lp=FAKE) == 1                                   # log pi needs the gumbel draw
    assert call(gum=g, lp=FAKE, kp=None) == 1
    assert call(maxb=0) == 5
    assert call() == 6                                          # row keys need the workspace
    assert call(dims=_dims(dtype=B.DC_F32)) == 3                # ragged caches are bf16
    kv = B.dc_kv(FAKE, FAKE, 50, FAKE)
    assert call(kv=kv, gum=B.make_gumbel(0.0, 1, 0), ws=FAKE, wsb=1 << 40) == 8
    assert kv.len == 50


def test_decode_evict_units_rejects_bad_arguments_and_leaves_host_fields():
    L = B.lib()
    pol = B.dc_policy(4, 1, (ctypes.c_int32 * 2)(32, 0), FAKE)

    def call(kv, feat=None, budgets=FAKE, maxb=64, kn=FAKE, vn=FAKE, ws=None, wsb=0, dims=None):
        return L.dc_decode_evict_units(ctypes.byref(dims or _dims()), ctypes.byref(kv),
                                       ctypes.byref(feat or _feat()), ctypes.byref(pol), budgets,
                                       maxb, FAKE, kn, vn, FAKE, FAKE, FAKE, ws, wsb, None)

    kv = B.dc_kv(FAKE, FAKE, 50, FAKE)
    feat = _feat()
    assert call(kv, feat, budgets=None) == 1
    assert call(B.dc_kv(FAKE, FAKE, 50, None), feat) == 1      # per-unit lengths are required
    assert call(kv, feat, kn=None, vn=None) == 1                # a step appends
    assert call(kv, feat, maxb=0, ws=FAKE, wsb=1 << 40) == 5
    assert call(kv, feat) == 6                                  # the chunked decode needs the workspace
    assert call(kv, feat, dims=_dims(dtype=B.DC_F32)) == 3      # ragged caches are bf16
    assert call(B.dc_kv(FAKE, FAKE, 100, FAKE), feat, ws=FAKE, wsb=1 << 40) == 4   # capacity
    assert kv.len == 50 and feat.step == 5 and feat.next_pos == 50


def test_ragged_decode_needs_bf16_and_moves_fit_on_chip():
    L = B.lib()
    kv = B.dc_kv(FAKE, FAKE, 10, FAKE)
    feat = _feat()
    assert _decode(_dims(dtype=B.DC_F32), kv, feat) == 3
    assert kv.len == 10
    # a compaction that would move more than 16384 rows is refused (the move list is in LDS)
    big = _dims(capacity=40960, n_layers=1)
    kvb = B.dc_kv(FAKE, FAKE, 40000, None)
    pol = B.dc_policy(4, 1, (ctypes.c_int32 * 2)(32, 0), FAKE)
    assert L.dc_score_evict(ctypes.byref(big), ctypes.byref(kvb), ctypes.byref(_feat()),
                            ctypes.byref(pol), 20000, None, None, FAKE, 1 << 40, None) == 3
    assert kvb.len == 40000


def test_global_alpha_rejects_bad_arguments():
    L = B.lib()
    dims = _dims()
    kv = B.dc_kv(FAKE, FAKE, 50)

    def call(d=dims, k=kv, f=None, ws=FAKE, wsb=1 << 30):
        f = f if f is not None else _feat(alpha_recent=1)
        return L.dc_global_alpha(ctypes.byref(d), ctypes.byref(k) if k is not None else None,
                                 ctypes.byref(f), ws, wsb, None)

    assert call(k=None) == 1
    assert call(f=_feat(alpha=None, alpha_recent=1)) == 1
    assert call(f=_feat(pos=None, alpha_recent=1)) == 1
    assert call(k=B.dc_kv(FAKE, FAKE, 0)) == 2                       # no rows
    assert call(k=B.dc_kv(FAKE, FAKE, 101)) == 2                     # beyond the capacity
    assert call(f=_feat(next_pos=0, alpha_recent=1)) == 2
    assert call(f=_feat()) == 3                                      # alpha accumulates: not this mode
    assert call(d=_dims(n_layers=300, n_kv_heads=8, n_q_heads=8)) == 3   # 2400 units per sequence
    need = B.dc_global_alpha_workspace_bytes(dims, 50)
    assert need >= 1 * 50 * 8 and need % 256 == 0
    assert call(wsb=need - 1) == 6
    assert call(ws=None) == 6
    assert B.dc_global_alpha_workspace_bytes(_dims(batch=3), 1000) >= 3 * 1000 * 8
    assert B.dc_global_alpha_workspace_bytes(dims, 0) == 0


def test_decode_rejects_an_alpha_mode_outside_its_two_values():
    dims = _dims()
    kv = B.dc_kv(FAKE, FAKE, 50)
    assert _decode(dims, kv, _feat(alpha_recent=2), ws=FAKE, wsb=1 << 40) == 8
    assert _decode(dims, kv, _feat(alpha_recent=-1), ws=FAKE, wsb=1 << 40) == 8
