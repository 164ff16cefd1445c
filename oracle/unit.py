"""One unit's cache and feature state stepped through the decode step.

Test infrastructure only (see ``oracle/__init__``).

A unit is one (batch, layer, KV head) cache.  Algorithm 1 orders one decode
step as: the forward pass appends the new key/value pair and attends over the
cache that now contains it; features are built from that step's attention and
the cache; the policy scores every cached token; the top-B tokens are kept and
the pruned cache serves the *next* step.  Sec. 3.1.3 adds the teacher cache
(never pruned, same appends) whose distribution defines the reward.

``StudentState`` holds, per cached row (in slot order: ascending position until
the first eviction, then the hole-filling order of ``compact``): key and
value rows, absolute position p, alpha, the windowed-entropy history, and —
for the add/retire cross-check — running N/Z sums plus the per-step records
(q, m, l, H, largest position present) of the last w steps.
``TeacherState`` holds only keys, values and positions.

Parity pinned by the module pins of ``attention``, ``features``, ``policy`` and
``select`` plus the end-to-end pins in tests/test_oracle_unit.py (budget >= L
reproduces the teacher exactly; kept rows carry their bytes and state; the
hand-worked golden example in tests/golden/).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from . import attention, compact, features, policy, select


@dataclass
class StepRecord:
    q: np.ndarray
    m: np.ndarray
    l: np.ndarray
    H: np.ndarray
    pmax: int          # largest absolute position present at that step (T - 1)


@dataclass
class StudentState:
    K: np.ndarray
    V: np.ndarray
    pos: np.ndarray
    alpha: np.ndarray
    hist: features.WindowHistory
    N: np.ndarray                  # running sums for the add/retire cross-check
    Z: np.ndarray
    step: int
    next_pos: int
    window: int
    G: int
    scale: float
    records: dict = field(default_factory=dict)
    sigma: np.ndarray | None = None    # per-row head variance of the last step's attention
    alpha_recent: bool = False         # alpha = the last step's mass only (not accumulated)

    @property
    def L(self) -> int:
        return self.K.shape[0]


@dataclass
class TeacherState:
    K: np.ndarray
    V: np.ndarray
    pos: np.ndarray
    next_pos: int
    scale: float


def new_student(K, V, positions, *, G: int, scale: float, window: int = 64,
                next_pos: int | None = None, alpha_recent: bool = False) -> StudentState:
    """State for a cache whose rows carry no attention history yet (features zero)."""
    K = np.asarray(K, np.float64)
    V = np.asarray(V, np.float64)
    pos = np.asarray(positions, np.int64)
    L = K.shape[0]
    return StudentState(K=K.copy(), V=V.copy(), pos=pos.copy(), alpha=np.zeros(L),
                        hist=features.WindowHistory(L, window), N=np.zeros(L), Z=np.zeros(L),
                        step=0, next_pos=int(pos.max()) + 1 if next_pos is None else next_pos,
                        window=window, G=G, scale=scale, sigma=np.zeros(L),
                        alpha_recent=alpha_recent)


def new_teacher(K, V, positions, *, scale: float, next_pos: int | None = None) -> TeacherState:
    pos = np.asarray(positions, np.int64)
    return TeacherState(K=np.asarray(K, np.float64).copy(), V=np.asarray(V, np.float64).copy(),
                        pos=pos.copy(), next_pos=int(pos.max()) + 1 if next_pos is None else next_pos,
                        scale=scale)


def _append(st, k_new, v_new):
    st.K = np.vstack([st.K, np.asarray(k_new, np.float64)[None, :]])
    st.V = np.vstack([st.V, np.asarray(v_new, np.float64)[None, :]])
    st.pos = np.append(st.pos, st.next_pos)
    st.next_pos += 1


def teacher_step(st: TeacherState, q, k_new=None, v_new=None) -> attention.Attention:
    """Plain attention over the never-pruned cache (after the append)."""
    if k_new is not None:
        _append(st, k_new, v_new)
    return attention.attend(q, st.K, st.V, st.scale)


def decode_step(st: StudentState, q, k_new=None, v_new=None) -> attention.Attention:
    """Append (optional), attend, and accumulate alpha / the entropy window."""
    if k_new is not None:
        _append(st, k_new, v_new)
        st.alpha = np.append(st.alpha, 0.0)
        st.hist.append_rows(1)
        st.N = np.append(st.N, 0.0)
        st.Z = np.append(st.Z, 0.0)
    att = attention.attend(q, st.K, st.V, st.scale)
    cz, cn = features.step_contributions(att.a, att.H)
    st.sigma = features.head_variance(att.a)
    t = st.step
    st.alpha = (0.0 if st.alpha_recent else st.alpha) + cz / st.G
    st.hist.record(t, cz, cn)
    # add/retire form of the same window (cross-check only)
    if st.window > 0 and t >= st.window:
        rec = st.records.pop(t - st.window)
        present = st.pos <= rec.pmax
        rz, rn = features.retire_contribution(rec.q, rec.m, rec.l, rec.H, st.K[present], st.scale)
        st.Z[present] -= rz
        st.N[present] -= rn
    st.Z = st.Z + cz
    st.N = st.N + cn
    if st.window > 0:
        st.records[t] = StepRecord(q=np.asarray(q, np.float64).copy(), m=att.m.copy(),
                                   l=att.l.copy(), H=att.H.copy(), pmax=st.next_pos - 1)
    st.step += 1
    return att


def feature_matrix(st: StudentState, n_in: int = 4) -> np.ndarray:
    Z, N = st.hist.sums()
    if n_in == 5:
        return features.feature_matrix5(st.alpha, st.V, st.sigma, Z, N, st.pos, st.next_pos)
    return features.feature_matrix(st.alpha, st.V, Z, N, st.pos, st.next_pos)


def scores(st: StudentState, params, hidden, n_in: int = 4, layer_norm: bool = False) -> np.ndarray:
    return policy.scores(params, feature_matrix(st, n_in), hidden, layer_norm=layer_norm)


def evict(st: StudentState, scores_, budget: int) -> np.ndarray:
    """Keep the top-``budget`` rows under ``scores_`` and store them in the
    hole-filling order of ``compact.hole_fill``; returns that slot map (old slot
    of every new slot)."""
    slot_map = compact.hole_fill(select.top_budget(scores_, st.pos, budget), st.L)
    st.K, st.V, st.pos = st.K[slot_map], st.V[slot_map], st.pos[slot_map]
    st.alpha, st.N, st.Z = st.alpha[slot_map], st.N[slot_map], st.Z[slot_map]
    st.sigma = st.sigma[slot_map]
    st.hist.keep_rows(slot_map)
    return slot_map


def score_evict(st: StudentState, params, hidden, budget: int):
    s = scores(st, params, hidden)
    kept = evict(st, s, budget)
    return s, kept
