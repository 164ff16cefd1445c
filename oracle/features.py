"""Per-token eviction features (Sec. 3.1.1, "State Space").

Test infrastructure only (see ``oracle/__init__``).

The paper's state vector is x_i = [alpha_i, ||v_i||_2, sigma_i, H_i, pos_i];
the decode step built here uses the four features without sigma_i, in that
order: x_i = [alpha_i, ||v_i||_2, H_i, pos_i].  Readings of the text:

* alpha_i — attention mass received by token i, averaged over the G query heads
  that share the token's KV head, accumulated over decode steps since the state
  was initialised (the ablation table calls it "cumulative attention").  The
  state definition itself (Sec. 3.1.1) takes the mass of the most recent
  forward pass averaged over all heads and layers: ``alpha_recent`` keeps only
  the step's mass, and ``global_alpha`` averages it over every KV unit of the
  sequence (all layers and KV heads), position by position.
* H_i — for the queries of the last w decode steps (current step included;
  every (step, query head) pair is one query; w = 64):
      Z_i = sum_q a_q(i),  N_i = sum_q a_q(i) H(a_q),  H_i = N_i / Z_i,
  and H_i = 0 when Z_i = 0.  A token absent at some step contributes nothing
  for that step.
* pos_i = p_i / T, p_i the token's 0-based absolute position and T the number
  of tokens seen so far ("normalized sequence position").
* ||v_i||_2 — Euclidean norm of the stored value row.

``WindowHistory`` keeps, for every cached token, its contribution from each of
the last w steps; Z and N are the plain sums over that history.  This is the
definition.  ``retire_contribution`` is the add/retire bookkeeping that a
streaming implementation uses instead (it recomputes the retiring step's
weights from that step's query and softmax statistics); tests assert that the
two agree.

Parity pinned by: per-step sums (sum_i d_alpha_i = 1, sum_i dZ_i = G,
sum_i dN_i = sum_j H_j), H_i lying between the smallest and largest window
entropy, w = 64 versus an unbounded window before step 64, the add/retire form
versus the history form, and a hand-computed two-token example.
"""
from __future__ import annotations

import numpy as np


class WindowHistory:
    """Per-token contributions (sum_j a_{t,j}(i), sum_j a_{t,j}(i) H_{t,j}) of the
    last ``window`` steps; ``window == 0`` keeps an unbounded running sum."""

    def __init__(self, n_rows: int, window: int):
        self.window = window
        cols = max(window, 1)
        self.z = np.zeros((n_rows, cols))
        self.n = np.zeros((n_rows, cols))

    def append_rows(self, k: int):
        cols = self.z.shape[1]
        self.z = np.vstack([self.z, np.zeros((k, cols))])
        self.n = np.vstack([self.n, np.zeros((k, cols))])

    def keep_rows(self, idx):
        self.z = self.z[idx]
        self.n = self.n[idx]

    def record(self, step: int, cz, cn):
        if self.window == 0:
            self.z[:, 0] += cz
            self.n[:, 0] += cn
        else:
            c = step % self.window        # the column of step - window is replaced
            self.z[:, c] = cz
            self.n[:, c] = cn

    def sums(self):
        return self.z.sum(axis=1), self.n.sum(axis=1)


def step_contributions(a, H):
    """cz_i = sum_j a_j(i), cn_i = sum_j a_j(i) H_j for one step's weights a (G, L)."""
    a = np.asarray(a, np.float64)
    return a.sum(axis=0), (a * np.asarray(H, np.float64)[:, None]).sum(axis=0)


def retire_contribution(q_old, m_old, l_old, H_old, K, scale: float):
    """Recompute a past step's (cz, cn) for the current rows K from that step's
    queries (G, d) and softmax statistics m, l (G,), entropies H (G,)."""
    s = scale * (np.asarray(q_old, np.float64) @ np.asarray(K, np.float64).T)
    a = np.exp(s - np.asarray(m_old, np.float64)[:, None]) / np.asarray(l_old, np.float64)[:, None]
    return step_contributions(a, H_old)


def entropy_feature(Z, N) -> np.ndarray:
    Z = np.asarray(Z, np.float64)
    N = np.asarray(N, np.float64)
    out = np.zeros_like(Z)
    nz = Z > 0
    out[nz] = N[nz] / Z[nz]
    return out


def feature_matrix(alpha, V, Z, N, pos, T: int) -> np.ndarray:
    """x = [alpha, ||v||_2, H, pos/T] as an (L, 4) matrix (sigma left out)."""
    vnorm = np.sqrt((np.asarray(V, np.float64) ** 2).sum(axis=1))
    return np.stack([np.asarray(alpha, np.float64), vnorm, entropy_feature(Z, N),
                     np.asarray(pos, np.float64) / float(T)], axis=1)


def head_variance(a) -> np.ndarray:
    """sigma_i (Sec. 3.1.1): the variance over the G query heads of the unit of
    the attention mass token i receives at the step, (1/G) sum_j (a_j(i) - abar(i))^2
    with abar the head mean (population variance; 0 for G = 1).  Reading: taken at
    the current step, like the attention the step's other features come from."""
    a = np.asarray(a, np.float64)
    G = a.shape[0]
    mean = a.sum(axis=0) / G
    return ((a - mean[None, :]) ** 2).sum(axis=0) / G


def global_alpha(alphas, positions, n_units: int):
    """The paper's alpha (Sec. 3.1.1): the attention mass token p received in
    the most recent forward pass, averaged over all heads and layers.  Input:
    for each of the ``n_units`` KV units of one sequence (every layer and KV
    head), its rows' step masses (group means over the unit's G query heads)
    and positions.  Every unit has the same number of query heads, so the mean
    over all heads is the mean over units of the group means; a unit that no
    longer holds p contributes 0 (its heads cannot attend to p).  Returns, per
    unit, that average at each of its rows' positions."""
    total = {}
    for al, ps in zip(alphas, positions):
        for a_i, p_i in zip(np.asarray(al, np.float64), np.asarray(ps, np.int64)):
            total[int(p_i)] = total.get(int(p_i), 0.0) + float(a_i)
    return [np.array([total[int(p_i)] / n_units for p_i in np.asarray(ps, np.int64)], np.float64)
            for ps in positions]


def feature_matrix5(alpha, V, sigma, Z, N, pos, T: int) -> np.ndarray:
    """x = [alpha, ||v||_2, sigma, H, pos/T] (the paper's five features, in its order)."""
    x4 = feature_matrix(alpha, V, Z, N, pos, T)
    return np.stack([x4[:, 0], x4[:, 1], np.asarray(sigma, np.float64), x4[:, 2], x4[:, 3]], axis=1)
