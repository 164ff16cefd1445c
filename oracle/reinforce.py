"""Rollout reward math of the REINFORCE update (Sec. 3.2, policy optimisation).

Test infrastructure only (see ``oracle/__init__``).  Binary64, plain loops.

Inputs of one update: per-step rewards R[t][k] = -KL_t (Sec. 3.1.4) and the
log-probabilities log pi(a_t | s_t) of the sampled kept sets (App. C) for
t = 0..T-1 decode steps and k = 0..K-1 sampled rollouts (the batch).

* Discounted return:  G[t][k] = sum_{tau = t}^{T-1} gamma^(tau - t) R[tau][k].
* Baseline, RLOO (K >= 2): b[t][k] = (sum_{k' != k} G[t][k']) / (K - 1), the
  mean return of the other K - 1 rollouts at the same step.
* Baseline, EMA: a running mean of returns kept across updates,
  e <- d e + (1 - d) mean_{t,k} G[t][k], updated after this update's baseline
  is taken; with a single rollout (K = 1) the baseline is e.
* Advantage A = G - b.
* Entropy surrogate H^[t][k] = -log pi (single-sample estimate).
* Surrogate objective, to be maximised by gradient ascent on the policy
  parameters, J = mean_{t,k} ( log pi * A + beta H^ ), A treated as a
  constant; the loss is -J and its derivative with respect to each
  log-probability is w[t][k] = -(A[t][k] - beta) / (T K).

Readings recorded with the design notes: the leave-one-out baseline averages
the other rollouts' returns (it is subtracted from G_t, so it lives on the
return scale); the paper keeps both an RLOO and an EMA baseline without saying
how they combine, so RLOO is used whenever K >= 2 and the EMA otherwise, and
the EMA is always updated.

Parity pinned by: constant rewards (finite geometric series), gamma = 0
(G = R), gamma = 1 (suffix sums), RLOO advantages summing to zero over the
rollouts of every step, K = 2 (A_0 = G_0 - G_1 = -A_1), the EMA's closed form
over repeated updates, and the loss derivative checked by finite differences.
"""
from __future__ import annotations

import numpy as np


def discounted_returns(rewards, gamma: float) -> np.ndarray:
    R = np.asarray(rewards, np.float64)
    T, K = R.shape
    G = np.zeros((T, K))
    for k in range(K):
        for t in range(T):
            acc, w = 0.0, 1.0
            for tau in range(t, T):
                acc += w * R[tau, k]
                w *= gamma
            G[t, k] = acc
    return G


def rloo_baseline(G) -> np.ndarray:
    G = np.asarray(G, np.float64)
    T, K = G.shape
    if K < 2:
        raise ValueError("RLOO needs at least two rollouts")
    b = np.zeros((T, K))
    for t in range(T):
        for k in range(K):
            b[t, k] = sum(G[t, j] for j in range(K) if j != k) / (K - 1)
    return b


def reinforce_terms(rewards, logp, gamma: float, beta: float, ema: float, ema_decay: float):
    """Returns a dict with returns, baseline, advantage, weight (all [T][K]),
    loss, entropy (mean surrogate) and the updated EMA."""
    R = np.asarray(rewards, np.float64)
    lp = np.asarray(logp, np.float64)
    T, K = R.shape
    G = discounted_returns(R, gamma)
    b = rloo_baseline(G) if K >= 2 else np.full((T, K), float(ema))
    A = G - b
    H = -lp
    n = T * K
    J = sum(lp[t, k] * A[t, k] + beta * H[t, k] for t in range(T) for k in range(K)) / n
    w = -(A - beta) / n
    new_ema = ema_decay * ema + (1.0 - ema_decay) * (G.sum() / n)
    return {"returns": G, "baseline": b, "advantage": A, "weight": w, "loss": -J,
            "entropy": H.sum() / n, "ema": new_ema}
