"""Per-step KL reward (Sec. 3.1.4): R_t = -KL(P_t || P^_t).

Test infrastructure only (see ``oracle/__init__``).

P_t and P^_t are the next-token distributions of the full-cache (teacher) and
the pruned-cache (student) forward passes.  Here each comes from a final hidden
state times the lm head: logits = h W^T with W stored [vocab][hidden]; the
distributions are softmaxes over the whole vocabulary at temperature 1 with
the max-subtraction ("standard numerical stabilization" of Sec. 3.1.4), and

    KL(P || Q) = sum_v P_v (log P_v - log Q_v)      (natural log).

Parity pinned by: KL(P, P) = 0, KL >= 0, invariance to shifting all logits,
the two-symbol closed form, scipy.stats.entropy, and Pinsker's inequality.
"""
from __future__ import annotations

import numpy as np


def log_softmax(z) -> np.ndarray:
    z = np.asarray(z, np.float64)
    m = z.max(axis=-1, keepdims=True)
    return z - (m + np.log(np.exp(z - m).sum(axis=-1, keepdims=True)))


def kl_from_logits(lp_logits, lq_logits) -> np.ndarray:
    lp = log_softmax(lp_logits)
    lq = log_softmax(lq_logits)
    return (np.exp(lp) * (lp - lq)).sum(axis=-1)


def kl_reward(h_full, h_comp, w_lm) -> np.ndarray:
    """KL per row for hidden states [rows][hidden] and W [vocab][hidden]."""
    W = np.asarray(w_lm, np.float64)
    lf = np.asarray(h_full, np.float64) @ W.T
    lc = np.asarray(h_comp, np.float64) @ W.T
    return kl_from_logits(lf, lc)
