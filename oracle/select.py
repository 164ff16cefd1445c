"""Deterministic top-B selection (argtop_B of Algorithm 1; Sec. 3.1.2 "At
inference, the policy selects the top-B tokens deterministically").

Test infrastructure only (see ``oracle/__init__``).

Order used (the paper does not fix ties): token i ranks above token k when
s_i > s_k, or s_i == s_k and i is the earlier token (smaller absolute
position).  -0.0 equals +0.0.  A NaN score ranks below every number (and NaNs
rank among themselves by position).  If B >= L every token is kept.

Dynamic budget (App. D): B_t = max(floor(r T_t), B_min), with T_t read as the
number of tokens seen (the paper's |C_t| would collapse the budget
geometrically once eviction starts; reading recorded with the design notes).

Parity pinned by: exhaustive enumeration of all size-B subsets on small L
(the kept set maximises the score sum, ties resolved toward earlier tokens),
|kept| = min(B, L), min kept score >= max evicted score, and all-equal scores.
"""
from __future__ import annotations

import numpy as np


def ranking(scores, positions) -> np.ndarray:
    """Row indices sorted from best to worst under the order above."""
    s = np.asarray(scores, np.float64)
    p = np.asarray(positions, np.int64)
    nan = np.isnan(s)
    key = np.where(nan, 0.0, s) + 0.0          # -0.0 -> +0.0
    # np.lexsort sorts by the last key first: NaN flag, then -score, then position
    return np.lexsort((p, -key, nan.astype(np.int8)))


def top_budget(scores, positions, budget: int) -> np.ndarray:
    """Indices (into the current rows) of the kept tokens, in ascending row order."""
    n = len(scores)
    if budget >= n:
        return np.arange(n)
    if budget < 1:
        raise ValueError("budget must be >= 1")
    order = ranking(scores, positions)
    return np.sort(order[:budget])


def dynamic_budget(ratio: float, seq_len: int, b_min: int = 32) -> int:
    """max(floor(ratio * seq_len), b_min); the ratio is taken as its float32 value."""
    r = float(np.float32(ratio))
    if not (0.0 < r <= 1.0) or seq_len < 0 or b_min < 1:
        raise ValueError("ratio in (0, 1], seq_len >= 0, b_min >= 1")
    return max(int(np.floor(r * seq_len)), b_min)
