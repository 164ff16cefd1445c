"""Decode attention over one unit's cache, with per-query entropy.

Test infrastructure only (see ``oracle/__init__``).

Definitions followed:
* logits s_{j,i} = scale * q_j . k_i, with scale = 1/sqrt(d) unless given
  (the paper is silent on the scale; the standard scaled dot product is used);
* a_j = softmax_i(s_j) (the attention distribution a_q of Sec. 3.1.1), taken
  with the usual max subtraction: m_j = max_i s_{j,i},
  l_j = sum_i exp(s_{j,i} - m_j), a_{j,i} = exp(s_{j,i} - m_j) / l_j;
* o_j = sum_i a_{j,i} v_i (the attention output o_t of Sec. 3.1.4);
* H_j = -sum_i a_{j,i} log a_{j,i}, natural log (the entropy H(a_q) defined in
  Sec. 3.1.1), with 0 log 0 = 0.

Parity pinned by: weights summing to one, L = 1, equal keys (uniform weights,
H = ln L), the two-key closed form, permutation invariance, 0 <= H <= ln L,
and the eviction bound ||o - o^|| <= 2 C eps of Sec. 3.1.4.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


@dataclass
class Attention:
    s: np.ndarray   # (G, L) logits
    m: np.ndarray   # (G,)  max logit
    l: np.ndarray   # (G,)  sum_i exp(s - m)
    a: np.ndarray   # (G, L) attention weights
    H: np.ndarray   # (G,)  entropy of each query's weights, nats
    o: np.ndarray   # (G, d) attention output


def attend(q, K, V, scale: float) -> Attention:
    q = np.asarray(q, np.float64)
    K = np.asarray(K, np.float64)
    V = np.asarray(V, np.float64)
    s = scale * (q @ K.T)
    m = s.max(axis=1)
    e = np.exp(s - m[:, None])
    l = e.sum(axis=1)
    a = e / l[:, None]
    with np.errstate(divide="ignore", invalid="ignore"):
        alog = np.where(a > 0.0, a * np.log(a), 0.0)
    H = -alog.sum(axis=1)
    o = a @ V
    return Attention(s=s, m=m, l=l, a=a, H=H, o=o)


def default_scale(head_dim: int) -> float:
    return 1.0 / np.sqrt(float(head_dim))
