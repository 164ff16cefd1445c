"""Policy scoring MLP s_i = f_phi(x_i) (Sec. 3.1.2; architecture in App. D).

Test infrastructure only (see ``oracle/__init__``).

The paper names a small ReLU MLP; the workloads use 4 -> 32 -> 1 and
4 -> 64 -> 64 -> 1 without LayerNorm (reading recorded in the design notes).
Parameters are one packed float32 blob, row-major:

    W1[h1][n_in], b1[h1], (W2[h2][h1], b2[h2]), w_out[h_last], b_out

so h = relu(W1 x + b1) [, h = relu(W2 h + b2)], s = w_out . h + b_out.

Parity pinned by: zero weights (s = b_out), one-hot probes that pick single
features and hidden units (catch a transposed W or a shuffled feature order),
and a hand-computed integer example.
"""
from __future__ import annotations

import numpy as np


def unpack(params, n_in: int, hidden):
    p = np.asarray(params, np.float64)
    layers, off, prev = [], 0, n_in
    for h in hidden:
        W = p[off:off + h * prev].reshape(h, prev)
        off += h * prev
        b = p[off:off + h]
        off += h
        layers.append((W, b))
        prev = h
    w_out = p[off:off + prev]
    off += prev
    b_out = p[off]
    off += 1
    if off != p.size:
        raise ValueError(f"policy blob has {p.size} values, layout needs {off}")
    return layers, w_out, b_out


def scores(params, x, hidden) -> np.ndarray:
    """x: (L, n_in) features -> (L,) scores."""
    x = np.asarray(x, np.float64)
    layers, w_out, b_out = unpack(params, x.shape[1], hidden)
    h = x
    for W, b in layers:
        h = np.maximum(h @ W.T + b, 0.0)
    return h @ w_out + b_out
