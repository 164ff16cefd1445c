"""Policy scoring MLP s_i = f_phi(x_i) (Sec. 3.1.2; architecture in App. D).

Test infrastructure only (see ``oracle/__init__``).

The paper names a small ReLU MLP; the workloads use 4 -> 32 -> 1 and
4 -> 64 -> 64 -> 1 without LayerNorm (reading recorded in the design notes).
Parameters are one packed float32 blob, row-major:

    W1[h1][n_in], b1[h1], (W2[h2][h1], b2[h2]), w_out[h_last], b_out

so h = relu(W1 x + b1) [, h = relu(W2 h + b2)], s = w_out . h + b_out.

The paper's own description adds LayerNorm (App. D); with ``layer_norm`` every
hidden layer is Linear -> LayerNorm -> ReLU (placement, epsilon 1e-5 and the
per-layer gain/bias packed after b are readings recorded with the design
notes), and the input may carry the fifth feature sigma_i.  Packed layout:

    per hidden layer: W[h][prev], b[h], (gain[h], bias[h] with LayerNorm); w_out, b_out

Parity pinned by: zero weights (s = b_out), one-hot probes that pick single
features and hidden units (catch a transposed W or a shuffled feature order),
a hand-computed integer example; LayerNorm: normalised units have mean 0 and
variance var / (var + eps), invariance to a shift of every pre-activation,
and a hand-computed two-unit case.
"""
from __future__ import annotations

import numpy as np


LN_EPS = 1e-5


def unpack(params, n_in: int, hidden, layer_norm: bool = False):
    p = np.asarray(params, np.float64)
    layers, off, prev = [], 0, n_in
    for h in hidden:
        W = p[off:off + h * prev].reshape(h, prev)
        off += h * prev
        b = p[off:off + h]
        off += h
        g = be = None
        if layer_norm:
            g = p[off:off + h]
            be = p[off + h:off + 2 * h]
            off += 2 * h
        layers.append((W, b, g, be))
        prev = h
    w_out = p[off:off + prev]
    off += prev
    b_out = p[off]
    off += 1
    if off != p.size:
        raise ValueError(f"policy blob has {p.size} values, layout needs {off}")
    return layers, w_out, b_out


def layer_norm_rows(z, g, be, eps: float = LN_EPS) -> np.ndarray:
    """Per row: g * (z - mean) / sqrt(var + eps) + be over the layer's units
    (population variance)."""
    mean = z.mean(axis=1, keepdims=True)
    var = ((z - mean) ** 2).mean(axis=1, keepdims=True)
    return g * (z - mean) / np.sqrt(var + eps) + be


def scores(params, x, hidden, layer_norm: bool = False) -> np.ndarray:
    """x: (L, n_in) features -> (L,) scores.  With layer_norm, every hidden layer
    is Linear -> LayerNorm -> ReLU."""
    x = np.asarray(x, np.float64)
    layers, w_out, b_out = unpack(params, x.shape[1], hidden, layer_norm)
    h = x
    for W, b, g, be in layers:
        z = h @ W.T + b
        if layer_norm:
            z = layer_norm_rows(z, g, be)
        h = np.maximum(z, 0.0)
    return h @ w_out + b_out
