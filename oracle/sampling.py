"""Training-mode selection: Gumbel-perturbed top-B and the log-probability of
the sampled subset (Sec. 3.1.2, stochastic ranking during training; App. C,
policy-gradient derivation for Gumbel-top-B).

Test infrastructure only (see ``oracle/__init__``).  Binary64 throughout.

Noise
-----
The paper perturbs every score with an independent standard Gumbel draw.  The
draw is made reproducible by a counter-based generator, Philox4x32-10 (Salmon,
Moraes, Dror and Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC'11),
written here from its published definition: ten rounds of

    (c0, c1, c2, c3) <- (hi(M1 c2) ^ c1 ^ k0, lo(M1 c2), hi(M0 c0) ^ c3 ^ k1, lo(M0 c0))

with M0 = 0xD2511F53, M1 = 0xCD9E8D57 and the key advanced by the Weyl constants
(0x9E3779B9, 0xBB67AE85) between rounds.  For token position p of unit u at
draw number `draw` under the 64-bit seed (k0, k1) the counter is (p, u, draw, 0);
the first output word x gives

    U = (2 (x >> 9) + 1) 2^-24      (exactly representable in binary32, 0 < U < 1)
    g = -ln(-ln U)                   (standard Gumbel by inversion of its CDF)

Selection
---------
Perturbed score s~_i = s_i / tau + g_i (App. C; tau = 1 gives Sec. 3.1.2's
form).  The kept set is the top B of s~ under the order of the deterministic
selection (higher first, ties to the earlier token; see ``oracle.select``).

Log-probability (App. C, taken as written)
-----------------------------------------
    log pi(a | s) = sum_{i in a} s_i / tau - log Z(s, B, tau),
    Z(s, B, tau)  = sum over the size-B subsets a' of exp(sum_{i in a'} s_i / tau).

log Z is computed exactly by the paper's O(L B) dynamic programme over the rows
with logaddexp: E[0] = 0, E[j > 0] = -inf; for each row i,
E[j] <- logaddexp(E[j], E[j-1] + s_i / tau) for j = B .. 1; log Z = E[B].
If B >= L the only subset is the whole cache: log Z = sum_i s_i / tau and the
kept set has log-probability 0.

Reading recorded with the design notes: App. C calls exp(sum s / tau) / Z the
Plackett-Luce law of the top-B set.  The law that Gumbel-top-B sampling
actually induces is the Plackett-Luce law of the first B items drawn without
replacement, which is a different distribution for B > 1; these functions follow
the paper's formula, and a test documents the difference.

Parity pinned by: the Random123 known-answer vectors (generator); Gumbel mean
(Euler-Mascheroni constant), variance (pi^2 / 6) and Kolmogorov-Smirnov
distance on a million draws; the Gumbel-max property (argmax frequencies match
softmax) and the without-replacement law of the top-B set; brute-force subset
enumeration of Z on small L for every B; B = 1 (logsumexp), B = L (sum),
B = L - 1, all-equal scores (log of a binomial coefficient), the temperature
identity Z(s, B, tau) = Z(s / tau, B, 1), the complement identity
log Z(s, B) = sum s + log Z(-s, L - B), and normalisation of pi over all subsets.
"""
from __future__ import annotations

import numpy as np

_MUL = (0xD2511F53, 0xCD9E8D57)
_WEYL = (0x9E3779B9, 0xBB67AE85)
_M32 = 0xFFFFFFFF


def philox4x32_10(counter, key):
    """Philox4x32-10 of one or many counters.

    counter: 4 integer arrays (broadcastable) of 32-bit words; key: 2 integers.
    Returns the 4 output words as uint64 arrays holding 32-bit values."""
    c = [np.asarray(w, dtype=np.uint64) & np.uint64(_M32) for w in counter]
    c = list(np.broadcast_arrays(*c))
    k0, k1 = int(key[0]) & _M32, int(key[1]) & _M32
    m0, m1 = np.uint64(_MUL[0]), np.uint64(_MUL[1])
    for rnd in range(10):
        if rnd:
            k0 = (k0 + _WEYL[0]) & _M32
            k1 = (k1 + _WEYL[1]) & _M32
        p0 = c[0] * m0          # < 2^64: exact in uint64
        p1 = c[2] * m1
        hi0, lo0 = p0 >> np.uint64(32), p0 & np.uint64(_M32)
        hi1, lo1 = p1 >> np.uint64(32), p1 & np.uint64(_M32)
        c = [hi1 ^ c[1] ^ np.uint64(k0), lo1, hi0 ^ c[3] ^ np.uint64(k1), lo0]
    return c


def gumbel_uniform(seed: int, unit: int, draw: int, pos) -> np.ndarray:
    """U in (0, 1) for the tokens at positions `pos` of `unit` (see module doc)."""
    pos = np.asarray(pos, dtype=np.int64)
    x = philox4x32_10((pos, unit, draw, 0), (seed & _M32, (seed >> 32) & _M32))[0]
    return (2.0 * (x >> np.uint64(9)).astype(np.float64) + 1.0) * 2.0 ** -24


def gumbel(seed: int, unit: int, draw: int, pos) -> np.ndarray:
    """Standard Gumbel draws g = -ln(-ln U)."""
    return -np.log(-np.log(gumbel_uniform(seed, unit, draw, pos)))


def perturbed_scores(scores, tau: float, noise) -> np.ndarray:
    """s~ = s / tau + g."""
    return np.asarray(scores, np.float64) / float(tau) + np.asarray(noise, np.float64)


def sample_top_budget(scores, positions, budget: int, tau: float, noise) -> np.ndarray:
    """Rows (ascending) of the top-`budget` tokens under the perturbed scores.
    Ordering and tie rule as in the deterministic selection."""
    from oracle import select
    return select.top_budget(perturbed_scores(scores, tau, noise), positions, budget)


def log_partition(scores, budget: int, tau: float = 1.0) -> float:
    """log Z(s, B, tau) by the logaddexp dynamic programme (App. C)."""
    r = np.asarray(scores, np.float64) / float(tau)
    L = r.size
    if budget < 1:
        raise ValueError("budget must be >= 1")
    if budget >= L:
        return float(r.sum())
    E = np.full(budget + 1, -np.inf)
    E[0] = 0.0
    for i in range(L):
        # E[j] takes row i in (E[j-1] + r_i) or leaves it out (E[j]); the right
        # side is evaluated from the values before row i
        E[1:] = np.logaddexp(E[1:], E[:-1] + r[i])
    return float(E[budget])


def log_prob(scores, kept, budget: int, tau: float = 1.0) -> float:
    """log pi(a | s) of the kept rows `kept` (indices into `scores`)."""
    r = np.asarray(scores, np.float64) / float(tau)
    if budget >= r.size:
        return 0.0
    return float(r[np.asarray(kept, np.int64)].sum()) - log_partition(scores, budget, tau)
