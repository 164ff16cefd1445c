"""Seeded counter-based input generator (host side, numpy).

This module produces every synthetic input of the decode-step workloads: queries,
keys, values, per-row structure draws, policy parameters, hidden states and the
lm-head matrix.  It holds none of the method's arithmetic; both the CPU oracle and
the GPU path take their inputs from it (the GPU side through a bit-identical HIP
twin in ``synth/csrc/synth_gen.hip``, checked element by element in the tests).

Definition
----------
* Bits: Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as
  easy as 1, 2, 3", SC'11).  Counter = (call_lo, call_hi, stream, step), key =
  (seed_lo, seed_hi).  One call yields four 32-bit words x0..x3.
* Uniforms: u = (x + 0.5) * 2^-32, exact in binary64, strictly inside (0, 1).
  Element ``e`` of a uniform stream uses word ``e & 3`` of call ``e >> 2``.
* Normals: Box-Muller on the word pairs (x0, x1) and (x2, x3) of a call:
  r = sqrt(-2 ln u_a), theta = 2 pi u_b; even elements take r cos(theta), odd
  elements r sin(theta).  Element ``e`` uses call ``e >> 2``, pair ``(e >> 1) & 1``.
* ln, sin, cos and exp are evaluated in binary64 with the fixed polynomial
  schemes below, using only IEEE-754 correctly rounded operations (+, -, *, /,
  sqrt) and exact scalings (frexp/ldexp/floor), so that any implementation that
  performs the same operations in the same order (no fused multiply-add)
  reproduces every bit.
* Narrowing: binary64 -> binary32 with round-to-nearest-even, then (for bf16
  tensors) binary32 -> bfloat16 with round-to-nearest-even on the bit pattern.
"""
from __future__ import annotations

import numpy as np

M0 = np.uint64(0xD2511F53)
M1 = np.uint64(0xCD9E8D57)
W0 = 0x9E3779B9
W1 = 0xBB67AE85
MASK32 = np.uint64(0xFFFFFFFF)

# Polynomial coefficients, written as exact binary64 hex literals so that the HIP
# twin can carry the very same values (a CPU test compares the two tables).
LOG_COEF = [float.fromhex(h) for h in (
    "0x1.0000000000000p+0", "0x1.5555555555555p-2", "0x1.999999999999ap-3",
    "0x1.2492492492492p-3", "0x1.c71c71c71c71cp-4", "0x1.745d1745d1746p-4",
    "0x1.3b13b13b13b14p-4", "0x1.1111111111111p-4", "0x1.e1e1e1e1e1e1ep-5",
    "0x1.af286bca1af28p-5", "0x1.8618618618618p-5", "0x1.642c8590b2164p-5",
    "0x1.47ae147ae147bp-5", "0x1.2f684bda12f68p-5")]           # 1/(2k+1)
SIN_COEF = [float.fromhex(h) for h in (
    "0x1.0000000000000p+0", "-0x1.5555555555555p-3", "0x1.1111111111111p-7",
    "-0x1.a01a01a01a01ap-13", "0x1.71de3a556c734p-19", "-0x1.ae64567f544e4p-26",
    "0x1.6124613a86d09p-33", "-0x1.ae7f3e733b81fp-41", "0x1.952c77030ad4ap-49",
    "-0x1.2f49b46814157p-57", "0x1.71b8ef6dcf572p-66", "-0x1.761b41316381ap-75",
    "0x1.3f3ccdd165fa9p-84")]                                   # (-1)^k/(2k+1)!
COS_COEF = [float.fromhex(h) for h in (
    "0x1.0000000000000p+0", "-0x1.0000000000000p-1", "0x1.5555555555555p-5",
    "-0x1.6c16c16c16c17p-10", "0x1.a01a01a01a01ap-16", "-0x1.27e4fb7789f5cp-22",
    "0x1.1eed8eff8d898p-29", "-0x1.93974a8c07c9dp-37", "0x1.ae7f3e733b81fp-45",
    "-0x1.6827863b97d97p-53", "0x1.e542ba4020225p-62", "-0x1.0ce396db7f853p-70",
    "0x1.f2cf01972f578p-80")]                                   # (-1)^k/(2k)!
EXP_COEF = [float.fromhex(h) for h in (
    "0x1.0000000000000p+0", "0x1.0000000000000p+0", "0x1.0000000000000p-1",
    "0x1.5555555555555p-3", "0x1.5555555555555p-5", "0x1.1111111111111p-7",
    "0x1.6c16c16c16c17p-10", "0x1.a01a01a01a01ap-13", "0x1.a01a01a01a01ap-16",
    "0x1.71de3a556c734p-19", "0x1.27e4fb7789f5cp-22", "0x1.ae64567f544e4p-26",
    "0x1.1eed8eff8d898p-29", "0x1.6124613a86d09p-33", "0x1.93974a8c07c9dp-37",
    "0x1.ae7f3e733b81fp-41", "0x1.ae7f3e733b81fp-45", "0x1.952c77030ad4ap-49")]  # 1/k!
LN2 = float.fromhex("0x1.62e42fefa39efp-1")
INV_LN2 = float.fromhex("0x1.71547652b82fep+0")
PI_2 = float.fromhex("0x1.921fb54442d18p+0")
SQRT_HALF = float.fromhex("0x1.6a09e667f3bcdp-1")
TWO_M32 = float.fromhex("0x1.0000000000000p-32")


def philox4x32_10(c0, c1, c2, c3, k0: int, k1: int):
    """Philox4x32 with 10 rounds on uint64 arrays holding 32-bit lanes."""
    c0 = np.asarray(c0, np.uint64) & MASK32
    c1 = np.asarray(c1, np.uint64) & MASK32
    c2 = np.asarray(c2, np.uint64) & MASK32
    c3 = np.asarray(c3, np.uint64) & MASK32
    c0, c1, c2, c3 = np.broadcast_arrays(c0, c1, c2, c3)
    k0 &= 0xFFFFFFFF
    k1 &= 0xFFFFFFFF
    for r in range(10):
        if r:
            k0 = (k0 + W0) & 0xFFFFFFFF
            k1 = (k1 + W1) & 0xFFFFFFFF
        p0 = M0 * c0
        p1 = M1 * c2
        hi0, lo0 = p0 >> np.uint64(32), p0 & MASK32
        hi1, lo1 = p1 >> np.uint64(32), p1 & MASK32
        c0, c1, c2, c3 = (hi1 ^ c1 ^ np.uint64(k0), lo1,
                          hi0 ^ c3 ^ np.uint64(k1), lo0)
    return c0, c1, c2, c3


def _words(seed: int, stream: int, step: int, call):
    call = np.asarray(call, np.uint64)
    return philox4x32_10(call & MASK32, call >> np.uint64(32),
                         np.uint64(stream), np.uint64(step),
                         seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF)


def _to_unit(x):
    return (x.astype(np.float64) + 0.5) * TWO_M32


def _horner(coefs, x):
    p = np.full_like(x, coefs[-1])
    for c in coefs[-2::-1]:
        p = p * x
        p = p + c
    return p


def det_log(u):
    """ln(u) for u > 0: frexp range reduction, then 2*atanh((m-1)/(m+1))."""
    m, e = np.frexp(u)                      # u = m * 2^e, m in [0.5, 1)
    low = m < SQRT_HALF
    m = np.where(low, m * 2.0, m)
    e = np.where(low, e - 1, e).astype(np.float64)
    z = (m - 1.0) / (m + 1.0)
    z2 = z * z
    s = _horner(LOG_COEF, z2)
    s = s * z
    s = s * 2.0
    return e * LN2 + s


def det_sincos(u):
    """(cos(2 pi u), sin(2 pi u)) for u in [0, 1): quadrant split + Taylor."""
    v = u * 4.0
    q = np.floor(v)
    f = v - q
    x = f * PI_2
    x2 = x * x
    s = _horner(SIN_COEF, x2)
    s = s * x
    c = _horner(COS_COEF, x2)
    qi = q.astype(np.int64) & 3
    cos_t = np.select([qi == 0, qi == 1, qi == 2], [c, -s, -c], s)
    sin_t = np.select([qi == 0, qi == 1, qi == 2], [s, c, -s], -c)
    return cos_t, sin_t


def det_exp(x):
    """exp(x) for |x| < 700: k = rint(x / ln2), Taylor on the remainder."""
    k = np.rint(x * INV_LN2)
    r = x - k * LN2
    p = _horner(EXP_COEF, r)
    return np.ldexp(p, k.astype(np.int64))


def uniform(seed: int, stream: int, step: int, idx) -> np.ndarray:
    """Uniform (0,1) binary64 values for element indices ``idx``."""
    idx = np.asarray(idx, np.uint64)
    if idx.size >= FAST_MIN and _fast() is not None:
        return _fast_values(idx, seed, stream, step, 1)
    return uniform_np(seed, stream, step, idx)


def uniform_np(seed: int, stream: int, step: int, idx) -> np.ndarray:
    """numpy evaluation of ``uniform`` (the readable definition)."""
    idx = np.asarray(idx, np.uint64)
    w = _words(seed, stream, step, idx >> np.uint64(2))
    lane = (idx & np.uint64(3)).astype(np.int64)
    x = np.select([lane == 0, lane == 1, lane == 2], [w[0], w[1], w[2]], w[3])
    return _to_unit(x)


def normal(seed: int, stream: int, step: int, idx) -> np.ndarray:
    """Standard normal binary64 values for element indices ``idx``."""
    idx = np.asarray(idx, np.uint64)
    if idx.size >= FAST_MIN and _fast() is not None:
        return _fast_values(idx, seed, stream, step, 0)
    return normal_np(seed, stream, step, idx)


def normal_np(seed: int, stream: int, step: int, idx) -> np.ndarray:
    """numpy evaluation of ``normal`` (the readable definition)."""
    idx = np.asarray(idx, np.uint64)
    w = _words(seed, stream, step, idx >> np.uint64(2))
    pair = ((idx >> np.uint64(1)) & np.uint64(1)).astype(bool)
    ua = _to_unit(np.where(pair, w[2], w[0]))
    ub = _to_unit(np.where(pair, w[3], w[1]))
    r = np.sqrt(det_log(ua) * -2.0)
    cos_t, sin_t = det_sincos(ub)
    odd = (idx & np.uint64(1)).astype(bool)
    return np.where(odd, r * sin_t, r * cos_t)


def to_f32(x) -> np.ndarray:
    """binary64 -> binary32, round to nearest even."""
    return np.asarray(x, np.float64).astype(np.float32)


def f32_to_bf16_bits(x) -> np.ndarray:
    """binary32 -> bfloat16 bit pattern, round to nearest even (no NaN inputs)."""
    b = np.asarray(x, np.float32).view(np.uint32).astype(np.uint64)
    b = (b + np.uint64(0x7FFF) + ((b >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    return b.astype(np.uint16)


def bf16_bits_to_f32(bits) -> np.ndarray:
    return (np.asarray(bits, np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def narrow(x, dtype: str) -> np.ndarray:
    """Round binary64 values to the storage dtype; returns float32 values that
    are exactly representable in that dtype ('f32' or 'bf16')."""
    f = to_f32(x)
    if dtype == "f32":
        return f
    if dtype == "bf16":
        return bf16_bits_to_f32(f32_to_bf16_bits(f))
    raise ValueError(dtype)


# ---------------------------------------------------------------------------
# Bulk evaluation through the host build of the generator library (the same
# binary64 operations compiled as C++ for the CPU); tests check it against the
# numpy evaluation above, element by element.
FAST_MIN = 1 << 14
_FAST = None
_FAST_TRIED = False


def _fast():
    global _FAST, _FAST_TRIED
    if not _FAST_TRIED:
        _FAST_TRIED = True
        import ctypes
        import os
        path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libdcsynth.so")
        if os.path.exists(path):
            try:
                L = ctypes.CDLL(path)
                L.synth_cpu_values.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint64,
                                               ctypes.c_uint64, ctypes.c_int, ctypes.c_int,
                                               ctypes.c_int, ctypes.c_int]
                L.synth_cpu_values.restype = None
                _FAST = L
            except OSError:
                _FAST = None
    return _FAST


def _threads() -> int:
    import os
    return max(1, min(16, os.cpu_count() or 1))


def _fast_values(idx, seed, stream, step, kind):
    idx = np.ascontiguousarray(idx, np.uint64)
    out = np.empty(idx.shape, np.float64)
    _fast().synth_cpu_values(out.ctypes.data, idx.ctypes.data, idx.size, seed, stream, step, kind,
                             _threads())
    return out
