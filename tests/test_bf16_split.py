"""The arithmetic behind the scoring pass's matrix-core contraction (CPU).

Every float32 operand is split into three bf16 parts by round-to-nearest-even
conversions, x = h + m + l, and a product of two operands keeps six of the
nine part products.  These tests check, on the host with an independent
round-to-nearest-even emulation, that the split is exact for float32 values
across the exponent range the features and weights take, that the part
products are exact in float32, and that the six kept products differ from
the exact product by at most about 2^-23 of it (one float32 rounding).
"""
import numpy as np


def to_bf16_rne(x: np.ndarray) -> np.ndarray:
    """float32 -> nearest bf16 (ties to even), returned as float32."""
    b = np.asarray(x, np.float32).view(np.uint32).astype(np.uint64)
    lsb = (b >> 16) & 1
    r = ((b + 0x7FFF + lsb) >> 16) << 16
    return r.astype(np.uint32).view(np.float32)


def split3(x: np.ndarray):
    x = np.asarray(x, np.float32)
    h = to_bf16_rne(x)
    r1 = (x - h).astype(np.float32)
    m = to_bf16_rne(r1)
    r2 = (r1 - m).astype(np.float32)
    l = to_bf16_rne(r2)
    return h, m, l


def _operands(n, seed, lo=-20, hi=20):
    rng = np.random.default_rng(seed)
    mant = rng.uniform(1.0, 2.0, n)
    sign = rng.choice([-1.0, 1.0], n)
    return (sign * mant * np.exp2(rng.integers(lo, hi, n))).astype(np.float32)


def test_bf16_rounding_emulation_matches_hand_cases():
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7: to even gives 1
    x = np.array([1.0, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -2.5, 3.0e-5], np.float32)
    got = to_bf16_rne(x)
    assert got[0] == 1.0
    assert got[1] == 1.0
    assert got[2] == np.float32(1.0 + 2.0 ** -6)
    assert got[3] == -2.5
    # a bf16 value has at most 8 significant bits
    assert np.all((got.view(np.uint32) & 0xFFFF) == 0)


def test_three_parts_reconstruct_float32_exactly():
    x = _operands(1 << 20, 1)
    h, m, l = split3(x)
    for part in (h, m, l):
        assert np.all((part.view(np.uint32) & 0xFFFF) == 0)     # genuine bf16 values
    back = (h.astype(np.float64) + m.astype(np.float64)) + l.astype(np.float64)
    assert np.array_equal(back, x.astype(np.float64))
    # the residual parts shrink by about 2^-8 each
    nz = x != 0
    assert np.all(np.abs(m[nz]) <= np.abs(x[nz]) * 2.0 ** -8 * 1.0001)
    assert np.all(np.abs(l[nz]) <= np.abs(x[nz]) * 2.0 ** -16 * 1.0001)


def test_part_products_are_exact_in_float32():
    a, b = _operands(1 << 18, 2), _operands(1 << 18, 3)
    ha, ma, la = split3(a)
    hb, mb, lb = split3(b)
    for p, q in ((ha, hb), (ha, mb), (ma, hb), (ha, lb), (ma, mb), (la, hb)):
        exact = p.astype(np.float64) * q.astype(np.float64)
        assert np.array_equal((p * q).astype(np.float64), exact)


def test_six_kept_products_are_within_one_float32_rounding():
    a, b = _operands(1 << 20, 4), _operands(1 << 20, 5)
    ha, ma, la = split3(a)
    hb, mb, lb = split3(b)
    f = lambda v: v.astype(np.float64)
    kept = (f(la) * f(hb) + f(ma) * f(mb) + f(ha) * f(lb) + f(ma) * f(hb) + f(ha) * f(mb)
            + f(ha) * f(hb))
    exact = f(a) * f(b)
    rel = np.abs(kept - exact) / np.abs(exact)
    assert rel.max() <= 2.0 ** -22
    # the float32 product it replaces rounds by up to 2^-24
    rel32 = np.abs(f((a * b).astype(np.float32)) - exact) / np.abs(exact)
    assert rel32.max() <= 2.0 ** -24 * 1.0001


def test_dot_product_error_matches_float32_accumulation():
    """A 128-term dot product through the six kept products, summed in
    float32, stays within the error bound of a plain float32 dot product."""
    rng = np.random.default_rng(6)
    n = 128
    for trial in range(200):
        a = rng.standard_normal(n).astype(np.float32)
        b = (0.1 * rng.standard_normal(n)).astype(np.float32)
        ha, ma, la = split3(a)
        hb, mb, lb = split3(b)
        acc = np.float32(0.0)
        for k in range(n):
            for p, q in ((la, hb), (ma, mb), (ha, lb), (ma, hb), (ha, mb), (ha, hb)):
                acc = np.float32(acc + p[k] * q[k])
        exact = float(np.dot(a.astype(np.float64), b.astype(np.float64)))
        bound = (6 * n + 2) * 2.0 ** -24 * float(np.abs(a.astype(np.float64)) @ np.abs(b.astype(np.float64)))
        assert abs(float(acc) - exact) <= bound, trial
