"""Input generator checks (CPU): Philox known-answer vectors, random access,
rounding, and the workload recipes."""
import math
import os
import re

import numpy as np
import torch

from synth import philox as px
from synth import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_philox4x32_10_known_answers():
    # Known-answer vectors published with the Random123 library (Salmon et al., SC'11).
    cases = [
        ((0, 0, 0, 0), (0, 0), (0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8)),
        ((0xFFFFFFFF,) * 4, (0xFFFFFFFF, 0xFFFFFFFF), (0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD)),
        ((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344), (0xA4093822, 0x299F31D0),
         (0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1)),
    ]
    for ctr, key, want in cases:
        got = px.philox4x32_10(*ctr, *key)
        assert tuple(int(x) for x in got) == want


def test_transcendentals_are_accurate():
    u = np.random.default_rng(0).uniform(1e-12, 1, 200000)
    assert np.max(np.abs(px.det_log(u) - np.log(u)) / np.abs(np.log(u))) < 1e-14
    c, s = px.det_sincos(u)
    assert np.max(np.abs(c - np.cos(2 * np.pi * u))) < 1e-14
    assert np.max(np.abs(s - np.sin(2 * np.pi * u))) < 1e-14
    x = np.random.default_rng(1).uniform(-20, 20, 200000)
    assert np.max(np.abs(px.det_exp(x) / np.exp(x) - 1)) < 1e-14


def test_normal_moments_and_random_access():
    idx = np.arange(1 << 20, dtype=np.uint64)
    z = px.normal(7, 3, 2, idx)
    assert abs(z.mean()) < 5e-3 and abs(z.std() - 1) < 5e-3
    kurt = ((z - z.mean()) ** 4).mean() / z.var() ** 2
    assert abs(kurt - 3) < 0.05
    sub = np.array([5, 99999, 123456, 1048575], dtype=np.uint64)
    assert np.array_equal(px.normal(7, 3, 2, sub), z[sub.astype(np.int64)])
    assert not np.array_equal(px.normal(7, 3, 3, sub), z[sub.astype(np.int64)])


def test_bf16_rounding_matches_torch_round_to_nearest_even():
    x = np.random.default_rng(2).normal(size=100000).astype(np.float32) * 10
    x[:4] = [1.00390625, 1.01171875, -1.00390625, 3.0]   # exact halfway cases
    ours = px.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


def test_hip_twin_uses_the_same_constants():
    """The GPU generator must carry bit-identical polynomial constants."""
    src = open(os.path.join(ROOT, "synth", "csrc", "synth_gen.hip")).read()
    tables = {}
    for name in ("LOG_COEF", "SIN_COEF", "COS_COEF", "EXP_COEF"):
        m = re.search(name + r"\[\]\s*=\s*\{([^}]*)\}", src)
        assert m, name
        tables[name] = [float.fromhex(t.strip()) for t in m.group(1).split(",") if t.strip()]
        assert tables[name] == getattr(px, name), name
    for name in ("LN2", "INV_LN2", "PI_2", "SQRT_HALF"):
        m = re.search(r"\b" + name + r"\s*=\s*([-0-9a-fA-Fx.p+]+)", src)
        assert m and float.fromhex(m.group(1)) == getattr(px, name), name


def test_workload_shapes_match_the_recipes():
    c3 = wl.WORKLOADS[3]
    assert (c3.units, c3.group, c3.capacity) == (16 * 32 * 8, 4, 16384 + 128)
    assert wl.WORKLOADS[1].n_params == 4 * 32 + 32 + 32 + 1
    assert wl.WORKLOADS[4].n_params == 4 * 64 + 64 + 64 * 64 + 64 + 64 + 1
    k = wl.key_rows(wl.WORKLOADS[2], 3, np.arange(4096))
    heavy = np.abs(k).max(axis=1) > 6 * 3.5
    assert 10 < heavy.sum() < 90           # about 1 % of 4096 rows scaled x8
    k4 = wl.key_rows(wl.WORKLOADS[4], 0, np.arange(128))
    assert np.sqrt((k4[:64] ** 2).mean()) > 3 * np.sqrt((k4[64:] ** 2).mean())
    # bf16 workloads hold bf16-exact values
    b = px.f32_to_bf16_bits(k)
    assert np.array_equal(px.bf16_bits_to_f32(b), k)
    # an appended row is the row of that position in the same index space
    assert np.array_equal(wl.key_rows(c3, 11, [16384]), wl.key_rows(c3, 11, np.arange(16380, 16385))[-1:])
