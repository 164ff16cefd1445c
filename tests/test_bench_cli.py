"""bench.py on the CPU: the one-GPU refusal and the algorithmic byte count that
its roofline line divides by the measured kernel time."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def _run_bench(args, env_extra=None):
    env = dict(os.environ)
    env.update(env_extra or {})
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], cwd=ROOT,
                          env=env, capture_output=True, text=True, timeout=120)


@pytest.mark.parametrize("args,env", [(["--gpus", "2"], None), (["--gpus", "8"], None),
                                      ([], {"WORLD_SIZE": "2"})])
def test_bench_refuses_more_than_one_gpu(args, env):
    r = _run_bench(args, env)
    assert r.returncode == 2
    assert "measures one GPU" in r.stderr
    assert not r.stdout.strip()          # no JSON line is printed


def test_step_bytes_of_the_headline_launch():
    """4096 units of 4097 rows (after the append), 4 query heads of 128 bf16
    elements per unit, the window full, 2061 compaction moves: the per-unit
    terms of a steady step added one by one."""
    import bench

    U, L, G, D, moved = 4096, 4097, 4, 128, 2061
    row = 2 * D * 2                       # one K row and one V row, bf16
    per_unit = 0
    per_unit += (L - 1) * row             # cached K/V read once
    per_unit += row + row                 # the new row read from k_new/v_new and written
    per_unit += L * (4 + 8 + 8) * 2       # alpha, N, Z read and written
    per_unit += L * (4 + 4)               # pos and the value norm read
    per_unit += G * D * 2 * 2             # queries read, outputs written
    per_unit += G * D * 2 * 2             # retiring queries read, this step's written to the ring
    per_unit += 2 * G * 3 * 4             # per-query statistics read and written
    moves = moved * 2 * (row + 4 + 8 + 8 + 4 + 4)   # K/V and 28 B of state, read and written
    assert U * per_unit + moves == 9_419_028_184
    assert bench.step_alg_bytes(U, L, G, D, 2, True, moved) == U * per_unit + moves
    # before the window is full no retiring queries are read
    assert (bench.step_alg_bytes(U, L, G, D, 2, True, moved)
            - bench.step_alg_bytes(U, L, G, D, 2, False, moved)) == U * G * D * 2
