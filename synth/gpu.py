"""Device-side twin of the input generator (libdcsynth.so): fills torch tensors
with exactly the values ``synth.philox`` / ``synth.workloads`` define."""
from __future__ import annotations

import ctypes
import os

import torch

from . import workloads as W

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdcsynth.so")
KEY_STRUCTURE = {"none": 0, "heavy": 1, "lognormal": 2, "sink": 3}
_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with python -m synth.build")
        L = ctypes.CDLL(LIB_PATH)
        u64, i32, i64, vp = ctypes.c_uint64, ctypes.c_int, ctypes.c_int64, ctypes.c_void_p
        L.synth_fill_rows.argtypes = [vp, i32, u64, i32, i32, i64, i32, i32, i64, i64, i32, i64, vp]
        L.synth_fill_normal.argtypes = [vp, i32, u64, i32, i32, u64, ctypes.c_double, vp]
        L.synth_fill_noisy.argtypes = [vp, vp, u64, i32, i32, u64, ctypes.c_double, vp]
        for f in (L.synth_fill_rows, L.synth_fill_normal, L.synth_fill_noisy):
            f.restype = ctypes.c_int
        _lib = L
    return _lib


def _dt(t: torch.Tensor) -> int:
    return {torch.float32: 0, torch.bfloat16: 1}[t.dtype]


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ok(rc: int):
    if rc != 0:
        raise RuntimeError(f"synth launch failed: hipError {rc}")


def fill_rows(out: torch.Tensor, wl: W.Workload, which: str, units: int, unit_stride_rows: int,
              pos0: int, nrows: int, dst_row0: int = 0, unit0: int = 0) -> None:
    """Key ('k') or value ('v') rows at positions pos0..pos0+nrows-1 of units
    unit0..unit0+units-1, into out viewed as [units][unit_stride_rows][head_dim]
    starting at row dst_row0."""
    assert out.is_contiguous() and out.numel() >= units * unit_stride_rows * wl.head_dim
    assert dst_row0 + nrows <= unit_stride_rows
    stream = W.S_K if which == "k" else W.S_V
    ks = KEY_STRUCTURE[wl.key_structure] if which == "k" else -1
    _ok(lib().synth_fill_rows(out.data_ptr(), _dt(out), wl.seed, stream, ks, unit0, units,
                              wl.head_dim, unit_stride_rows, pos0, nrows, dst_row0, _stream()))


def fill_normal(out: torch.Tensor, wl: W.Workload, stream: int, step: int, std: float) -> None:
    assert out.is_contiguous()
    _ok(lib().synth_fill_normal(out.data_ptr(), _dt(out), wl.seed, stream, step, out.numel(),
                                std, _stream()))


def fill_noisy(out: torch.Tensor, base: torch.Tensor, wl: W.Workload, step: int, eps: float) -> None:
    assert out.is_contiguous() and base.is_contiguous() and out.dtype == torch.bfloat16
    _ok(lib().synth_fill_noisy(out.data_ptr(), base.data_ptr(), wl.seed, W.S_HCOMP, step,
                               out.numel(), eps, _stream()))


def queries(wl: W.Workload, step: int, out: torch.Tensor) -> torch.Tensor:
    """All units' queries of a decode step, [units][G][head_dim]."""
    fill_normal(out, wl, W.S_Q, step, 1.0)
    return out


def new_rows(wl: W.Workload, step: int, k_out: torch.Tensor, v_out: torch.Tensor, units: int):
    """The key/value rows appended at decode step `step` (position n0 + step)."""
    fill_rows(k_out, wl, "k", units, 1, wl.n0 + step, 1, 0)
    fill_rows(v_out, wl, "v", units, 1, wl.n0 + step, 1, 0)


def init_cache(wl: W.Workload, k: torch.Tensor, v: torch.Tensor, units: int, capacity: int,
               n0: int | None = None, unit0: int = 0) -> None:
    """Positions 0..n0-1 of units unit0.. into slots 0..n0-1 of every unit."""
    n0 = wl.n0 if n0 is None else n0
    fill_rows(k, wl, "k", units, capacity, 0, n0, 0, unit0)
    fill_rows(v, wl, "v", units, capacity, 0, n0, 0, unit0)
