"""Compile the HIP kernels and the C-ABI host layer into libdistillcache.so (gfx950)."""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libdistillcache.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SOURCES = ["dc_api.cpp", "dc_decode.hip", "dc_step.hip", "dc_evict.hip", "dc_kl.hip",
           "dc_logz.hip", "dc_reinforce.hip", "dc_mlp.hip", "dc_alpha.hip"]
# -ffp-contract=off: every fused multiply-add in the kernels is written explicitly, so the
# retire step can reproduce the arithmetic of the step that added a contribution.
# packed-fp32-ops is disabled: the compiler must not emit packed float32 arithmetic.
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-ffp-contract=off",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wno-unused-result", "-Wno-unused-value", "-I", os.path.join(ROOT, "include")]


def _compile(src: str, obj: str, extra=()) -> None:
    cmd = [HIPCC, *FLAGS, *extra, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")


def build_library(sources, out: str, srcdir: str, extra=()) -> str:
    bdir = os.path.join(ROOT, "_build", os.path.splitext(os.path.basename(out))[0])
    os.makedirs(bdir, exist_ok=True)
    objs = [os.path.join(bdir, s + ".o") for s in sources]
    with ThreadPoolExecutor(max_workers=min(8, len(sources))) as ex:
        list(ex.map(lambda so: _compile(os.path.join(srcdir, so[0]), so[1], extra), zip(sources, objs)))
    tmp = out + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed for {out}:\n{r.stderr}")
    os.replace(tmp, out)
    return out


def build() -> str:
    return build_library(SOURCES, LIB, CSRC)


if __name__ == "__main__":
    print(build())
    sys.exit(0)
