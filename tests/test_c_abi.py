"""The C ABI from C: a C99 program compiled against include/distillcache.h and
linked with the library calls entry points whose validation fails on the host
(no device work) and checks the status codes and strings; no GPU needed."""
import os
import shutil
import subprocess

import pytest

from paper_2608_08878_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

PROGRAM = r"""
#include <stdio.h>
#include <string.h>
#include "distillcache.h"

#define CHECK(expr, want)                                                   \
  do {                                                                      \
    dc_status s_ = (expr);                                                  \
    if (s_ != (want)) {                                                     \
      printf("FAIL %s: %d != %d\n", #expr, (int)s_, (int)(want));           \
      return 1;                                                             \
    }                                                                       \
  } while (0)

int main(void) {
  void *fake = (void *)0x10000;
  dc_dims d;
  memset(&d, 0, sizeof d);
  d.batch = 1; d.n_layers = 1; d.n_q_heads = 8; d.n_kv_heads = 2; d.head_dim = 128;
  d.capacity = 100; d.dtype = DC_BF16; d.ent_window = 64; d.scale = 0.0f;
  CHECK(dc_decode_step(NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, 0, NULL), DC_ERR_NULL);
  CHECK(dc_kl_reward(8, 4096, 32768, NULL, fake, fake, fake, fake, 1u << 30, NULL), DC_ERR_NULL);
  CHECK(dc_kl_reward(8, 4000, 32768, fake, fake, fake, fake, fake, 1u << 30, NULL), DC_ERR_UNSUPPORTED);
  CHECK(dc_kl_pack_lm_head(4096, 32768, fake, fake, NULL), DC_ERR_UNSUPPORTED);
  CHECK(dc_kl_reward_static(1025, 4096, 32768, fake, fake, fake, fake, NULL), DC_ERR_SCRATCH);
  if (dc_workspace_bytes(&d, 1000, 8, 32768) == 0) { printf("FAIL workspace\n"); return 1; }
  d.n_q_heads = 6;          /* G = 3 */
  if (dc_workspace_bytes(&d, 1000, 0, 0) != 0) { printf("FAIL bad dims\n"); return 1; }
  if (strncmp(dc_status_str(DC_ERR_SCRATCH), "DC_ERR_SCRATCH", 14) != 0) { printf("FAIL str\n"); return 1; }
  printf("c abi ok\n");
  return 0;
}
"""


@pytest.mark.skipif(not os.path.exists(B.LIB_PATH) or shutil.which("gcc") is None,
                    reason="library not built or no C compiler")
def test_c_program_calls_the_abi(tmp_path):
    src = tmp_path / "abi.c"
    src.write_text(PROGRAM)
    exe = tmp_path / "abi"
    libdir = os.path.dirname(B.LIB_PATH)
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror",
                    "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe),
                    "-L", libdir, "-ldistillcache", "-Wl,-rpath," + libdir],
                   check=True, capture_output=True, text=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "c abi ok" in r.stdout
