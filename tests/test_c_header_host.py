"""include/sao.h is a plain C header: a C99 program that includes it compiles with
warnings as errors, links against libsao.so, and gets the documented synchronous
errors from every entry point (argument checks run before any device work, so no
GPU is needed)."""
import os
import shutil
import subprocess

import pytest

from paper_2607_07508_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

PROGRAM = r"""
#include <stdio.h>
#include <string.h>
#include "sao.h"

static int fails = 0;
#define EXPECT(call, code) do { sao_status_t s_ = (call); if (s_ != (code)) { \
    printf("%s: got %d (%s), want %d\n", #call, (int)s_, sao_last_error_message(), (int)(code)); ++fails; } } while (0)

int main(void) {
  void* p = (void*)0x10000;   /* never dereferenced: every call below fails validation or is T == 0 */
  if (strlen(sao_status_string(SAO_ERR_SHAPE)) == 0) ++fails;
  if (sao_workspace_size(SAO_OP_LOSS, 1000, 1, 1, SAO_F32) == 0) ++fails;
  EXPECT(sao_token_logprob(NULL, 64, p, 64, p, NULL, 16, 64, 1000, SAO_BF16, p, p, NULL, p, 1u << 30, NULL),
         SAO_ERR_NULL);
  EXPECT(sao_advantage(p, p, p, p, 0, 10, 1.0, 1.0, 0.0, p, p, NULL, NULL, p, 4096, NULL), SAO_ERR_SHAPE);
  EXPECT(sao_clipped_loss(p, p, p, p, 10, -0.2f, 0.2f, NULL, p, p, p, p, p, 1u << 20, NULL), SAO_ERR_VALUE);
  EXPECT(sao_loss_backward(p, 64, p, 64, p, p, p, 16, 64, 100, (sao_dtype_t)7, p, p, p, 1u << 30, NULL),
         SAO_ERR_DTYPE);
  EXPECT(sao_value_forward(p, 64, p, 0, 64, SAO_BF16, p, NULL, 0, NULL), SAO_OK);
  EXPECT(sao_value_loss(p, 64, p, p, p, p, 16, 64, NULL, SAO_BF16, p, p, p, p, 8, NULL), SAO_ERR_WORKSPACE);
  EXPECT(sao_ppo_loss(p, NULL, NULL, p, p, 10, 0.2f, 0.28f, NULL, p, p, p, p, p, 1u << 20, NULL), SAO_ERR_NULL);
  EXPECT(sao_explained_variance(p, p, p, -1, p, NULL, p, 4096, NULL), SAO_ERR_SHAPE);
  EXPECT(sao_step_advantage(p, p, p, p, 2, 10, 1.0, 1.0, 0.0, (sao_step_value_t)9, p, p, NULL, NULL, NULL, p,
                            1u << 20, NULL), SAO_ERR_VALUE);
  EXPECT(sao_group_advantage(p, p, p, 6, 10, 4, 1e-6, p, p, p, NULL, NULL, p, 4096, NULL), SAO_ERR_SHAPE);
  EXPECT(sao_running_mean_advantage(p, p, p, 2, 10, NULL, 1, 0, p, p, p, p, p, NULL, NULL, p, 4096, NULL),
         SAO_ERR_SHAPE);
  sao_debug_time_kernel(SAO_KERNEL_NONE, NULL, NULL);
  if (strlen(sao_version()) == 0) ++fails;
  printf("%s\n", fails ? "FAIL" : "ok");
  return fails != 0;
}
"""


@pytest.mark.skipif(shutil.which("gcc") is None, reason="no C compiler")
def test_header_compiles_as_c99_and_links(tmp_path):
    if not os.path.exists(binding.LIB_PATH):
        pytest.skip("libsao.so not built")
    src = tmp_path / "abi.c"
    src.write_text(PROGRAM)
    exe = tmp_path / "abi"
    libdir = os.path.dirname(binding.LIB_PATH)
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-I", os.path.join(ROOT, "include"), str(src),
           "-L", libdir, "-lsao", f"-Wl,-rpath,{libdir}", "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert run.returncode == 0 and run.stdout.strip().endswith("ok"), run.stdout + run.stderr
