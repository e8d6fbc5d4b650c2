"""The C ABI from C: include/smat.h compiles as C99 with gcc (-Wall -Wextra -Werror) and a C program
linked against libsmat.so gets the documented status codes and messages on argument errors.  Only
host-side paths run (no device memory is touched), so the test needs no GPU."""
import os
import shutil
import subprocess

import pytest

import paper_2609_33437_amd as smat

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIBDIR = os.path.join(ROOT, "paper_2609_33437_amd")

PROGRAM = r"""
#include <stdio.h>
#include <string.h>
#include "smat.h"

#define EXPECT(cond) do { if (!(cond)) { printf("FAIL line %d: %s\n", __LINE__, #cond); return 1; } } while (0)

int main(void) {
  smat_op_params p = {1.0f, 0.5f, 0.0f, 1, SMAT_NOISE_GAUSSIAN};
  smat_rng_key k = {7u, 3u, 1u, 0u};
  smat_plan* plan = NULL;
  smat_tensor_desc d;
  memset(&d, 0, sizeof d);
  /* a negative element count is refused before anything is enqueued */
  EXPECT(smat_simulate(NULL, NULL, SMAT_BF16, NULL, SMAT_BF16, -1, p, k, NULL) == SMAT_ERR_INVALID);
  EXPECT(strlen(smat_last_error()) > 0);
  /* an unknown dtype */
  EXPECT(smat_backward_accum(NULL, (smat_dtype)7, NULL, 4, p, 1.0f, k, NULL) == SMAT_ERR_DTYPE);
  /* keep outside [0, 1] */
  p.keep = 1.5f;
  EXPECT(smat_simulate(NULL, NULL, SMAT_BF16, NULL, SMAT_BF16, 4, p, k, NULL) == SMAT_ERR_INVALID);
  EXPECT(strstr(smat_last_error(), "keep") != NULL);
  p.keep = 0.5f;
  /* n == 0 is a valid no-op */
  EXPECT(smat_simulate(NULL, NULL, SMAT_BF16, NULL, SMAT_BF16, 0, p, k, NULL) == SMAT_OK);
  /* plans: a bad count, then a valid host-only plan that has no workspace yet */
  EXPECT(smat_plan_create(&d, -1, SMAT_BF16, SMAT_BF16, SMAT_BF16, 0, &plan) == SMAT_ERR_INVALID);
  EXPECT(plan == NULL);
  EXPECT(smat_plan_create(&d, 1, SMAT_BF16, SMAT_BF16, SMAT_BF16, 0, &plan) == SMAT_OK);
  size_t bytes = 0;
  EXPECT(smat_plan_workspace_bytes(plan, &bytes) == SMAT_OK && bytes >= 256);
  EXPECT(smat_simulate_multi(plan, 7u, 3u, NULL) == SMAT_ERR_STATE);
  EXPECT(smat_switch_storage(plan, 5, NULL) == SMAT_ERR_INVALID);
  EXPECT(smat_plan_clear_grads(plan, 3) == SMAT_OK);
  EXPECT(smat_plan_destroy(plan) == SMAT_OK);
  EXPECT(smat_plan_destroy(NULL) == SMAT_OK);
  printf("ok\n");
  return 0;
}
"""


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc is needed to build the C consumer")
def test_c_program_against_the_library(tmp_path):
    smat.lib()                                   # the library is built and loads
    src = tmp_path / "consumer.c"
    src.write_text(PROGRAM)
    exe = tmp_path / "consumer"
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include", str(src),
           "-L", LIBDIR, "-lsmat", f"-Wl,-rpath,{LIBDIR}", "-o", str(exe)]
    build = subprocess.run(cmd, capture_output=True, text=True)
    assert build.returncode == 0, build.stderr
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert run.returncode == 0 and run.stdout.strip() == "ok", run.stdout + run.stderr
