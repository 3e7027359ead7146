"""include/cmsd.h is plain C: a C99 program compiled with gcc -Wall -Werror links
against libcmsd.so and gets the host-side answers (version, status strings,
workspace sizes, argument errors returned before any device work).  CPU only."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB_DIR = os.path.join(ROOT, "paper_2508_15371_amd")

PROGRAM = r"""
#include <stdio.h>
#include <string.h>
#include "cmsd.h"

int main(void) {
  int bad = 0;
  cmsd_conf_params cp = {0.25f, 0.25f, 0.5f, 1.0f};
  cmsd_draft_params dp = {1, 8, 1.0f};
  cmsd_verify_params vp = {CMSD_MODE_CM, 3, 0.1f, 1.0f};
  cmsd_row_stats st;
  float x = 0.f;
  int32_t k = 0, off = 0;
  if (cmsd_version() != ((1 << 16) | 7)) bad |= 1;
  if (strcmp(cmsd_status_string(CMSD_OK), "ok") != 0) bad |= 2;
  if (cmsd_verify_workspace_bytes(0, 8, 1000) != 0) bad |= 4;
  if (cmsd_verify_workspace_bytes(4, 8, 1000) == 0) bad |= 8;
  /* argument errors come back before anything is enqueued */
  if (cmsd_confidence(&x, 7, 1, 100, 100, &cp, &st, NULL) != CMSD_ERR_DTYPE) bad |= 16;
  if (cmsd_confidence(&x, CMSD_F32, 1, 1, 1, &cp, &st, NULL) != CMSD_ERR_ARG) bad |= 32;
  if (cmsd_confidence(&x, CMSD_F32, 0, 100, 100, &cp, &st, NULL) != CMSD_OK) bad |= 64;
  dp.k_min = 9;
  if (cmsd_draft_len(&st, 1, &dp, &k, &off, NULL) != CMSD_ERR_ARG) bad |= 128;
  vp.mode = 7;
  if (cmsd_verify(&x, 100, &st, &x, 100, 9, &off, &k, &k, &x, CMSD_F32, 1, 8, 100, &vp, NULL, &k, &k,
                  &x, 1, NULL) != CMSD_ERR_ARG) bad |= 256;
  if (cmsd_draft_sample_workspace_bytes(3, 1) != 0) bad |= 512;
  if (cmsd_logit_pass_fused_workspace_bytes(4, 8, 1000) != cmsd_verify_workspace_bytes(4, 8, 1000) + 16) bad |= 1024;
  if (cmsd_logit_pass_fused(&x, 100, &x, 100, &k, &x, 9, 1, 8, 100, &cp, &dp, &vp, 0, &st, &k, NULL, &k, &k, &x,
                            1 << 20, NULL) != CMSD_ERR_DTYPE) bad |= 2048;
  /* the no-allocation pass: its scratch bound is checked on the host */
  dp.k_min = 1;
  dp.k_max = 16;
  vp.mode = CMSD_MODE_CM;
  if (cmsd_logit_pass_noalloc(&x, 128256, &x, 128256, &k, &x, CMSD_BF16, 4096, 16, 128256, &cp, &dp, &vp, 0, &st,
                              &k, NULL, &k, &k, NULL) != CMSD_ERR_ARG) bad |= 4096;  /* target_stats NULL */
  if (cmsd_verify_workspace_bytes(4096, 16, 128256) <= CMSD_STATIC_SCRATCH_BYTES) bad |= 8192;
  if (cmsd_set_row_shape(48, 0) != CMSD_ERR_ARG || cmsd_set_row_shape(0, 0) != CMSD_OK) bad |= 16384;
  if (cmsd_set_pass_decisions(3) != CMSD_ERR_ARG || cmsd_set_pass_decisions(0) != CMSD_OK) bad |= 32768;
  {
    void* half[2] = {&x, NULL};
    if (cmsd_set_row_events(half) != CMSD_ERR_ARG || cmsd_set_row_events(NULL) != CMSD_OK) bad |= 65536;
  }
  if (cmsd_logit_pass(&x, 100, &x, 100, &k, &x, 9, 1, 8, 100, &cp, &dp, &vp, 0, &st, &k, NULL, &k, &k, &x,
                      1 << 20, NULL) != CMSD_ERR_DTYPE) bad |= 131072;
  printf("bad=%d\n", bad);
  return bad;
}
"""


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_header_compiles_as_c99_and_links(tmp_path):
    if not os.path.exists(os.path.join(LIB_DIR, "libcmsd.so")):
        pytest.skip("libcmsd.so is not built")
    src = tmp_path / "abi.c"
    src.write_text(PROGRAM)
    exe = tmp_path / "abi"
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic", "-I", os.path.join(ROOT, "include"),
           str(src), "-L", LIB_DIR, "-lcmsd", "-Wl,-rpath," + LIB_DIR, "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, (r.stdout, r.stderr)
    assert "bad=0" in r.stdout
