"""include/avtp.h as a plain C99 header: a C program that includes it, links
libavtp.so and calls the host-side entry points (the ABI version, the status
strings, the workspace query, and argument errors that are returned before
any HIP call) compiles with -std=c99 -pedantic -Werror and runs on a machine
without a GPU.  The boundary then needs neither Python nor torch."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIBDIR = os.path.join(ROOT, "paper_2608_26806_amd")

PROGRAM = r"""
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "avtp.h"

/* one sequence: 2 text tokens, an image of 5 tokens, 1 text token */
static const int32_t cu_seqlens[] = {0, 8}, img_start[] = {2}, img_len[] = {5},
                     cu_img[] = {0, 1}, text_pos[] = {0, 1, 7}, cu_text[] = {0, 3},
                     keep_total[] = {2};
static int32_t dev_stand_in[8]; /* never dereferenced by the host checks */

static avtp_layout make_layout(void) {
  avtp_layout L;
  memset(&L, 0, sizeof L);
  L.B = 1;
  L.n_img = 1;
  L.N_tok = 8;
  L.T_tot = 3;
  L.cu_seqlens = L.img_start = L.img_len = L.cu_img = L.text_pos = L.cu_text = L.keep_total =
      dev_stand_in;
  L.h_cu_seqlens = cu_seqlens;
  L.h_img_start = img_start;
  L.h_img_len = img_len;
  L.h_cu_img = cu_img;
  L.h_text_pos = text_pos;
  L.h_cu_text = cu_text;
  L.h_keep_total = keep_total;
  return L;
}

int main(void) {
  int fails = 0;
  avtp_layout L = make_layout();
  const int codes[] = {AVTP_OK, AVTP_ERR_INVALID_ARG, AVTP_ERR_UNSUPPORTED, AVTP_ERR_INFEASIBLE,
                       AVTP_ERR_WORKSPACE, AVTP_ERR_HIP};
  size_t i;
  for (i = 0; i < sizeof codes / sizeof codes[0]; ++i) {
    const char *s = avtp_status_string(codes[i]);
    if (!s || !s[0]) ++fails;
  }
  if (avtp_version() <= 0) ++fails;
  /* the score workspace of a valid layout is a host computation */
  if (avtp_score_workspace_size(&L, AVTP_SCORE_ATTN, AVTP_BF16, 8, 2, 128) == 0) ++fails;
  /* unsupported head size and an invalid layout: 0 bytes */
  if (avtp_score_workspace_size(&L, AVTP_SCORE_ATTN, AVTP_BF16, 8, 2, 96) != 0) ++fails;
  if (avtp_score_workspace_size(NULL, AVTP_SCORE_ATTN, AVTP_BF16, 8, 2, 128) != 0) ++fails;
  /* argument errors come back before any HIP call */
  if (avtp_budget(NULL, NULL, NULL, AVTP_BUDGET_PROPORTIONAL, 1.f, 50, 950, 0, NULL, NULL) !=
      AVTP_ERR_INVALID_ARG)
    ++fails;
  if (avtp_budget(NULL, &L, NULL, AVTP_BUDGET_PROPORTIONAL, 1.f, 50, 950, 0, NULL, NULL) !=
      AVTP_ERR_INVALID_ARG)
    ++fails;
  {
    avtp_layout bad = make_layout();
    static const int32_t bad_start[] = {1}; /* the image overlaps text token 1 */
    bad.h_img_start = bad_start;
    if (avtp_score_workspace_size(&bad, AVTP_SCORE_ATTN, AVTP_BF16, 8, 2, 128) != 0) ++fails;
  }
  printf("fails=%d\n", fails);
  return fails != 0;
}
"""


def test_header_is_c99_and_links_from_c(tmp_path):
    cc = shutil.which("gcc") or shutil.which("cc")
    lib = os.path.join(LIBDIR, "libavtp.so")
    if cc is None:
        pytest.skip("no C compiler")
    if not os.path.exists(lib):
        pytest.skip("libavtp.so is not built")
    src = tmp_path / "use_avtp.c"
    src.write_text(PROGRAM)
    exe = tmp_path / "use_avtp"
    r = subprocess.run([cc, "-std=c99", "-pedantic", "-Wall", "-Wextra", "-Werror",
                        "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe),
                        "-L", LIBDIR, "-lavtp", "-Wl,-rpath," + LIBDIR],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and "fails=0" in r.stdout, r.stdout + r.stderr
