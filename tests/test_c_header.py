"""The boundary is a C ABI: include/rgd.h compiles as C99 on its own, and a
plain C program links against the built library and calls the entry points
that need no GPU (version, last error, workspace size, argument validation)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB_DIR = os.path.join(ROOT, "paper_2607_20791_amd")

PROGRAM = r"""
#include <stdio.h>
#include <string.h>
#include "rgd.h"

int main(void) {
  const char* v = rgd_version();
  if (!v || !v[0]) return 1;
  /* argument validation happens before any HIP call */
  if (rgd_kernel_argmax(NULL, 2, 8, NULL, NULL, NULL) != RGD_E_INVALID_ARG) return 2;
  if (strlen(rgd_last_error()) == 0) return 3;
  if (rgd_sampler_workspace_bytes(0, 8) != 0) return 4;
  if (rgd_sampler_workspace_bytes(4, 152064) == 0) return 5;
  if (rgd_gate(NULL, NULL, 1, NULL, NULL, NULL, NULL) != RGD_E_INVALID_ARG) return 6;
  printf("%s\n", v);
  return 0;
}
"""


def _cc():
    return shutil.which("gcc") or shutil.which("cc")


@pytest.mark.skipif(_cc() is None, reason="no C compiler")
def test_header_is_c99(tmp_path):
    src = tmp_path / "h.c"
    src.write_text('#include "rgd.h"\nint main(void) { return RGD_OK; }\n')
    r = subprocess.run([_cc(), "-std=c99", "-Wall", "-Werror", "-pedantic", "-fsyntax-only",
                        "-I", os.path.join(ROOT, "include"), str(src)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


@pytest.mark.skipif(_cc() is None, reason="no C compiler")
def test_plain_c_program_links_and_runs(tmp_path):
    lib = os.path.join(LIB_DIR, "librgd.so")
    if not os.path.exists(lib):
        pytest.skip("library not built")
    src = tmp_path / "p.c"
    src.write_text(PROGRAM)
    exe = tmp_path / "p"
    r = subprocess.run([_cc(), "-std=c99", "-Wall", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe),
                        "-L", LIB_DIR, "-lrgd", "-Wl,-rpath," + LIB_DIR], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, (r.returncode, r.stdout, r.stderr)
    assert r.stdout.strip()
