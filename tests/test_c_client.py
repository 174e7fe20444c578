"""The boundary from C: a plain C11 program includes include/speechkv.h
(warnings as errors), links libspeechkv.so and calls the host helpers and an
invalid decode (rejected before any HIP work), so no GPU is needed.  The
header also compiles as C++."""
import os
import shutil
import subprocess

import pytest

from paper_2607_06827_amd import speechkv as skv

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
INCLUDE = os.path.join(ROOT, "include")
LIBDIR = os.path.join(ROOT, "paper_2607_06827_amd")

PROGRAM = r"""
#include <stdio.h>
#include <string.h>
#include "speechkv.h"

int main(void) {
  speechkv_paged_kv cache;
  int st;
  printf("version %s\n", speechkv_version());
  printf("clen %d\n", (int)speechkv_compressed_len(32, 750, 0, 4, 14, 14));
  printf("splits %d\n", (int)speechkv_decode_num_splits(16, 8, 2163));
  printf("ws %zu\n", speechkv_decode_workspace_bytes(16, 16, 8, 128, 2163, 0));
  memset(&cache, 0, sizeof cache);
  st = speechkv_decode_attn(NULL, 1, 1, &cache, NULL, 0, NULL, NULL, 1.0f, 0, NULL, NULL, 0, NULL);
  printf("decode %d %s\n", st, speechkv_status_string(st));
  return 0;
}
"""


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_c_program_links_and_calls_the_library(tmp_path):
    src, exe = tmp_path / "client.c", tmp_path / "client"
    src.write_text(PROGRAM)
    subprocess.run(["gcc", "-std=c11", "-Wall", "-Wextra", "-Werror", "-pedantic", f"-I{INCLUDE}",
                    str(src), f"-L{LIBDIR}", "-lspeechkv", f"-Wl,-rpath,{LIBDIR}", "-o", str(exe)],
                   check=True, capture_output=True, text=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True, timeout=120).stdout
    got = dict(line.split(" ", 1) for line in out.strip().splitlines())
    assert got["version"] == skv.speechkv_version()
    assert int(got["clen"]) == 32 + 188 == skv.speechkv_compressed_len(32, 750, 0, 4, 14, 14)
    assert int(got["splits"]) == skv.speechkv_decode_num_splits(16, 8, 2163)
    assert int(got["ws"]) == skv.speechkv_decode_workspace_bytes(16, 16, 8, 128, 2163, 0) > 0
    assert got["decode"] == f"{skv.ERR_INVALID_ARG} invalid argument"


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_header_compiles_as_cxx(tmp_path):
    src = tmp_path / "client.cc"
    src.write_text('#include "speechkv.h"\nint main() { return speechkv_version() == nullptr; }\n')
    subprocess.run(["g++", "-std=c++17", "-Wall", "-Wextra", "-Werror", "-pedantic", f"-I{INCLUDE}",
                    "-fsyntax-only", str(src)], check=True, capture_output=True, text=True)
