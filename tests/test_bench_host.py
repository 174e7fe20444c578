"""Host-side checks of the benchmark script and its streaming-read ceiling
library (no GPU: argument rejection happens before any HIP call)."""
import ctypes
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BENCH_LIB = os.path.join(ROOT, "paper_2607_06827_amd", "libskv_bench.so")


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode != 0
    assert "one GPU" in r.stdout + r.stderr
    assert not any(line.startswith("{") for line in r.stdout.splitlines())


@pytest.fixture(scope="module")
def stream_read():
    if not os.path.exists(BENCH_LIB):
        pytest.skip("libskv_bench.so not built (run __graft_entry__.build())")
    f = ctypes.CDLL(BENCH_LIB).skv_stream_read
    f.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int, ctypes.c_int,
                  ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    f.restype = ctypes.c_int
    return f


@pytest.mark.parametrize("args", [
    (0, 16, 1024, 4, 256, 2, 16),        # null buffer
    (16, 16, 1000, 4, 256, 2, 16),       # not a multiple of 1 KB
    (16, 16, 0, 4, 256, 2, 16),          # empty
    (16, 16, 1024, 0, 256, 2, 16),       # no blocks
    (16, 16, 1024, 4, 96, 2, 16),        # threads not a multiple of 64
    (16, 16, 1024, 4, 2048, 2, 16),      # too many threads
    (16, 16, 1024, 4, 256, 3, 16),       # unsupported depth
    (16, 16, 1024, 4, 256, 2, 0),        # null sink
])
def test_stream_read_rejects_bad_arguments(stream_read, args):
    a, b, n, blocks, threads, depth, sink = args
    assert stream_read(a, b, n, blocks, threads, depth, sink, None) == -1
