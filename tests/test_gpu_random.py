"""GPU parity on seeded random configurations.

Each case draws, from its own seed, a batch of 1-4 sequences with random
prefix, speech and suffix lengths (empty spans included), a window of 1-9
frames, a layer below or above l0, a group size, head size, element type,
page size, mask mode, gate scale, split count and how far decode's host
bound on the cache length exceeds the longest cache, and runs pool -> prefill
-> decode steps through the C ABI against the fp64 oracle (tests/gpu_case.py).
A second set draws multi-run sequences (segment tables) and checks pooling
and prefill against the multi-run oracle; a third draws cases for the two
backward calls (attention and pooling), one-run and multi-run.  The draws are
fixed by the seeds, so every run checks the same cases.
"""
import numpy as np
import pytest
import torch

from gpu_case import Case, run_and_check
from test_gpu_bwd import check_attention_bwd, check_pool_bwd
from test_gpu_segments import check as check_segments
from test_gpu_segments import check_backward as check_segments_backward

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


def draw_case(seed: int) -> Case:
    r = np.random.default_rng(1000 + seed)
    B = int(r.integers(1, 5))
    G = int(r.choice([1, 2, 4, 8]))
    Hkv = int(r.choice([1, 2])) if G < 8 else 1
    D = int(r.choice([64, 128]))
    dtype = "bf16" if r.random() < 0.75 else "f32"
    P = [int(r.integers(0, 40)) for _ in range(B)]
    T = [int(r.integers(0, 300)) for _ in range(B)]
    N = [int(r.integers(0, 30)) for _ in range(B)]
    if sum(P) + sum(T) + sum(N) == 0:
        T[0] = 17
    layer, l0 = (1, 0) if r.random() < 0.8 else (2, 5)
    return Case(P=P, T=T, N=N, w=int(r.integers(1, 10)), layer=layer, l0=l0, Hq=G * Hkv, Hkv=Hkv,
                D=D, dtype=dtype, page_size=int(r.choice([8, 16, 32, 64])), mode=int(r.integers(0, 2)),
                decode_steps=2, seed=seed, gate_scale=float(r.choice([0.5, 1.0, 4.0])),
                num_splits=int(r.choice([0, 0, 1, 3])), zero_gate=bool(r.random() < 0.1),
                bound_slack=int(r.choice([0, 0, 3, 50])))


@pytest.mark.parametrize("seed", range(24))
def test_random_case_matches_oracle(seed):
    case = draw_case(seed)
    print(f"seed {seed}: {case}", flush=True)
    run_and_check(case)


def draw_segments(seed: int):
    r = np.random.default_rng(2000 + seed)
    B = int(r.integers(1, 4))
    segs = []
    for _ in range(B):
        n = int(r.integers(0, 6))
        segs.append([(int(r.integers(0, 12)), int(r.integers(0, 80))) for _ in range(n)])
    if all(sum(t + s for t, s in x) == 0 for x in segs):
        segs[0] = [(3, 20)]
    G = int(r.choice([1, 2, 4]))
    kw = dict(Hq=2 * G, Hkv=2, D=int(r.choice([64, 128])),
              dtype="bf16" if r.random() < 0.75 else "f32", page_size=int(r.choice([8, 16, 64])),
              w=int(r.integers(1, 9)), mode=int(r.integers(0, 2)), seed=seed)
    return segs, kw


@pytest.mark.parametrize("seed", range(12))
def test_random_segments_match_oracle(seed):
    segs, kw = draw_segments(seed)
    print(f"seed {seed}: {segs} {kw}", flush=True)
    check_segments(segs, **kw)


def draw_bwd_case(seed: int) -> Case:
    """A one-run case for the backward calls; every sequence has a row."""
    r = np.random.default_rng(3000 + seed)
    B = int(r.integers(1, 4))
    G = int(r.choice([1, 2, 4, 8]))
    Hkv = int(r.choice([1, 2])) if G < 8 else 1
    P = [int(r.integers(0, 30)) for _ in range(B)]
    T = [int(r.integers(0, 200)) for _ in range(B)]
    N = [int(r.integers(0, 20)) for _ in range(B)]
    for b in range(B):
        if P[b] + T[b] + N[b] == 0:
            T[b] = 9
    layer, l0 = (1, 0) if r.random() < 0.8 else (2, 5)
    return Case(P=P, T=T, N=N, w=int(r.integers(1, 10)), layer=layer, l0=l0, Hq=G * Hkv, Hkv=Hkv,
                D=int(r.choice([64, 128])), dtype="bf16" if r.random() < 0.75 else "f32",
                page_size=int(r.choice([8, 16, 64])), mode=int(r.integers(0, 2)), seed=seed,
                gate_scale=float(r.choice([0.5, 1.0, 4.0])), zero_gate=bool(r.random() < 0.1))


@pytest.mark.parametrize("seed", range(12))
def test_random_attention_bwd_matches_oracle(seed):
    case = draw_bwd_case(seed)
    print(f"seed {seed}: {case}", flush=True)
    check_attention_bwd(case)


@pytest.mark.parametrize("seed", range(12))
def test_random_pool_bwd_matches_oracle(seed):
    case = draw_bwd_case(seed)
    print(f"seed {seed}: {case}", flush=True)
    check_pool_bwd(case)


@pytest.mark.parametrize("seed", range(8))
def test_random_segments_backward_matches_oracle(seed):
    segs, kw = draw_segments(100 + seed)
    print(f"seed {seed}: {segs} {kw}", flush=True)
    check_segments_backward(segs, **kw)
