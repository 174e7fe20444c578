"""GPU parity on small and adversarial shapes, through the C ABI.

Each case runs pool -> prefill -> decode steps and is compared with the fp64
oracle element by element (tests/gpu_case.py): pooled K/V, prefill outputs and
LSE, every decode output, and the bit-exact text copies and new-token writes.
Sizes span several tiles and a ragged tail while the oracle stays fast.
"""
import pytest
import torch

from gpu_case import Case, run_and_check

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

CASES = {
    # name: Case
    "basic-bf16": Case(P=[8], T=[60], N=[5], D=128, Hq=4, Hkv=2),
    "basic-f32": Case(P=[8], T=[60], N=[5], dtype="f32", D=64),
    "prefix-empty": Case(P=[0, 0], T=[37, 9], N=[3, 0], w=4),          # rows that see nothing
    "speech-shorter-than-w": Case(P=[5], T=[3], N=[4], w=8),
    "no-speech": Case(P=[7], T=[0], N=[6]),
    "no-suffix": Case(P=[4], T=[45], N=[0], w=6),                       # ragged last window
    "window-start-mask": Case(P=[3, 9], T=[41, 30], N=[2, 7], mode=1),
    "identity-below-l0": Case(P=[6], T=[50], N=[4], layer=2, l0=5),
    "w1": Case(P=[6], T=[50], N=[4], w=1),
    "varlen-batch": Case(P=[0, 17, 3, 40], T=[150, 7, 91, 0], N=[9, 33, 0, 1], w=3, D=128,
                         Hq=8, Hkv=2),
    "page8": Case(P=[5, 2], T=[77, 64], N=[6, 1], page_size=8),
    "page64-w5": Case(P=[5, 2], T=[77, 64], N=[6, 1], page_size=64, w=5),
    "identity-pages": Case(P=[9], T=[70], N=[3], shuffle=False),
    "g1": Case(P=[4], T=[70], N=[3], Hq=2, Hkv=2, D=128),
    "g4": Case(P=[4], T=[70], N=[3], Hq=8, Hkv=2, D=128),
    "g8": Case(P=[4], T=[70], N=[3], Hq=8, Hkv=1, D=128),
    "g8-f32-d64": Case(P=[4], T=[70], N=[3], Hq=16, Hkv=2, D=64, dtype="f32"),
    # bf16, 64-wide heads, group 8: half the waves of a prefill block load no
    # tile rows and wait only for their query rows
    "g8-bf16-d64": Case(P=[4, 9], T=[170, 61], N=[3, 12], Hq=16, Hkv=2, D=64),
    "zero-gate": Case(P=[4], T=[70], N=[3], zero_gate=True),
    "sharp-gate-and-queries": Case(P=[4, 1], T=[70, 33], N=[3, 2], gate_scale=10.0, q_scale=3.0,
                                   D=128),
    "long-split": Case(P=[32, 0], T=[1100, 700], N=[10, 0], D=128, Hq=16, Hkv=8, decode_steps=2),
    "forced-splits": Case(P=[32, 5], T=[500, 130], N=[10, 2], D=128, num_splits=7),
    "f32-d128-split": Case(P=[3], T=[400], N=[2], D=128, dtype="f32", num_splits=3),
    # decode's host bound well above every cache length: the batches requested
    # from the bound before the lengths arrive must not be reduced
    "loose-decode-bound": Case(P=[8, 0, 30], T=[300, 45, 9], N=[5, 3, 0], D=128, Hq=8, Hkv=2,
                               bound_slack=200),
    "loose-decode-bound-split": Case(P=[8, 2], T=[300, 45], N=[5, 3], D=128, num_splits=3,
                                     bound_slack=150),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_case_matches_oracle(name):
    print(f"case {name}", flush=True)
    run_and_check(CASES[name])
