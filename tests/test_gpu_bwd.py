"""GPU parity of the training backward through the C ABI (Sec. III-C: the
pooling of Eq. 4 and the attention of Eq. 5 are optimised jointly).

Each stage is compared element by element with the fp64 oracle on that
stage's own inputs:
  - speechkv_prefill_attn_bwd against oracle.attention_bwd evaluated on the
    GPU's cache contents (the bf16 K^/V^ the kernel reads) and the same q and
    dO; the kernel uses the forward's stored output and LSE, as in training;
  - speechkv_pool_kv_bwd against oracle.pool_bwd on the same raw K/V, gate and
    fp32 dK^/dV^.
The whole chain is then checked end to end (dQ, raw dK, raw dV and du)
against the all-fp64 oracle chain, and for the invariant that a window's
raw-key gradients add up to its pooled gradient.  The benchmark's training
layer (1596 rows over 471 keys, 8 sequences, 16/8 heads) is checked in its own
launch configuration.  Tolerances: tests/helpers.py GRAD_TOL.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from gpu_case import Case, build
from helpers import GRAD_TOL, f64, gather, grad_err
from paper_2607_06827_amd import inputs
from paper_2607_06827_amd import speechkv as skv
from paper_2607_06827_amd.workload import TrainJob

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

CASES = {
    "bf16-d128": Case(P=[8, 3], T=[60, 37], N=[5, 9], D=128, Hq=4, Hkv=2),
    "bf16-d64-g1": Case(P=[6], T=[45], N=[3], D=64, Hq=2, Hkv=2),
    "f32-d64": Case(P=[8], T=[60], N=[4], D=64, dtype="f32"),
    "window-start-mask": Case(P=[3, 9], T=[41, 30], N=[2, 7], mode=1, D=128),
    "identity-below-l0": Case(P=[6], T=[50], N=[4], layer=2, l0=5, D=128),
    "prefix-empty": Case(P=[0, 0], T=[37, 9], N=[3, 0], w=4, D=128),
    "gqa-g4": Case(P=[5], T=[70], N=[6], Hq=8, Hkv=2, D=128),
    "gqa-g8": Case(P=[5], T=[33], N=[2], Hq=8, Hkv=1, D=64),
    "gqa-g8-d64-tiles": Case(P=[5, 2], T=[300, 90], N=[8, 4], Hq=16, Hkv=2, D=64),
    "w8": Case(P=[4, 2], T=[77, 64], N=[6, 1], w=8, D=128),
    "w12-three-groups": Case(P=[1], T=[61], N=[2], w=12, D=64),
    "zero-gate": Case(P=[4], T=[70], N=[3], zero_gate=True, D=128),
    "sharp-gate": Case(P=[4], T=[70], N=[3], gate_scale=10.0, D=128),
    "page64": Case(P=[5, 2], T=[77, 64], N=[6, 1], page_size=64, w=5, D=128),
    "varlen": Case(P=[0, 17, 3, 40], T=[150, 7, 91, 0], N=[9, 33, 0, 1], w=3, D=128, Hq=8, Hkv=2),
    "long-rows": Case(P=[32], T=[750], N=[16], D=128, Hq=4, Hkv=2),
    # 26 (sequence, KV head) pairs of 11 key blocks: 286 dK/dV blocks, more
    # than 32 per XCD and pairs that straddle the XCD ranges, so the key
    # blocks of some pairs run in descending order
    "dkdv-grid-rounds": Case(P=[9, 3, 17, 0, 5, 11, 2, 8, 14, 6, 1, 12, 4],
                             T=[660, 655, 640, 670, 650, 645, 665, 652, 648, 661, 657, 643, 668],
                             N=[5, 12, 3, 8, 0, 9, 6, 2, 11, 4, 7, 10, 1], layer=2, l0=5, D=128,
                             Hq=2, Hkv=2),
}


def forward(case, x):
    """pool -> prefill on the GPU; returns (out, lse) and fills the cache."""
    B, Hq, D = case.B, case.Hq, case.D
    skv.speechkv_pool_kv(x["t"](x["k_raw"]), x["t"](x["v_raw"]), x["spans"], case.w,
                         x["t"](x["u"]), case.layer, case.l0, x["cache"])
    out = torch.full((B, x["S"], Hq, D), float("nan"), dtype=x["dt"], device=x["dev"])
    lse = torch.full((B, Hq, x["S"]), float("nan"), dtype=torch.float32, device=x["dev"])
    skv.speechkv_prefill_attn(x["t"](x["q"]), x["cache"], x["spans"], case.w, case.layer, case.l0,
                              out, mask_mode=case.mode, scale=D ** -0.5, lse=lse)
    return out, lse


def attention_bwd(case, x, out, lse, dout, cap):
    B, Hq, Hkv, D = case.B, case.Hq, case.Hkv, case.D
    dq = torch.full_like(out, float("nan"))
    dk = torch.full((B, cap, Hkv, D), float("nan"), dtype=torch.float32, device=x["dev"])
    dv = torch.full_like(dk, float("nan"))
    ws = torch.empty(skv.speechkv_prefill_attn_bwd_workspace_bytes(B, Hq, x["S"]), dtype=torch.uint8,
                     device=x["dev"])
    skv.speechkv_prefill_attn_bwd(x["t"](x["q"]), x["cache"], x["spans"], case.w, case.layer, case.l0,
                                  out, lse, dout, dq, dk, dv, ws, mask_mode=case.mode, scale=D ** -0.5)
    return dq, dk, dv


@pytest.mark.parametrize("name", list(CASES))
def test_attention_bwd_matches_oracle(name):
    print(f"case {name}", flush=True)
    check_attention_bwd(CASES[name])


def check_attention_bwd(case):
    x = build(case)
    B, Hq, Hkv, D = case.B, case.Hq, case.Hkv, case.D
    out, lse = forward(case, x)
    dout = inputs.normal((B, x["S"], Hq, D), case.seed * 1000 + 8, dtype=x["dt"]).to(x["dev"])
    cap = max(x["clen"]) + 3
    dq, dk, dv = attention_bwd(case, x, out, lse, dout, cap)
    torch.cuda.synchronize()
    tol = GRAD_TOL[case.dtype]
    for b in range(B):
        L = x["clen"][b]
        R = case.P[b] + case.T[b] + case.N[b]
        # the oracle on the GPU's cache rows (the bf16 K^/V^ the kernel reads)
        gk, gv = gather(x["cache"], b, L)
        kh, vh = f64(gk)[None], f64(gv)[None]
        rq, rk, rv = oracle.attention_bwd(f64(x["q"][b:b + 1]), kh, vh, [case.P[b]], [case.T[b]],
                                          [case.N[b]], case.w, case.layer, case.l0,
                                          f64(dout[b:b + 1]), case.mode, D ** -0.5)
        e = {"dq": grad_err(f64(dq[b, :R]), rq[0, :R]), "dk": grad_err(f64(dk[b, :L]), rk[0, :L]),
             "dv": grad_err(f64(dv[b, :L]), rv[0, :L])}
        print(f"  seq {b}: " + " ".join(f"{k} {v:.2e}" for k, v in e.items()), flush=True)
        assert e["dq"] <= tol["dq"] and e["dk"] <= tol["dkv_hat"] and e["dv"] <= tol["dkv_hat"]
        # rows that see no key get exactly 0; rows past the sequence are not written
        seen = np.isfinite(f64(lse[b, :, :R]))  # [Hq, R]
        for h in range(Hq):
            assert not torch.any(dq[b, :R][torch.from_numpy(~seen[h]), h].cpu() != 0)
        assert torch.isnan(dq[b, R:]).all()
        assert torch.isnan(dk[b, L:]).all() and torch.isnan(dv[b, L:]).all()


POOL_CASES = {k: CASES[k] for k in ("bf16-d128", "bf16-d64-g1", "f32-d64", "identity-below-l0",
                                     "prefix-empty", "w8", "w12-three-groups", "zero-gate",
                                     "sharp-gate", "varlen", "long-rows")}
# 64 sequences of 17 pooling-backward blocks each: 1088 gate partials, more
# than the 1024 that one round of the gate-gradient sum's threads takes
POOL_CASES["many-partials"] = Case(P=[(7 * i) % 23 for i in range(64)],
                                   T=[1000 - (13 * i) % 37 for i in range(64)],
                                   N=[(5 * i) % 11 for i in range(64)], w=2, D=64, Hq=2, Hkv=1)


def pool_bwd(case, x, dkh, dvh, with_du=True):
    B, Hkv, D = case.B, case.Hkv, case.D
    k, v = x["t"](x["k_raw"]), x["t"](x["v_raw"])
    dkr = torch.full_like(k, float("nan"))
    dvr = torch.full_like(v, float("nan"))
    du = torch.full((Hkv, D), float("nan"), dtype=torch.float32, device=x["dev"]) if with_du else None
    nbytes = skv.speechkv_pool_kv_bwd_workspace_bytes(B, x["spans"].max_total_len, Hkv, D)
    ws = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=x["dev"]) if with_du else None
    skv.speechkv_pool_kv_bwd(k, v, x["spans"], case.w, x["t"](x["u"]), case.layer, case.l0, dkh, dvh,
                             dkr, dvr, du, ws)
    return dkr, dvr, du


@pytest.mark.parametrize("name", list(POOL_CASES))
def test_pool_bwd_matches_oracle(name):
    print(f"case {name}", flush=True)
    check_pool_bwd(POOL_CASES[name])


def check_pool_bwd(case):
    x = build(case)
    B, Hkv, D = case.B, case.Hkv, case.D
    cap = max(x["clen"]) + 2
    dkh = inputs.normal((B, cap, Hkv, D), case.seed * 1000 + 9).to(x["dev"])
    dvh = inputs.normal((B, cap, Hkv, D), case.seed * 1000 + 10).to(x["dev"])
    dkr, dvr, du = pool_bwd(case, x, dkh, dvh)
    torch.cuda.synchronize()
    u64 = None if x["u"] is None else f64(x["u"])
    rk, rv, ru = oracle.pool_bwd(f64(x["k_raw"]), f64(x["v_raw"]), case.P, case.T, case.N, case.w,
                                 case.layer, case.l0, u64, f64(dkh), f64(dvh))
    tol = GRAD_TOL[case.dtype]
    for b in range(B):
        R = case.P[b] + case.T[b] + case.N[b]
        e = (grad_err(f64(dkr[b, :R]), rk[b, :R]), grad_err(f64(dvr[b, :R]), rv[b, :R]))
        print(f"  seq {b}: dk {e[0]:.2e} dv {e[1]:.2e}", flush=True)
        assert max(e) <= tol["dkv_raw"]
        assert torch.isnan(dkr[b, R:]).all() and torch.isnan(dvr[b, R:]).all()
        # text rows take their slot's gradient, rounded once
        P, nW = case.P[b], x["clen"][b] - case.P[b] - case.N[b]
        assert torch.equal(dkr[b, :P], dkh[b, :P].to(x["dt"]))
        assert torch.equal(dvr[b, P + case.T[b]:R], dvh[b, P + nW:P + nW + case.N[b]].to(x["dt"]))
    eu = grad_err(f64(du), ru)
    print(f"  du {eu:.2e}", flush=True)
    assert eu <= tol["du"]
    if case.layer < case.l0:  # the identity: every raw row takes its slot's gradient, du = 0
        for b in range(B):
            R = case.P[b] + case.T[b] + case.N[b]
            assert torch.equal(dkr[b, :R], dkh[b, :R].to(x["dt"]))
        assert not torch.any(du != 0)


def test_pool_bwd_without_gate_gradient_and_determinism():
    case = CASES["varlen"]
    x = build(case)
    cap = max(x["clen"])
    dkh = inputs.normal((case.B, cap, case.Hkv, case.D), 11).to(x["dev"])
    dvh = inputs.normal((case.B, cap, case.Hkv, case.D), 12).to(x["dev"])
    a = pool_bwd(case, x, dkh, dvh)
    b = pool_bwd(case, x, dkh, dvh)
    c = pool_bwd(case, x, dkh, dvh, with_du=False)
    torch.cuda.synchronize()
    bits = lambda t: t.view({2: torch.int16, 4: torch.int32}[t.element_size()])
    for p, q in zip(a, b):  # bit for bit, the gate gradient included
        assert torch.equal(bits(p), bits(q))
    # skipping the gate gradient changes nothing else
    assert torch.equal(bits(a[0]), bits(c[0])) and torch.equal(bits(a[1]), bits(c[1])) and c[2] is None


def test_attention_bwd_is_deterministic():
    case = CASES["gqa-g4"]
    x = build(case)
    out, lse = forward(case, x)
    dout = inputs.normal((case.B, x["S"], case.Hq, case.D), 13, dtype=x["dt"]).to(x["dev"])
    r1 = attention_bwd(case, x, out, lse, dout, max(x["clen"]))
    r2 = attention_bwd(case, x, out, lse, dout, max(x["clen"]))
    torch.cuda.synchronize()
    assert torch.equal(r1[0].view(torch.int16), r2[0].view(torch.int16))
    assert torch.equal(r1[1].view(torch.int32), r2[1].view(torch.int32))
    assert torch.equal(r1[2].view(torch.int32), r2[2].view(torch.int32))


@pytest.mark.parametrize("name", ["bf16-d128", "f32-d64", "w8"])
def test_training_step_end_to_end(name):
    """pool -> prefill -> prefill backward -> pool backward, all on the GPU:
    dQ against the all-fp64 oracle chain, and each window's raw-key
    gradients adding up to its pooled gradient (any gate)."""
    case = CASES[name]
    x = build(case)
    B, Hq, Hkv, D = case.B, case.Hq, case.Hkv, case.D
    out, lse = forward(case, x)
    dout = inputs.normal((B, x["S"], Hq, D), case.seed * 1000 + 14, dtype=x["dt"]).to(x["dev"])
    cap = max(x["clen"])
    dq, dkh, dvh = attention_bwd(case, x, out, lse, dout, cap)
    dkr, dvr, du = pool_bwd(case, x, dkh, dvh)
    torch.cuda.synchronize()
    u64 = None if x["u"] is None else f64(x["u"])
    kh, vh, _ = oracle.pool(f64(x["k_raw"]), f64(x["v_raw"]), case.P, case.T, case.N, case.w,
                            case.layer, case.l0, u64, cap)
    rq, rkh, rvh = oracle.attention_bwd(f64(x["q"]), kh, vh, case.P, case.T, case.N, case.w,
                                        case.layer, case.l0, f64(dout), case.mode, D ** -0.5)
    rk, rv, ru = oracle.pool_bwd(f64(x["k_raw"]), f64(x["v_raw"]), case.P, case.T, case.N, case.w,
                                 case.layer, case.l0, u64, rkh, rvh)
    tol = GRAD_TOL[case.dtype]
    w_eff = case.w if case.layer >= case.l0 else 1
    for b in range(B):
        R = case.P[b] + case.T[b] + case.N[b]
        e = {"dq": grad_err(f64(dq[b, :R]), rq[b, :R]),
             "dk": grad_err(f64(dkr[b, :R]), rk[b, :R]),
             "dv": grad_err(f64(dvr[b, :R]), rv[b, :R])}
        print(f"  seq {b} vs the fp64 chain: " + " ".join(f"{k} {v:.2e}" for k, v in e.items()),
              flush=True)
        assert e["dq"] <= tol["dq"]
        assert e["dk"] <= tol["chain"] and e["dv"] <= tol["chain"]
        sums = np.zeros((x["clen"][b], Hkv, D))
        gk = f64(dkr[b, :R])
        for i in range(-(-case.T[b] // w_eff)):
            a0 = case.P[b] + i * w_eff
            a1 = min(a0 + w_eff, case.P[b] + case.T[b])
            sums[case.P[b] + i] = gk[a0:a1].sum(0)
        P = case.P[b]
        nW = x["clen"][b] - P - case.N[b]
        ref = f64(dkh[b, P:P + nW])
        # each frame gradient is rounded once (2^-9 of its size at bf16)
        assert np.max(np.abs(sums[P:P + nW] - ref)) <= (1e-2 if case.dtype == "bf16" else 1e-5) * \
            max(1.0, np.max(np.abs(gk)))
    eu = grad_err(f64(du), ru)
    print(f"  du vs the fp64 chain {eu:.2e}", flush=True)
    assert eu <= tol["chain"]


def test_training_backward_at_benched_shape():
    """The training layer the benchmark times (workload.TrainJob on the 1596-row
    workload: 8 sequences, 32 + 1500 + 64 rows over 471 keys, 16/8 heads,
    d = 128, w = 4), run in that launch configuration.  Attention backward on
    sequences 0, 3 and 7 against the oracle over the GPU's cache rows; pooling
    backward on the whole batch (du sums over every sequence) against the
    oracle on the GPU's dK^/dV^."""
    wl = inputs.PREFILL_1500
    tj = TrainJob(wl)
    tj.run_forward()
    tj.run_backward()
    torch.cuda.synchronize()
    f = tj.fwd
    tol = GRAD_TOL["bf16"]
    P, T, N, R, L = wl.prefix_len, wl.speech_len, wl.suffix_len, wl.prefill_len, tj.clen
    assert L == 471
    for b in (0, 3, 7):
        gk, gv = gather(f.caches[0], b, L)
        rq, rk, rv = oracle.attention_bwd(f64(f.q_prefill[0][b:b + 1]), f64(gk)[None],
                                          f64(gv)[None], [P], [T], [N], tj.w, tj.layer, f.l0,
                                          f64(tj.dout[b:b + 1]), 0, f.scale)
        e = {"dq": grad_err(f64(tj.dq[b]), rq[0, :R]), "dk": grad_err(f64(tj.dk_hat[b]), rk[0, :L]),
             "dv": grad_err(f64(tj.dv_hat[b]), rv[0, :L])}
        print(f"  seq {b}: " + " ".join(f"{k} {v:.2e}" for k, v in e.items()), flush=True)
        assert e["dq"] <= tol["dq"] and e["dk"] <= tol["dkv_hat"] and e["dv"] <= tol["dkv_hat"]
    B = wl.batch
    rk, rv, ru = oracle.pool_bwd(f64(f.k_raw[0]), f64(f.v_raw[0]), [P] * B, [T] * B, [N] * B, tj.w,
                                 tj.layer, f.l0, f64(f.gate[0]), f64(tj.dk_hat), f64(tj.dv_hat))
    ek = grad_err(f64(tj.dk_raw), rk)
    ev = grad_err(f64(tj.dv_raw), rv)
    eu = grad_err(f64(tj.du), ru)
    print(f"  pooling backward, whole batch: dk {ek:.2e} dv {ev:.2e} du {eu:.2e}", flush=True)
    assert ek <= tol["dkv_raw"] and ev <= tol["dkv_raw"] and eu <= tol["du"]
