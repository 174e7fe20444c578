"""GPU parity of the one-launch pooling + prefill attention
(speechkv_pool_prefill_attn, the on-the-fly pooling of Sec. III-C).

It must leave exactly what speechkv_pool_kv followed by speechkv_prefill_attn
leave: the cache rows, the cache lengths, the outputs and the LSE, bit for
bit (the pooled rows come from the same arithmetic).  It is also compared
with the fp64 oracle directly, on small and adversarial shapes (windows
longer than four frames, ragged windows, empty spans, every group size, both
head sizes and masks, strided raw views) and on full-size workloads.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_case import Case, build
from helpers import TOL, f64, fwd_err, gather
from paper_2607_06827_amd import inputs
from paper_2607_06827_amd import speechkv as skv
from paper_2607_06827_amd.workload import Job

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

CASES = {
    "basic-d128": Case(P=[8], T=[60], N=[5], D=128, Hq=4, Hkv=2),
    "basic-d64": Case(P=[8], T=[60], N=[5], D=64),
    "prefix-empty": Case(P=[0, 0], T=[37, 9], N=[3, 0]),  # rows that see nothing
    "speech-shorter-than-w": Case(P=[5], T=[3], N=[4], w=8),
    "no-speech": Case(P=[7], T=[0], N=[6]),
    "no-suffix-w6": Case(P=[4], T=[45], N=[0], w=6),  # ragged last window, two groups of frames
    "window-start-mask": Case(P=[3, 9], T=[41, 30], N=[2, 7], mode=1),
    "identity-below-l0": Case(P=[6], T=[50], N=[4], layer=2, l0=5),
    "w1": Case(P=[6], T=[50], N=[4], w=1),
    "w16-long-windows": Case(P=[3, 0], T=[200, 77], N=[5, 2], w=16, D=128),
    "w5": Case(P=[2, 11], T=[131, 64], N=[9, 0], w=5, D=128, Hq=8, Hkv=4),
    "varlen-batch": Case(P=[0, 17, 3, 40], T=[150, 7, 91, 0], N=[9, 33, 0, 1], w=3, D=128,
                         Hq=8, Hkv=2),
    "empty-sequence": Case(P=[0, 5], T=[0, 40], N=[0, 2]),
    "page8": Case(P=[5, 2], T=[77, 64], N=[6, 1], page_size=8),
    "page64": Case(P=[5, 2], T=[77, 64], N=[6, 1], page_size=64),
    "g1": Case(P=[4], T=[170], N=[3], Hq=2, Hkv=2, D=128),
    "g4": Case(P=[4], T=[170], N=[3], Hq=8, Hkv=2, D=128),
    "g8": Case(P=[4], T=[170], N=[3], Hq=8, Hkv=1, D=128),
    "g8-d64": Case(P=[4], T=[170], N=[3], Hq=16, Hkv=2, D=64),
    "zero-gate": Case(P=[4], T=[70], N=[3], zero_gate=True),
    "sharp-gate-and-queries": Case(P=[4, 1], T=[70, 33], N=[3, 2], gate_scale=10.0, q_scale=3.0,
                                   D=128),
    "long": Case(P=[32, 0], T=[1100, 700], N=[10, 0], D=128, Hq=16, Hkv=8),
}


def fresh_cache(like):
    return skv.PagedKV(torch.full_like(like.k_pages, float("nan")),
                       torch.full_like(like.v_pages, float("nan")), like.block_table)


def run_both(case: Case, raw_view: bool = False):
    """The two-call path into the case's cache and the fused call into a
    fresh one (same block table); returns everything each wrote."""
    x = build(case)
    t, dev, spans = x["t"], x["dev"], x["spans"]
    B, Hq, D = case.B, case.Hq, case.D
    scale = D ** -0.5
    k, v = t(x["k_raw"]), t(x["v_raw"])
    if raw_view:  # K and V as views into one [B, S, 3, Hkv, D] projection output
        qkv = torch.full((B, x["S"], 3, case.Hkv, D), float("nan"), dtype=x["dt"], device=dev)
        qkv[:, :, 1] = k
        qkv[:, :, 2] = v
        k, v = qkv[:, :, 1], qkv[:, :, 2]
    res = {}
    for name in ("split", "fused"):
        cache = x["cache"] if name == "split" else fresh_cache(x["cache"])
        clen = torch.full((B,), -7, dtype=torch.int32, device=dev)
        out = torch.full((B, x["S"], Hq, D), float("nan"), dtype=x["dt"], device=dev)
        lse = torch.full((B, Hq, x["S"]), float("nan"), dtype=torch.float32, device=dev)
        if name == "split":
            skv.speechkv_pool_kv(k, v, spans, case.w, t(x["u"]), case.layer, case.l0, cache, clen)
            skv.speechkv_prefill_attn(t(x["q"]), cache, spans, case.w, case.layer, case.l0, out,
                                      mask_mode=case.mode, scale=scale, lse=lse)
        else:
            skv.speechkv_pool_prefill_attn(t(x["q"]), k, v, spans, case.w, t(x["u"]), case.layer,
                                           case.l0, cache, out, cache_len_out=clen,
                                           mask_mode=case.mode, scale=scale, lse=lse)
        torch.cuda.synchronize()
        res[name] = dict(cache=cache, clen=clen.cpu().tolist(), out=out, lse=lse)
    return x, res


def check_same(case: Case, x, res):
    a, f = res["split"], res["fused"]
    assert f["clen"] == a["clen"] == x["clen"]
    for b in range(case.B):
        R = case.P[b] + case.T[b] + case.N[b]
        L = x["clen"][b]
        if L:
            ka, va = gather(a["cache"], b, L)
            kf, vf = gather(f["cache"], b, L)
            assert torch.equal(ka, kf) and torch.equal(va, vf), f"cache rows of sequence {b}"
        if R:
            assert torch.equal(a["out"][b, :R], f["out"][b, :R]), f"output of sequence {b}"
            la, lf = a["lse"][b, :, :R], f["lse"][b, :, :R]
            assert torch.equal(torch.isneginf(la), torch.isneginf(lf))
            fin = torch.isfinite(la)
            assert torch.equal(la[fin], lf[fin]), f"lse of sequence {b}"
        if R < x["S"]:  # rows past the sequence are neither read nor written
            assert torch.isnan(f["out"][b, R:]).all()


def check_oracle(case: Case, x, res):
    f = res["fused"]
    tol = TOL[case.dtype]
    u64 = None if x["u"] is None else f64(x["u"])
    kh, vh, oclen = oracle.pool(f64(x["k_raw"]), f64(x["v_raw"]), case.P, case.T, case.N, case.w,
                                case.layer, case.l0, u64)
    ref, ref_lse = oracle.attention(f64(x["q"]), kh, vh, case.P, case.T, case.N, case.w,
                                    case.layer, case.l0, case.mode, case.D ** -0.5)
    errs = {}
    for b in range(case.B):
        L, R = int(oclen[b]), case.P[b] + case.T[b] + case.N[b]
        if L:
            gk, gv = gather(f["cache"], b, L)
            errs[f"pool_k[{b}]"] = fwd_err(f64(gk), kh[b, :L], case.dtype)
            errs[f"pool_v[{b}]"] = fwd_err(f64(gv), vh[b, :L], case.dtype)
        if R:
            go = f64(f["out"][b, :R])
            assert np.all(np.isfinite(go))
            errs[f"prefill[{b}]"] = fwd_err(go, ref[b, :R], case.dtype)
            gl, rl = f64(f["lse"][b, :, :R]), ref_lse[b, :, :R]
            assert np.array_equal(np.isneginf(gl), np.isneginf(rl))
    bad = {k: e for k, e in errs.items() if not e <= tol}
    assert not bad, f"{case}: above {tol}: {bad}"


@pytest.mark.parametrize("name", sorted(CASES))
def test_fused_equals_split_and_oracle(name):
    case = CASES[name]
    print(f"case {name}", flush=True)
    x, res = run_both(case)
    check_same(case, x, res)
    check_oracle(case, x, res)


def test_fused_strided_raw_views():
    case = Case(P=[6, 1], T=[90, 45], N=[4, 8], D=128, Hq=8, Hkv=2)
    x, res = run_both(case, raw_view=True)
    check_same(case, x, res)
    check_oracle(case, x, res)


def test_fused_then_decode():
    """Decoding after the fused prefill reads the cache it wrote."""
    wl = inputs.LAYER_30S
    a = Job(wl, keep_decode=True)
    f = Job(wl, keep_decode=True, share_inputs=a)
    a.run()
    f.run_prefill_fused()
    for s in range(wl.decode_steps):
        f.run_decode_step(s)
    torch.cuda.synchronize()
    assert torch.equal(a.prefill_out, f.prefill_out)
    assert torch.equal(a.decode_out, f.decode_out)
    assert torch.equal(a.cache_len_out[0], f.cache_len_out[0])


@pytest.mark.parametrize("wl_name,layers", [("prefill", None), ("stack", (0, 14, 27))])
def test_fused_workloads(wl_name, layers):
    """Full-size workloads: the 1596-query prefill (b=8, every output checked
    against the oracle too) and layers of the 60 s stack below and above l0
    (b=64, bit-for-bit against the two-call path)."""
    wl = inputs.PREFILL_1500 if wl_name == "prefill" else inputs.STACK_60S.with_(decode_steps=0)
    a = Job(wl, layers=layers)
    f = Job(wl, layers=layers, share_inputs=a)
    for l in a.layers:
        a.run_prefill(layers=[l])
        f.run_prefill_fused(layers=[l])
        torch.cuda.synchronize()
        i = a.layers.index(l)
        assert torch.equal(a.prefill_out, f.prefill_out), f"layer {l}"
        assert torch.equal(a.cache_len_out[i], f.cache_len_out[i])
        L = a.prefill_clen[i]
        for b in (0, wl.batch - 1):
            ka, va = gather(a.caches[i], b, L)
            kf, vf = gather(f.caches[i], b, L)
            assert torch.equal(ka, kf) and torch.equal(va, vf)
    if wl_name == "prefill":
        from helpers import oracle_prefill_for
        ref, _ = oracle_prefill_for(f, 0, list(range(wl.batch)))
        err = fwd_err(f64(f.prefill_out), ref, "bf16")
        print(f"{wl.name}: fused prefill parity {err:.3e}", flush=True)
        assert err <= TOL["bf16"]
