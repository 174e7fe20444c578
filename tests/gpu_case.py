"""One SpeechKV case end to end on the GPU, checked against the fp64 oracle.

Builds seeded inputs with arbitrary per-sequence spans, runs pool -> prefill
-> decode steps through the C ABI, and compares pooled K/V, prefill outputs
and LSE, and every decode output with the oracle.  Test infrastructure only.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional

import numpy as np
import torch

import oracle
from helpers import TOL, f64, fwd_err, fwd_parts, gather, rms_err, tensor_err
from paper_2607_06827_amd import inputs
from paper_2607_06827_amd import speechkv as skv


@dataclasses.dataclass
class Case:
    P: List[int]
    T: List[int]
    N: List[int]
    w: int = 4
    layer: int = 1
    l0: int = 0
    Hq: int = 4
    Hkv: int = 2
    D: int = 64
    dtype: str = "bf16"
    page_size: int = 16
    mode: int = 0
    decode_steps: int = 3
    seed: int = 0
    gate_scale: float = 1.0
    q_scale: float = 1.0
    shuffle: bool = True
    num_splits: int = 0
    zero_gate: bool = False
    bound_slack: int = 0  # decode's host bound exceeds the longest cache by this (capped by capacity)

    @property
    def B(self):
        return len(self.P)


GUARD = 4096  # bytes of fixed pattern on each side of a guarded output
GUARD_BYTE = 0xA5


def guarded(shape, dtype, dev, fill=float("nan")):
    """A tensor of `shape` (filled with `fill`) inside a larger allocation
    whose GUARD bytes before and after it hold GUARD_BYTE.  Returns the
    tensor and a function asserting that the guards are intact."""
    n = 1
    for d in shape:
        n *= d
    esz = torch.tensor([], dtype=dtype).element_size()
    g = GUARD // esz
    buf = torch.empty(n + 2 * g, dtype=dtype, device=dev)
    raw = buf.view(torch.uint8)
    raw[:GUARD] = GUARD_BYTE
    raw[GUARD + n * esz:] = GUARD_BYTE
    t = buf[g:g + n].view(shape)
    t.fill_(fill)

    def check(what):
        torch.cuda.synchronize()
        assert bool(torch.all(raw[:GUARD] == GUARD_BYTE)), f"{what}: guard before it overwritten"
        assert bool(torch.all(raw[GUARD + n * esz:] == GUARD_BYTE)), f"{what}: guard after it overwritten"

    return t, check


def build(case: Case, device="cuda"):
    B, Hq, Hkv, D = case.B, case.Hq, case.Hkv, case.D
    dt = torch.bfloat16 if case.dtype == "bf16" else torch.float32
    rows = [p + t + n for p, t, n in zip(case.P, case.T, case.N)]
    S = max(max(rows), 1)
    s0 = case.seed * 1000
    k_raw = inputs.normal((B, S, Hkv, D), s0 + 1, dtype=dt)
    v_raw = inputs.normal((B, S, Hkv, D), s0 + 2, dtype=dt)
    u = None if case.zero_gate else inputs.normal((Hkv, D), s0 + 3, scale=case.gate_scale / math.sqrt(D))
    q = inputs.normal((B, S, Hq, D), s0 + 4, scale=case.q_scale, dtype=dt)
    steps = case.decode_steps
    qd = inputs.normal((max(steps, 1), B, Hq, D), s0 + 5, scale=case.q_scale, dtype=dt)
    kn = inputs.normal((max(steps, 1), B, Hkv, D), s0 + 6, dtype=dt)
    vn = inputs.normal((max(steps, 1), B, Hkv, D), s0 + 7, dtype=dt)
    clen = [skv.speechkv_compressed_len(p, t, n, case.w, case.layer, case.l0)
            for p, t, n in zip(case.P, case.T, case.N)]
    pages = max(1, -(-(max(clen) + steps + case.bound_slack) // case.page_size))
    table, total = inputs.block_table(B, pages, case.seed, shuffle=case.shuffle, spare_pages=3)
    dev = torch.device(device)
    t = lambda x: None if x is None else x.to(dev)
    cache = skv.PagedKV(torch.full((total, Hkv, case.page_size, D), float("nan"), dtype=dt, device=dev),
                        torch.full((total, Hkv, case.page_size, D), float("nan"), dtype=dt, device=dev),
                        table.to(dev))
    spans = skv.Spans(torch.tensor(case.P, dtype=torch.int32, device=dev),
                      torch.tensor(case.T, dtype=torch.int32, device=dev),
                      torch.tensor(case.N, dtype=torch.int32, device=dev),
                      max(case.T) if case.T else 0, max(rows))
    return dict(k_raw=k_raw, v_raw=v_raw, u=u, q=q, qd=qd, kn=kn, vn=vn, clen=clen, cache=cache,
                spans=spans, dev=dev, t=t, S=S, dt=dt)


def run_and_check(case: Case, check_prefill: bool = True, device="cuda") -> dict:
    """Run the case and assert parity; returns the error of every check."""
    x = build(case, device)
    t, dev, cache, spans = x["t"], x["dev"], x["cache"], x["spans"]
    B, Hq, Hkv, D = case.B, case.Hq, case.Hkv, case.D
    tol = TOL[case.dtype]
    scale = D ** -0.5
    errs = {}

    clen_dev = torch.full((B,), -7, dtype=torch.int32, device=dev)
    skv.speechkv_pool_kv(t(x["k_raw"]), t(x["v_raw"]), spans, case.w, t(x["u"]), case.layer,
                         case.l0, cache, clen_dev)
    torch.cuda.synchronize()
    assert clen_dev.cpu().tolist() == x["clen"]

    u64 = None if x["u"] is None else f64(x["u"])
    kh, vh, oclen = oracle.pool(f64(x["k_raw"]), f64(x["v_raw"]), case.P, case.T, case.N, case.w,
                                case.layer, case.l0, u64)
    assert list(oclen) == x["clen"]
    for b in range(B):
        L = x["clen"][b]
        if L == 0:
            continue
        gk, gv = gather(cache, b, L)
        errs[f"pool_k[{b}]"] = fwd_err(f64(gk), kh[b, :L], case.dtype)
        errs[f"pool_v[{b}]"] = fwd_err(f64(gv), vh[b, :L], case.dtype)
        # text rows are copies: bit for bit
        P, T = case.P[b], case.T[b]
        nW = L - P - case.N[b]
        assert torch.equal(gk[:P].cpu(), x["k_raw"][b, :P])
        assert torch.equal(gv[nW + P:].cpu(), x["v_raw"][b, P + T:P + T + case.N[b]])

    # pages that no sequence's table names are never written
    named = set(cache.block_table.flatten().tolist())
    spare = [p for p in range(cache.k_pages.shape[0]) if p not in named]
    assert spare
    assert torch.isnan(cache.k_pages[spare].float()).all() and torch.isnan(cache.v_pages[spare].float()).all()

    if check_prefill:
        out, out_guard = guarded((B, x["S"], Hq, D), x["dt"], dev)
        lse, lse_guard = guarded((B, Hq, x["S"]), torch.float32, dev)
        skv.speechkv_prefill_attn(t(x["q"]), cache, spans, case.w, case.layer, case.l0, out,
                                  mask_mode=case.mode, scale=scale, lse=lse)
        torch.cuda.synchronize()
        out_guard("prefill out")
        lse_guard("prefill lse")
        ref, ref_lse = oracle.attention(f64(x["q"]), kh, vh, case.P, case.T, case.N, case.w,
                                        case.layer, case.l0, case.mode, scale)
        for b in range(B):
            R = case.P[b] + case.T[b] + case.N[b]
            if R == 0:
                continue
            go = f64(out[b, :R])
            assert np.all(np.isfinite(go)), "prefill wrote non-finite values"
            errs[f"prefill[{b}]"] = fwd_err(go, ref[b, :R], case.dtype)
            parts = fwd_parts(go, ref[b, :R], case.dtype)
            print(f"prefill[{b}] parity {errs[f'prefill[{b}]']:.3e} (element {parts['elem']:.3e} "
                  f"scale {parts['scale']:.2e} bias {parts['bias']:.2e} per head "
                  f"{parts['group_scale']:.1e}/{parts['group_bias']:.1e}) rms-only "
                  f"{rms_err(go, ref[b, :R]):.3e} tensor-wide {tensor_err(go, ref[b, :R]):.3e}",
                  flush=True)
            gl = f64(lse[b, :, :R])
            rl = ref_lse[b, :, :R]
            assert np.array_equal(np.isneginf(gl), np.isneginf(rl))
            fin = np.isfinite(rl)
            if fin.any():
                errs[f"lse[{b}]"] = float(np.max(np.abs(gl[fin] - rl[fin])))
            if R < x["S"]:  # rows beyond the sequence are not written
                assert torch.isnan(out[b, R:]).all()

    kn, vn, qd = x["kn"], x["vn"], x["qd"]
    kext = [list(kh[b, :x["clen"][b]]) for b in range(B)]
    vext = [list(vh[b, :x["clen"][b]]) for b in range(B)]
    capacity = cache.block_table.shape[1] * cache.k_pages.shape[2]
    bound = lambda n: min(n + case.bound_slack, capacity)
    ws_bytes = skv.speechkv_decode_workspace_bytes(B, Hq, Hkv, D,
                                                   bound(max(x["clen"]) + case.decode_steps),
                                                   case.num_splits)
    ws, ws_guard = guarded((max(ws_bytes, 16) // 4,), torch.float32, dev)
    for s in range(case.decode_steps):
        lens = [c + s + 1 for c in x["clen"]]
        out, out_guard = guarded((B, Hq, D), x["dt"], dev)
        skv.speechkv_decode_attn(t(qd[s]), cache, torch.tensor(lens, dtype=torch.int32, device=dev),
                                 bound(max(lens)), out, k_new=t(kn[s]), v_new=t(vn[s]), scale=scale,
                                 num_splits=case.num_splits, workspace=ws)
        torch.cuda.synchronize()
        out_guard(f"decode out, step {s}")
        ws_guard(f"decode workspace, step {s}")
        for b in range(B):
            kext[b].append(f64(kn[s, b]))
            vext[b].append(f64(vn[s, b]))
        Lmax = max(lens)
        K = np.zeros((B, Lmax, Hkv, D))
        V = np.zeros((B, Lmax, Hkv, D))
        for b in range(B):
            K[b, :lens[b]] = np.array(kext[b])
            V[b, :lens[b]] = np.array(vext[b])
        ref, _ = oracle.decode(f64(qd[s]), K, V, lens, scale)
        errs[f"decode[{s}]"] = fwd_err(f64(out), ref, case.dtype)
        # the new token landed in its slot
        for b in range(B):
            gk, gv = gather(cache, b, lens[b])
            assert torch.equal(gk[-1].cpu(), kn[s, b]) and torch.equal(gv[-1].cpu(), vn[s, b])

    # the spare pages are still untouched after the decode steps stored their tokens
    assert torch.isnan(cache.k_pages[spare].float()).all() and torch.isnan(cache.v_pages[spare].float()).all()
    bad = {k: v for k, v in errs.items() if v > tol}
    assert not bad, f"{case}: errors above tolerance {tol}: {bad}"
    return errs
