"""GPU parity of speechkv_pool_hidden (HS Compression, Sec. IV-A method (4)):
the pooling of Eq. 4 applied to whole hidden states, through the C ABI.

The reference is the oracle's pooling with one "head" whose width is the
hidden size: the HS variant is the same window softmax over gate logits and
the same weighted sum, applied to the hidden state instead of per-head K/V.
Text rows and one-frame windows must come back bitwise; pooled rows within
the element type's tolerance.  The last test runs the whole HS path: pool the
hidden state, then plain causal attention over the shortened sequence
(prefill attention with w = 1), against the oracle.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from helpers import TOL, fwd_err
from paper_2607_06827_amd import inputs
from paper_2607_06827_amd import speechkv as skv

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


def f64(t):
    return t.detach().to("cpu", torch.float64).numpy()


def run_hidden(P, T, N, w, hidden, dtype="bf16", gate_scale=1.0, zero_gate=False, seed=0,
               cap=None):
    dt = torch.bfloat16 if dtype == "bf16" else torch.float32
    B = len(P)
    rows = [p + t + n for p, t, n in zip(P, T, N)]
    S = max(max(rows), 1)
    s0 = 7000 + seed * 10
    h = inputs.normal((B, S, hidden), s0 + 1, dtype=dt).cuda()
    u = None if zero_gate else inputs.normal((hidden,), s0 + 2, scale=gate_scale / math.sqrt(hidden)).cuda()
    out = torch.full((B, S, hidden), float("nan"), dtype=dt, device="cuda")
    out_len = torch.full((B,), -1, dtype=torch.int32, device="cuda")
    i32 = lambda x: torch.tensor(x, dtype=torch.int32, device="cuda")
    spans = skv.Spans(i32(P), i32(T), i32(N), max(T) if T else 0, max(rows))
    # out_capacity = cap rows: a view of the first cap rows of each sequence
    skv.speechkv_pool_hidden(h, spans, w, u, out if cap is None else out[:, :cap], out_len)
    torch.cuda.synchronize()
    # oracle: one head of width `hidden`, a compressed layer
    ref, _, clen = oracle.pool(f64(h).reshape(B, S, 1, hidden), f64(h).reshape(B, S, 1, hidden),
                               P, T, N, w, 1, 0, None if u is None else f64(u).reshape(1, hidden))
    return h, out, out_len, ref[:, :, 0, :], clen


def check(P, T, N, w, hidden, dtype, out, out_len, ref, clen, h):
    assert out_len.cpu().tolist() == [int(c) for c in clen]
    o = f64(out)
    hh = f64(h)
    for b in range(len(P)):
        L = int(clen[b])
        nW = -(-T[b] // w)
        assert fwd_err(o[b, :L], ref[b, :L], dtype) <= TOL[dtype]
        # text rows bitwise
        assert np.array_equal(o[b, :P[b]], hh[b, :P[b]])
        assert np.array_equal(o[b, P[b] + nW:L], hh[b, P[b] + T[b]:P[b] + T[b] + N[b]])
        # rows past the compressed length untouched
        assert np.all(np.isnan(o[b, L:]))


CASES = {
    "h512-bf16": dict(P=[8], T=[60], N=[5], w=4, hidden=512),
    "h1024-bf16-ragged": dict(P=[3, 0], T=[45, 22], N=[2, 4], w=3, hidden=1024),
    "h2048-bf16": dict(P=[32, 5], T=[150, 37], N=[0, 9], w=4, hidden=2048),
    "h4096-bf16": dict(P=[4], T=[33], N=[3], w=4, hidden=4096),
    "h2048-f32": dict(P=[6], T=[50], N=[4], w=4, hidden=2048, dtype="f32"),
    "h512-f32-w8": dict(P=[2], T=[70], N=[1], w=8, hidden=512, dtype="f32"),
    "w12-two-passes": dict(P=[1, 4], T=[61, 30], N=[2, 0], w=12, hidden=1024),
    "w1-identity": dict(P=[5], T=[20], N=[3], w=1, hidden=512),
    "no-prefix": dict(P=[0, 0], T=[37, 9], N=[3, 0], w=4, hidden=512),
    "no-speech": dict(P=[7], T=[0], N=[6], w=4, hidden=512),
    "speech-shorter-than-w": dict(P=[5], T=[3], N=[4], w=8, hidden=512),
    "zero-gate": dict(P=[4], T=[70], N=[3], w=4, hidden=2048, zero_gate=True),
    "sharp-gate": dict(P=[4, 1], T=[70, 33], N=[3, 2], w=4, hidden=2048, gate_scale=10.0),
    "w5-one-frame-second-pass": dict(P=[2, 0], T=[41, 26], N=[3, 1], w=5, hidden=2048),
    "w8-h4096-two-passes": dict(P=[3], T=[45], N=[2], w=8, hidden=4096),
    "zero-gate-w12-h512": dict(P=[5, 2], T=[50, 13], N=[1, 4], w=12, hidden=512, zero_gate=True),
    "zero-gate-f32-h1024": dict(P=[1], T=[23], N=[2], w=3, hidden=1024, dtype="f32", zero_gate=True),
    "varlen": dict(P=[0, 17, 3, 40], T=[150, 7, 91, 0], N=[9, 33, 0, 1], w=3, hidden=2048),
}


@pytest.mark.parametrize("name", list(CASES))
def test_pool_hidden_matches_oracle(name):
    c = dict(CASES[name])
    dtype = c.get("dtype", "bf16")
    h, out, out_len, ref, clen = run_hidden(**c)
    check(c["P"], c["T"], c["N"], c["w"], c["hidden"], dtype, out, out_len, ref, clen, h)


def test_pool_hidden_is_bitwise_repeatable():
    c = CASES["h2048-bf16"]
    _, out1, _, _, _ = run_hidden(**c)
    _, out2, _, _, _ = run_hidden(**c)
    assert torch.equal(out1.view(torch.int16), out2.view(torch.int16))


def test_hs_compression_path():
    """Pool the hidden state, then causal attention over the shortened sequence.

    hidden = 512 is read as 4 heads of 128 for queries, keys and values (the
    projections are the identity here).  The shortened sequence goes into a
    paged cache with w_eff = 1 (a bitwise copy) and prefill attention with w =
    1 is plain causal attention over it; the oracle does the same on its own
    pooled hidden state."""
    P, T, N, w, hidden, H, D = [6, 2], [57, 40], [5, 3], 4, 512, 4, 128
    h, out, out_len, ref, clen = run_hidden(P, T, N, w, hidden)
    B = len(P)
    L = [int(x) for x in clen]
    Tc = [-(-t // w) for t in T]  # speech rows of the shortened sequence
    S2 = max(L)
    x = out[:, :S2].contiguous()
    x = torch.nan_to_num(x)  # rows past a sequence's length were never written
    kv = x.view(B, S2, H, D)
    page = 16
    pages = -(-S2 // page)
    table, total = inputs.block_table(B, pages, 0)
    cache = skv.PagedKV(torch.zeros(total, H, page, D, dtype=torch.bfloat16, device="cuda"),
                        torch.zeros(total, H, page, D, dtype=torch.bfloat16, device="cuda"),
                        table.cuda())
    i32 = lambda v: torch.tensor(v, dtype=torch.int32, device="cuda")
    sp = skv.Spans(i32(P), i32(Tc), i32(N), max(Tc), S2)
    # layer < l0: w_eff = 1, the cache receives the rows bitwise
    skv.speechkv_pool_kv(kv, kv, sp, 1, None, 0, 1, cache)
    o = torch.full((B, S2, H, D), float("nan"), dtype=torch.bfloat16, device="cuda")
    skv.speechkv_prefill_attn(kv, cache, sp, 1, 0, 1, o)
    torch.cuda.synchronize()
    refx = np.zeros((B, S2, H, D))
    for b in range(B):
        refx[b, :L[b]] = ref[b, :L[b]].reshape(L[b], H, D)
    ro, _ = oracle.attention(refx, refx, refx, P, Tc, N, 1, 0, 1)
    oo = f64(o)
    for b in range(B):
        assert fwd_err(oo[b, :L[b]], ro[b, :L[b]], "bf16") <= TOL["bf16"]


def test_pool_hidden_tight_capacity():
    """An output buffer of exactly the longest compressed length is enough."""
    P, T, N, w, hidden = [3, 9], [41, 30], [2, 7], 4, 1024
    L = [p + -(-t // w) + n for p, t, n in zip(P, T, N)]
    h, out, out_len, ref, clen = run_hidden(P, T, N, w, hidden, cap=max(L))
    check(P, T, N, w, hidden, "bf16", out, out_len, ref, clen, h)


def test_pool_hidden_short_capacity_writes_nothing_past_it():
    """Rows at or past out_capacity stay untouched; out_len keeps the full
    compressed length, which is how a caller sees the short buffer."""
    P, T, N, w, hidden, cap = [6, 2], [57, 12], [5, 1], 4, 512, 10
    h, out, out_len, ref, clen = run_hidden(P, T, N, w, hidden, cap=cap)
    assert out_len.cpu().tolist() == [int(c) for c in clen]
    o = f64(out)
    for b in range(len(P)):
        n = min(int(clen[b]), cap)
        assert fwd_err(o[b, :n], ref[b, :n], "bf16") <= TOL["bf16"]
        assert np.all(np.isnan(o[b, n:]))


def test_pool_hidden_all_spans_empty():
    """Every span empty: nothing is written and every length is 0."""
    P, T, N = [0, 0, 0], [0, 0, 0], [0, 0, 0]
    h, out, out_len, _, _ = run_hidden(P, T, N, 4, 512)
    assert out_len.cpu().tolist() == [0, 0, 0]
    assert torch.isnan(out).all()
