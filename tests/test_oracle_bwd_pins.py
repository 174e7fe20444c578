"""Pins of the oracle's gradients (training mode, Sec. III-C: the pooling of
Eq. 4 and the attention of Eq. 5 are optimised jointly, so gradients flow to
the queries, the raw keys and values and the gate).

The backward functions are checked against things other than themselves:
central finite differences of the forward oracle (itself pinned in
test_oracle_pins.py), torch's autograd through scaled_dot_product_attention
for the uncompressed case, the closed form at the zero gate, and invariants
of Eq. 4 (the frame gradients of a window sum to the pooled gradient, for any
gate).  A dropped term (the logit path of dk, the mean in the softmax
Jacobian), a wrong sign or a wrong window or head index fails one of them.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle


def rnd(shape, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


def fd_grad(f, x, eps=1e-6):
    """Central differences of the scalar f at x (every element)."""
    g = np.zeros_like(x)
    flat, gf = x.reshape(-1), g.reshape(-1)
    for i in range(flat.size):
        old = flat[i]
        flat[i] = old + eps
        fp = f()
        flat[i] = old - eps
        fm = f()
        flat[i] = old
        gf[i] = (fp - fm) / (2 * eps)
    return g


CASES = {
    # B, Hq, Hkv, D, P, T, N, w, layer, l0, mode
    "pooled-w3": (2, 4, 2, 8, [3, 0], [10, 7], [2, 3], 3, 1, 0, 0),
    "pooled-w4-start-mask": (1, 2, 2, 8, [2], [9], [3], 4, 2, 1, 1),
    "identity-layer": (1, 4, 1, 4, [2], [6], [1], 4, 0, 3, 0),
    "gqa-g4-w2": (1, 4, 1, 8, [0], [7], [2], 2, 0, 0, 0),
}


@pytest.mark.parametrize("name", list(CASES))
def test_attention_bwd_matches_finite_differences(name):
    B, Hq, Hkv, D, P, T, N, w, layer, l0, mode = CASES[name]
    Sq = max(p + t + n for p, t, n in zip(P, T, N))
    Lc = max(oracle.compressed_len(p, t, n, w, layer, l0) for p, t, n in zip(P, T, N))
    q = rnd((B, Sq, Hq, D), 1)
    kh, vh = rnd((B, Lc, Hkv, D), 2), rnd((B, Lc, Hkv, D), 3)
    go = rnd((B, Sq, Hq, D), 4)
    # rows past a sequence's end carry no output
    for b in range(B):
        go[b, P[b] + T[b] + N[b]:] = 0.0

    def loss():
        o, _ = oracle.attention(q, kh, vh, P, T, N, w, layer, l0, mode)
        return float(np.sum(o * go))

    dq, dk, dv = oracle.attention_bwd(q, kh, vh, P, T, N, w, layer, l0, go, mode)
    for x, g in ((q, dq), (kh, dk), (vh, dv)):
        num = fd_grad(loss, x)
        assert np.max(np.abs(num - g)) < 1e-7 * max(1.0, np.max(np.abs(num)))


@pytest.mark.parametrize("name", list(CASES))
def test_pool_bwd_matches_finite_differences(name):
    B, _, H, D, P, T, N, w, layer, l0, _ = CASES[name]
    S = max(p + t + n for p, t, n in zip(P, T, N)) + 1  # one raw row past every span
    Lc = max(oracle.compressed_len(p, t, n, w, layer, l0) for p, t, n in zip(P, T, N))
    k, v = rnd((B, S, H, D), 5), rnd((B, S, H, D), 6)
    u = rnd((H, D), 7, 0.7)
    gk, gv = rnd((B, Lc, H, D), 8), rnd((B, Lc, H, D), 9)
    clen = [oracle.compressed_len(p, t, n, w, layer, l0) for p, t, n in zip(P, T, N)]
    for b in range(B):
        gk[b, clen[b]:] = 0.0
        gv[b, clen[b]:] = 0.0

    def loss():
        kh, vh, _ = oracle.pool(k, v, P, T, N, w, layer, l0, u, Lc)
        return float(np.sum(kh * gk) + np.sum(vh * gv))

    dk, dv, du = oracle.pool_bwd(k, v, P, T, N, w, layer, l0, u, gk, gv)
    for x, g in ((k, dk), (v, dv), (u, du)):
        num = fd_grad(loss, x)
        assert np.max(np.abs(num - g)) < 1e-7 * max(1.0, np.max(np.abs(num)))


def test_composed_gradient_matches_finite_differences():
    """Pool, then attend: the two backward functions chained give the gradient
    of the whole training-mode layer with respect to q, raw K/V and u."""
    B, Hq, H, D, P, T, N, w = 1, 4, 2, 4, [2], [9], [2], 3
    S = P[0] + T[0] + N[0]
    Lc = oracle.compressed_len(P[0], T[0], N[0], w, 1, 0)
    q = rnd((B, S, Hq, D), 11)
    k, v = rnd((B, S, H, D), 12), rnd((B, S, H, D), 13)
    u = rnd((H, D), 14)
    go = rnd((B, S, Hq, D), 15)

    def loss():
        kh, vh, _ = oracle.pool(k, v, P, T, N, w, 1, 0, u, Lc)
        o, _ = oracle.attention(q, kh, vh, P, T, N, w, 1, 0)
        return float(np.sum(o * go))

    kh, vh, _ = oracle.pool(k, v, P, T, N, w, 1, 0, u, Lc)
    dq, dkh, dvh = oracle.attention_bwd(q, kh, vh, P, T, N, w, 1, 0, go)
    dk, dv, du = oracle.pool_bwd(k, v, P, T, N, w, 1, 0, u, dkh, dvh)
    for x, g in ((q, dq), (k, dk), (v, dv), (u, du)):
        num = fd_grad(loss, x)
        assert np.max(np.abs(num - g)) < 1e-7 * max(1.0, np.max(np.abs(num)))


@pytest.mark.parametrize("Hq,Hkv", [(4, 4), (4, 2), (6, 1)])
def test_uncompressed_attention_bwd_matches_torch_autograd(Hq, Hkv):
    """w = 1: plain causal GQA attention, whose gradient torch's autograd
    through scaled_dot_product_attention (fp64, CPU) gives independently."""
    B, S, D = 2, 13, 8
    q, k, v = rnd((B, S, Hq, D), 21), rnd((B, S, Hkv, D), 22), rnd((B, S, Hkv, D), 23)
    go = rnd((B, S, Hq, D), 24)
    P, T, N = [4, 0], [6, 13], [3, 0]
    scale = 0.3
    G = Hq // Hkv
    tq, tk, tv = (torch.tensor(x, requires_grad=True) for x in (q, k, v))
    o = F.scaled_dot_product_attention(tq.permute(0, 2, 1, 3),
                                       tk.permute(0, 2, 1, 3).repeat_interleave(G, dim=1),
                                       tv.permute(0, 2, 1, 3).repeat_interleave(G, dim=1),
                                       is_causal=True, scale=scale).permute(0, 2, 1, 3)
    (o * torch.from_numpy(go)).sum().backward()
    dq, dk, dv = oracle.attention_bwd(q, k, v, P, T, N, 1, 0, 0, go, 0, scale)
    assert np.allclose(dq, tq.grad.numpy(), rtol=0, atol=1e-12)
    assert np.allclose(dk, tk.grad.numpy(), rtol=0, atol=1e-12)
    assert np.allclose(dv, tv.grad.numpy(), rtol=0, atol=1e-12)


def test_zero_gate_pool_bwd_closed_form():
    """Zero gate: alpha = 1/n, so dk_j = dK^/n, dv_j = dV^/n, and
    du = sum_j (1/n)(dalpha_j - mean dalpha) k_j with dalpha_j = dK^.k_j + dV^.v_j."""
    B, H, D, P, T, N, w = 1, 2, 6, 1, 7, 2, 3
    S = P + T + N
    k, v = rnd((B, S, H, D), 31), rnd((B, S, H, D), 32)
    Lc = oracle.compressed_len(P, T, N, w, 1, 0)
    gk, gv = rnd((B, Lc, H, D), 33), rnd((B, Lc, H, D), 34)
    dk, dv, du = oracle.pool_bwd(k, v, [P], [T], [N], w, 1, 0, None, gk, gv)
    want_du = np.zeros((H, D))
    for i, (a, e) in enumerate([(1, 4), (4, 7), (7, 8)]):  # windows of 3, 3 and 1 frames
        n = e - a
        assert np.allclose(dk[0, a:e], gk[0, P + i] / n, atol=1e-15)
        assert np.allclose(dv[0, a:e], gv[0, P + i] / n, atol=1e-15)
        da = np.einsum("jhd,hd->jh", k[0, a:e], gk[0, P + i]) + np.einsum("jhd,hd->jh", v[0, a:e], gv[0, P + i])
        want_du += np.einsum("jh,jhd->hd", (da - da.mean(0)) / n, k[0, a:e])
    assert np.allclose(du, want_du, atol=1e-13)
    # text rows: the gradient of the row they were copied to
    assert np.array_equal(dk[0, :P], gk[0, :P]) and np.array_equal(dk[0, P + T:], gk[0, P + 3:])


def test_window_gradients_sum_to_pooled_gradient():
    """sum_j alpha_j = 1 and sum_j ds_j = 0, so for any gate the raw-key
    gradients of a window add up to dK^ of that window (values likewise)."""
    B, H, D, P, T, N, w = 2, 2, 8, [3, 1], [14, 9], [1, 2], 4
    S = 18
    k, v = rnd((B, S, H, D), 41), rnd((B, S, H, D), 42)
    u = rnd((H, D), 43, 2.0)
    Lc = max(oracle.compressed_len(p, t, n, w, 1, 0) for p, t, n in zip(P, T, N))
    gk, gv = rnd((B, Lc, H, D), 44), rnd((B, Lc, H, D), 45)
    dk, dv, _ = oracle.pool_bwd(k, v, P, T, N, w, 1, 0, u, gk, gv)
    for b in range(B):
        nW = -(-T[b] // w)
        for i in range(nW):
            a, e = P[b] + i * w, min(P[b] + (i + 1) * w, P[b] + T[b])
            assert np.allclose(dk[b, a:e].sum(0), gk[b, P[b] + i], atol=1e-12)
            assert np.allclose(dv[b, a:e].sum(0), gv[b, P[b] + i], atol=1e-12)
        assert not np.any(dk[b, P[b] + T[b] + N[b]:])  # rows past the spans


def test_value_gradients_sum_to_output_gradients():
    """Every row's probabilities sum to 1, so the value gradients over all keys
    add up to the output gradients of the rows that see at least one key."""
    B, Hq, H, D, P, T, N, w = 1, 2, 1, 6, [0], [11], [3], 4
    Sq = 14
    Lc = oracle.compressed_len(0, 11, 3, w, 1, 0)
    q, kh, vh = rnd((B, Sq, Hq, D), 51), rnd((B, Lc, H, D), 52), rnd((B, Lc, H, D), 53)
    go = rnd((B, Sq, Hq, D), 54)
    _, lse = oracle.attention(q, kh, vh, P, T, N, w, 1, 0)
    dq, _, dv = oracle.attention_bwd(q, kh, vh, P, T, N, w, 1, 0, go)
    seen = np.isfinite(lse[0, 0])  # [Sq] rows with a visible key (same for both heads)
    assert not seen[:3].any() and seen[3:].all()  # rows before the first window ends see nothing
    assert np.allclose(dv[0, :, 0].sum(0), go[0, seen].sum((0, 1)), atol=1e-12)
    assert not np.any(dq[0, ~seen])
