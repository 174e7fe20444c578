"""Pins of the fp64 oracle against what arXiv 2607.06827 and mathematics fix.

Each test checks the oracle against something other than itself: a library
routine (torch's scaled_dot_product_attention for the w = 1 case), a closed
form (window mean for a zero gate, a logistic weight for two-frame windows,
the de-duplicated sequence for repeated frames), the brute force of
tests/brute.py, invariants of Eq. 4/5, or numbers the paper prints
(tests/golden/).  A dropped term, a wrong sign, a wrong window or head index
or an off-by-one in the mask fails at least one of them.
"""
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import brute
import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rnd(shape, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


def sdpa_causal(q, k, v, scale):
    """torch SDPA (fp64 CPU, causal, GQA by repeating KV heads).
    q [B, S, Hq, D], k/v [B, S, Hkv, D] -> [B, S, Hq, D]."""
    G = q.shape[2] // k.shape[2]
    tq = torch.from_numpy(q).permute(0, 2, 1, 3)
    tk = torch.from_numpy(k).permute(0, 2, 1, 3).repeat_interleave(G, dim=1)
    tv = torch.from_numpy(v).permute(0, 2, 1, 3).repeat_interleave(G, dim=1)
    o = F.scaled_dot_product_attention(tq, tk, tv, is_causal=True, scale=scale)
    return o.permute(0, 2, 1, 3).numpy()


# ---------------------------------------------------------------- pooling pins

@pytest.mark.parametrize("w,layer,l0", [(1, 3, 0), (4, 2, 5), (8, 0, 1)])
def test_identity_pool_is_bitwise(w, layer, l0):
    """w_eff = 1 (w = 1, or a layer before l0): every weight is 1 and the
    cache is the raw sequence, bit for bit (Sec. III-B)."""
    B, S, H, D = 2, 19, 2, 8
    k, v = rnd((B, S, H, D), 1), rnd((B, S, H, D), 2)
    u = rnd((H, D), 3, 5.0)
    P, T, N = [3, 0], [11, 17], [5, 2]
    kh, vh, clen = oracle.pool(k, v, P, T, N, w, layer, l0, u)
    assert list(clen) == [19, 19]
    assert np.array_equal(kh[:, :19], k) and np.array_equal(vh[:, :19], v)


def test_zero_gate_gives_window_mean():
    """A zero gate gives uniform weights 1/|window| (the paper's
    initialisation, Sec. III-B), including a short last window."""
    B, H, D, P, T, N, w = 1, 3, 5, 2, 11, 3, 4
    S = P + T + N
    k, v = rnd((B, S, H, D), 4), rnd((B, S, H, D), 5)
    kh, vh, clen = oracle.pool(k, v, [P], [T], [N], w, 7, 7, None)
    assert clen[0] == P + 3 + N
    windows = [range(2, 6), range(6, 10), range(10, 13)]
    for i, fr in enumerate(windows):
        np.testing.assert_allclose(kh[0, P + i], k[0, list(fr)].mean(axis=0), rtol=0, atol=1e-15)
        np.testing.assert_allclose(vh[0, P + i], v[0, list(fr)].mean(axis=0), rtol=0, atol=1e-15)


def test_two_frame_weights_are_logistic():
    """For a window of two keys the softmax of Eq. 4 is the logistic function
    of the logit difference: k^ = s(z1 - z2) k1 + s(z2 - z1) k2."""
    B, H, D, T = 1, 2, 6, 8
    k, v = rnd((B, T, H, D), 6), rnd((B, T, H, D), 7)
    u = rnd((H, D), 8)
    kh, vh, _ = oracle.pool(k, v, [0], [T], [0], 2, 0, 0, u)
    sig = lambda x: 1.0 / (1.0 + math.exp(-x))
    for i in range(T // 2):
        for g in range(H):
            z1 = float(u[g] @ k[0, 2 * i, g])
            z2 = float(u[g] @ k[0, 2 * i + 1, g])
            a1 = sig(z1 - z2)
            a2 = sig(z2 - z1)
            np.testing.assert_allclose(kh[0, i, g], a1 * k[0, 2 * i, g] + a2 * k[0, 2 * i + 1, g], atol=1e-14)
            np.testing.assert_allclose(vh[0, i, g], a1 * v[0, 2 * i, g] + a2 * v[0, 2 * i + 1, g], atol=1e-14)


def test_gate_scores_keys_not_values():
    """The gate reads the keys only (Sec. III-B): changing V leaves the weights
    alone, so V^ changes linearly, while changing K moves them."""
    B, H, D, T, w = 1, 1, 4, 4, 4
    k, v = rnd((B, T, H, D), 9), rnd((B, T, H, D), 10)
    u = rnd((H, D), 11, 3.0)
    kh1, vh1, _ = oracle.pool(k, v, [0], [T], [0], w, 0, 0, u)
    kh2, vh2, _ = oracle.pool(k, 2.0 * v, [0], [T], [0], w, 0, 0, u)
    np.testing.assert_array_equal(kh1, kh2)
    np.testing.assert_allclose(vh2, 2.0 * vh1, atol=1e-14)


def test_text_rows_copied_bitwise():
    """Text positions are left unchanged (Sec. III-B); the suffix moves up to
    follow the pooled speech."""
    B, H, D, w = 2, 2, 4, 3
    P, T, N = [4, 1], [9, 7], [6, 3]
    S = 19
    k, v = rnd((B, S, H, D), 12), rnd((B, S, H, D), 13)
    u = rnd((H, D), 14)
    kh, vh, clen = oracle.pool(k, v, P, T, N, w, 1, 0, u)
    for b in range(B):
        nW = -(-T[b] // w)
        assert clen[b] == P[b] + nW + N[b]
        assert np.array_equal(kh[b, :P[b]], k[b, :P[b]])
        assert np.array_equal(vh[b, :P[b]], v[b, :P[b]])
        s0 = P[b] + T[b]
        assert np.array_equal(kh[b, P[b] + nW:clen[b]], k[b, s0:s0 + N[b]])
        assert np.array_equal(vh[b, P[b] + nW:clen[b]], v[b, s0:s0 + N[b]])
        assert not kh[b, clen[b]:].any()


def test_pooled_rows_lie_within_window_range():
    """The weights are positive and sum to 1, so each pooled coordinate lies
    between the window's minimum and maximum."""
    B, H, D, T, w = 1, 2, 16, 37, 5
    k, v = rnd((B, T, H, D), 15), rnd((B, T, H, D), 16)
    u = rnd((H, D), 17, 4.0)
    kh, vh, clen = oracle.pool(k, v, [0], [T], [0], w, 0, 0, u)
    for i in range(clen[0]):
        fr = slice(i * w, min((i + 1) * w, T))
        for x, xh in ((k, kh), (v, vh)):
            assert np.all(xh[0, i] <= x[0, fr].max(axis=0) + 1e-15)
            assert np.all(xh[0, i] >= x[0, fr].min(axis=0) - 1e-15)


def test_permuting_frames_inside_a_window_changes_nothing():
    """Eq. 4 is symmetric in the frames of a window."""
    B, H, D, T, w = 1, 2, 8, 12, 4
    k, v = rnd((B, T, H, D), 18), rnd((B, T, H, D), 19)
    u = rnd((H, D), 20)
    perm = np.concatenate([np.random.default_rng(21).permutation(4) + 4 * i for i in range(3)])
    kh1, vh1, _ = oracle.pool(k, v, [0], [T], [0], w, 0, 0, u)
    kh2, vh2, _ = oracle.pool(k[:, perm], v[:, perm], [0], [T], [0], w, 0, 0, u)
    np.testing.assert_allclose(kh1, kh2, atol=1e-14)
    np.testing.assert_allclose(vh1, vh2, atol=1e-14)


def test_huge_gate_selects_the_argmax_frame():
    """A very large gate turns the window softmax into an argmax: the pooled
    key is (numerically) the frame with the largest logit, and nothing
    overflows."""
    B, H, D, T, w = 1, 1, 8, 8, 4
    k, v = rnd((B, T, H, D), 22), rnd((B, T, H, D), 23)
    u = rnd((H, D), 24, 1e4)
    kh, vh, _ = oracle.pool(k, v, [0], [T], [0], w, 0, 0, u)
    for i in range(2):
        logits = [float(u[0] @ k[0, j, 0]) for j in range(i * w, (i + 1) * w)]
        j = i * w + int(np.argmax(logits))
        np.testing.assert_allclose(kh[0, i, 0], k[0, j, 0], atol=1e-12)
        np.testing.assert_allclose(vh[0, i, 0], v[0, j, 0], atol=1e-12)


# -------------------------------------------------------------- attention pins

@pytest.mark.parametrize("Hq,Hkv", [(4, 4), (4, 2), (8, 2), (8, 1)])
def test_uncompressed_attention_matches_torch_sdpa(Hq, Hkv):
    """With w_eff = 1 the mask is ordinary causal attention (Eq. 5), checked
    against torch's scaled_dot_product_attention in fp64, GQA heads grouped
    consecutively."""
    B, D, P, T, N = 2, 16, 5, 13, 4
    S = P + T + N
    k, v = rnd((B, S, Hkv, D), 25), rnd((B, S, Hkv, D), 26)
    q = rnd((B, S, Hq, D), 27)
    kh, vh, _ = oracle.pool(k, v, [P] * B, [T] * B, [N] * B, 4, 0, 1, rnd((Hkv, D), 28))
    scale = 1.0 / math.sqrt(D)
    out, lse = oracle.attention(q, kh, vh, [P] * B, [T] * B, [N] * B, 4, 0, 1, 0, scale)
    ref = sdpa_causal(q, k, v, scale)
    np.testing.assert_allclose(out, ref, atol=1e-12, rtol=0)
    # lse against an explicit log-sum-exp of the causal logits
    G = Hq // Hkv
    for b in range(B):
        for h in range(Hq):
            for p in range(S):
                z = scale * (k[b, :p + 1, h // G] @ q[b, p, h])
                assert abs(lse[b, h, p] - np.log(np.exp(z - z.max()).sum()) - z.max()) < 1e-12


def test_decode_matches_torch_sdpa_last_row():
    """A decode step is the last causal row: every cached key is visible."""
    B, Hq, Hkv, D, L = 3, 8, 2, 16, 21
    k, v = rnd((B, L, Hkv, D), 29), rnd((B, L, Hkv, D), 30)
    q = rnd((B, L, Hq, D), 31)
    scale = 0.3
    out, _ = oracle.decode(q[:, -1], k, v, [L] * B, scale)
    ref = sdpa_causal(q, k, v, scale)[:, -1]
    np.testing.assert_allclose(out, ref, atol=1e-12, rtol=0)


@pytest.mark.parametrize("mode", [0, 1])
def test_repeated_frames_equal_deduplicated_causal_attention(mode):
    """If every frame of each window is the same vector, the pooled key is
    that vector for any gate, and attention over the compressed cache equals
    causal attention over the de-duplicated sequence (torch SDPA): the row of a
    window's last frame (mask 0) or first frame (mask 1) is the de-duplicated
    row of that window."""
    B, Hq, Hkv, D, P, N, w, nW = 2, 4, 2, 8, 3, 4, 4, 5
    T = w * nW
    L = P + nW + N
    base_k, base_v = rnd((B, L, Hkv, D), 32), rnd((B, L, Hkv, D), 33)
    frame_of = list(range(P)) + [P + i // w for i in range(T)] + [P + nW + m for m in range(N)]
    k, v = base_k[:, frame_of], base_v[:, frame_of]
    u = rnd((Hkv, D), 34, 3.0)
    kh, vh, clen = oracle.pool(k, v, [P] * B, [T] * B, [N] * B, w, 1, 1, u)
    np.testing.assert_allclose(kh[:, :L], base_k, atol=1e-14)
    np.testing.assert_allclose(vh[:, :L], base_v, atol=1e-14)
    S = P + T + N
    q = rnd((B, S, Hq, D), 35)
    scale = 1.0 / math.sqrt(D)
    out, _ = oracle.attention(q, kh, vh, [P] * B, [T] * B, [N] * B, w, 1, 1, mode, scale)
    rows = list(range(P))
    rows += [P + i * w + (w - 1 if mode == 0 else 0) for i in range(nW)]
    rows += [P + T + m for m in range(N)]
    ref = sdpa_causal(q[:, rows], base_k, base_v, scale)
    np.testing.assert_allclose(out[:, rows], ref, atol=1e-12, rtol=0)


def test_window_visibility_boundary_and_rows_sum_to_one():
    """One-hot values make the output the attention row itself: each row sums
    to 1, and a pooled window is visible from its last frame (mask 0) or its
    first frame (mask 1), never one frame earlier."""
    P, T, N, w = 2, 10, 3, 4           # windows [2,6) [6,10) [10,12)
    nW = 3
    L = P + nW + N
    D = L
    kh = np.zeros((1, L, 1, D))
    vh = np.eye(L)[None, :, None, :]
    q = rnd((1, P + T + N, 1, D), 36)
    for mode, first_row in ((0, [5, 9, 11]), (1, [2, 6, 10])):
        out, _ = oracle.attention(q, kh, vh, [P], [T], [N], w, 0, 0, mode, 1.0)
        np.testing.assert_allclose(out[0, :, 0].sum(axis=1), 1.0, atol=1e-14)
        for i, p in enumerate(first_row):
            assert out[0, p, 0, P + i] > 0
            assert out[0, p - 1, 0, P + i] == 0
        for m in range(N):
            p = P + T + m
            assert out[0, p, 0, P + nW + m] > 0 and out[0, p - 1, 0, P + nW + m] == 0


def test_constant_values_give_constant_output_and_empty_rows_give_zero():
    """V == 1 gives O == 1 on every row that sees a key; with no prefix the
    speech rows before the first window closes see nothing: O = 0,
    lse = -inf (mask 0)."""
    Hq, Hkv, D, P, T, N, w = 4, 2, 8, 0, 9, 2, 4
    S = P + T + N
    k = rnd((1, S, Hkv, D), 37)
    v = np.ones((1, S, Hkv, D))
    kh, vh, _ = oracle.pool(k, v, [P], [T], [N], w, 0, 0, rnd((Hkv, D), 38))
    q = rnd((1, S, Hq, D), 39, 3.0)
    out, lse = oracle.attention(q, kh, vh, [P], [T], [N], w, 0, 0, 0, 0.5)
    assert np.all(out[0, :3] == 0) and np.all(np.isneginf(lse[0, :, :3]))
    np.testing.assert_allclose(out[0, 3:], 1.0, atol=1e-14)
    out1, lse1 = oracle.attention(q, kh, vh, [P], [T], [N], w, 0, 0, 1, 0.5)
    np.testing.assert_allclose(out1[0], 1.0, atol=1e-14)
    assert np.all(np.isfinite(lse1[0]))


def test_single_key_row_returns_its_value():
    """A row with exactly one visible key returns that key's value."""
    Hq, Hkv, D = 2, 1, 4
    kh = rnd((1, 3, Hkv, D), 40)
    vh = rnd((1, 3, Hkv, D), 41)
    q = rnd((1, 3, Hq, D), 42, 10.0)
    out, lse = oracle.attention(q, kh, vh, [1], [0], [2], 4, 0, 0, 0, 1.0)
    np.testing.assert_allclose(out[0, 0, 0], vh[0, 0, 0], atol=1e-15)
    np.testing.assert_allclose(lse[0, 0, 0], q[0, 0, 0] @ kh[0, 0, 0], atol=1e-13)


# --------------------------------------------------------- brute-force agreement

CASES = [
    # B, Hq, Hkv, D, P, T, N, w, layer, l0, mode
    (1, 2, 1, 4, 2, 9, 3, 4, 1, 0, 0),
    (2, 4, 2, 4, 0, 7, 2, 3, 0, 0, 0),    # P = 0: empty rows
    (1, 4, 1, 3, 3, 2, 2, 4, 5, 5, 0),    # T < w
    (1, 2, 2, 4, 1, 0, 4, 4, 2, 0, 0),    # T = 0
    (1, 8, 2, 2, 2, 10, 0, 5, 3, 1, 1),   # N = 0, mask 1
    (2, 2, 1, 5, 4, 13, 1, 6, 0, 3, 0),   # layer < l0
    (1, 8, 8, 2, 0, 8, 0, 2, 9, 9, 1),
]


@pytest.mark.parametrize("case", CASES)
def test_oracle_agrees_with_brute_force(case):
    B, Hq, Hkv, D, P, T, N, w, layer, l0, mode = case
    S = P + T + N
    k = rnd((B, S, Hkv, D), 43)
    v = rnd((B, S, Hkv, D), 44)
    u = rnd((Hkv, D), 45, 2.0)
    q = rnd((B, S, Hq, D), 46)
    scale = 0.7
    weff = w if layer >= l0 else 1
    kh, vh, clen = oracle.pool(k, v, [P] * B, [T] * B, [N] * B, w, layer, l0, u)
    out, lse = oracle.attention(q, kh, vh, [P] * B, [T] * B, [N] * B, w, layer, l0, mode, scale)
    for b in range(B):
        bk, bv, groups = brute.pool_one(k[b].tolist(), v[b].tolist(), P, T, N, weff, u.tolist())
        assert clen[b] == len(groups)
        np.testing.assert_allclose(kh[b, :clen[b]], np.array(bk).reshape(-1, Hkv, D), atol=1e-12)
        np.testing.assert_allclose(vh[b, :clen[b]], np.array(bv).reshape(-1, Hkv, D), atol=1e-12)
        bo, bl = brute.attend_one(q[b].tolist(), bk, bv, groups, "end" if mode == 0 else "start", scale)
        if S:
            np.testing.assert_allclose(out[b, :S], np.array(bo), atol=1e-12)
            bl = np.array(bl)
            fin = np.isfinite(bl)
            assert np.array_equal(fin, np.isfinite(lse[b, :, :S]))
            np.testing.assert_allclose(lse[b, :, :S][fin], bl[fin], atol=1e-12)


def test_decode_step_equals_last_prefill_row():
    """Sec. III-C: decoding over the stored compressed cache gives the same
    row as full attention at the newest position."""
    B, Hq, Hkv, D, P, T, N, w = 2, 4, 2, 8, 3, 14, 5, 4
    S = P + T + N
    k, v = rnd((B, S, Hkv, D), 47), rnd((B, S, Hkv, D), 48)
    q = rnd((B, S, Hq, D), 49)
    kh, vh, clen = oracle.pool(k, v, [P] * B, [T] * B, [N] * B, w, 0, 0, rnd((Hkv, D), 50))
    out, lse = oracle.attention(q, kh, vh, [P] * B, [T] * B, [N] * B, w, 0, 0, 0, 0.4)
    dout, dlse = oracle.decode(q[:, S - 1], kh, vh, clen, 0.4)
    np.testing.assert_allclose(dout, out[:, S - 1], atol=1e-14)
    np.testing.assert_allclose(dlse, lse[:, :, S - 1], atol=1e-13)


# ------------------------------------------------------- numbers of the paper

def _golden(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if line:
                rows.append([float(x) for x in line.split()])
    return rows


def test_kv_memory_reduction_matches_the_paper():
    """Sec. V-D prints 2.8x (R = 4) and 4x (R = 8) less KV memory with the
    first 4 of 28 layers uncompressed (Sec. IV-A)."""
    rows = _golden("kv_memory_ratio.txt")
    assert rows
    T = 2400   # speech-only cache, a multiple of every R
    for layers, l0, R, ratio in rows:
        full = sum(oracle.compressed_len(0, T, 0, int(R), l, int(l0) + 10 ** 6) for l in range(int(layers)))
        comp = sum(oracle.compressed_len(0, T, 0, int(R), l, int(l0)) for l in range(int(layers)))
        assert abs(full / comp - ratio) < 1e-12


def test_frame_counts_match_the_paper():
    """80 ms frames (Sec. IV-A): 30 s -> 375 frames, 60 s -> 750, 10 min ->
    7500; a pooled position covers 80R ms.  A last partial window is kept, so
    the speech part of the cache holds ceil(frames / R) entries."""
    for secs, ms, frames, R, pooled_ms in _golden("frame_counts.txt"):
        assert round(secs * 1000 / ms) == frames
        assert ms * R == pooled_ms
        n = oracle.compressed_len(0, int(frames), 0, int(R), 0, 0)
        assert n == math.ceil(frames / R)
        assert (n - 1) * R < frames <= n * R
