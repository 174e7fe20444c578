"""fp64 oracle of SpeechKV over sequences with several speech runs.

TEST INFRASTRUCTURE ONLY: the tests may import this module; the product path
never does.  It shares no code with the GPU library (nor with the C oracle).

A sequence is a list of segments (text_len, speech_len): text_len text rows
followed by speech_len speech frames, the segments in order (a multi-turn
input whose LLM input interleaves speech and text, Sec. III-A).  Each speech
run is compressed on its own with Eq. 4 of Sec. III-B: non-overlapping
windows of w consecutive frames starting at the run's first frame (the last
window keeps the frames it has), each replaced by its frames weighted with
the softmax of the gate logits u . k_j over the window; text rows are kept.
Attention over the compressed sequence follows Eq. 5 with the causal mask
over compressed positions: a text key is visible from its own position, a
pooled window from its last frame (mask mode 0) or its first frame (mode 1).
Below layer l0 the window is 1 and every row is kept.

Plain numpy in float64; pure-Python loops over slots and rows, meant for the
small and medium sizes of the tests.
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

import numpy as np

Segs = Sequence[Tuple[int, int]]


def w_eff(w: int, layer: int, l0: int) -> int:
    return w if layer >= l0 else 1


def layout(segs: Segs, w: int):
    """Compressed slots of one sequence as (first raw row, frames, visible
    from in mode 0, visible from in mode 1), and its raw row count."""
    slots = []
    r = 0
    for t_len, s_len in segs:
        assert t_len >= 0 and s_len >= 0
        for i in range(t_len):
            slots.append((r + i, 1, r + i, r + i))
        r += t_len
        for f in range(0, s_len, w):
            n = min(w, s_len - f)
            slots.append((r + f, n, r + f + n - 1, r + f))
        r += s_len
    return slots, r


def raw_len(segs: Segs) -> int:
    return sum(t + s for t, s in segs)


def compressed_len(segs: Segs, w: int, layer: int, l0: int) -> int:
    return len(layout(segs, w_eff(w, layer, l0))[0])


def pool(k_raw, v_raw, segs_list: List[Segs], w, layer, l0, u=None, Lc=None):
    """Eq. 4 over every speech run of every sequence.  k_raw, v_raw:
    [B, S, Hkv, D]; u: [Hkv, D] or None (zero gate: uniform weights).
    Returns (k_hat, v_hat [B, Lc, Hkv, D], clen [B])."""
    k = np.asarray(k_raw, np.float64)
    v = np.asarray(v_raw, np.float64)
    B, S, H, D = k.shape
    we = w_eff(w, layer, l0)
    lays = [layout(s, we) for s in segs_list]
    clen = np.array([len(sl) for sl, _ in lays], np.int32)
    assert all(r <= S for _, r in lays)
    if Lc is None:
        Lc = max(int(clen.max(initial=0)), 1)
    kh = np.zeros((B, Lc, H, D))
    vh = np.zeros((B, Lc, H, D))
    uu = np.zeros((H, D)) if u is None else np.asarray(u, np.float64)
    for b, (slots, _) in enumerate(lays):
        for c, (first, n, _, _) in enumerate(slots):
            kw = k[b, first:first + n]  # [n, H, D]
            vw = v[b, first:first + n]
            for g in range(H):
                logits = kw[:, g] @ uu[g]  # gate logits of the window's frames
                a = np.exp(logits - logits.max())
                a /= a.sum()
                kh[b, c, g] = a @ kw[:, g]
                vh[b, c, g] = a @ vw[:, g]
    return kh, vh, clen


def visible_from(segs: Segs, w: int, mode: int) -> np.ndarray:
    """Raw position from which each compressed key is visible."""
    slots, _ = layout(segs, w)
    return np.array([s[2] if mode == 0 else s[3] for s in slots], np.int64)


def attention(q, k_hat, v_hat, segs_list: List[Segs], w, layer, l0, mask_mode=0, scale=None):
    """Eq. 5 under the causal mask over compressed positions, every row.
    q: [B, Sq, Hq, D]; k_hat, v_hat: [B, Lc, Hkv, D].  Returns
    (out [B, Sq, Hq, D], lse [B, Hq, Sq]); a row that sees no key gets 0 and
    -inf; rows past a sequence are 0 / NaN."""
    q = np.asarray(q, np.float64)
    kh = np.asarray(k_hat, np.float64)
    vh = np.asarray(v_hat, np.float64)
    B, Sq, Hq, D = q.shape
    Hkv = kh.shape[2]
    G = Hq // Hkv
    if scale is None:
        scale = 1.0 / np.sqrt(D)
    we = w_eff(w, layer, l0)
    out = np.zeros((B, Sq, Hq, D))
    lse = np.full((B, Hq, Sq), np.nan)
    for b, segs in enumerate(segs_list):
        R = raw_len(segs)
        tau = visible_from(segs, we, mask_mode)
        L = len(tau)
        vis = tau[None, :] <= np.arange(R)[:, None]  # [R, L]
        for h in range(Hq):
            g = h // G
            s = scale * (q[b, :R, h] @ kh[b, :L, g].T)  # [R, L]
            s = np.where(vis, s, -np.inf)
            m = s.max(axis=1, initial=-np.inf)
            seen = np.isfinite(m)
            p = np.where(vis, np.exp(s - np.where(seen, m, 0.0)[:, None]), 0.0)
            l = p.sum(axis=1)
            o = np.zeros((R, D))
            o[seen] = (p[seen] @ vh[b, :L, g]) / l[seen][:, None]
            out[b, :R, h] = o
            lse[b, h, :R] = np.where(seen, m + np.log(np.where(seen, l, 1.0)), -np.inf)
    return out, lse


def attention_bwd(q, k_hat, v_hat, segs_list: List[Segs], w, layer, l0, dout, mask_mode=0,
                  scale=None):
    """Gradients of attention() (the chain rule of Eq. 5 under the mask):
    with P the row softmax over visible keys, dV = P^T dO, dP = dO V^T,
    dZ = P o (dP - rowsum(P o dP)), dQ = scale dZ K, dK = scale dZ^T Q (key
    gradients summed over the query heads of a KV head).  Returns
    (dq [B, Sq, Hq, D], dk [B, Lc, Hkv, D], dv [B, Lc, Hkv, D])."""
    q = np.asarray(q, np.float64)
    kh = np.asarray(k_hat, np.float64)
    vh = np.asarray(v_hat, np.float64)
    do = np.asarray(dout, np.float64)
    B, Sq, Hq, D = q.shape
    Hkv = kh.shape[2]
    G = Hq // Hkv
    if scale is None:
        scale = 1.0 / np.sqrt(D)
    we = w_eff(w, layer, l0)
    dq = np.zeros_like(q)
    dk = np.zeros_like(kh)
    dv = np.zeros_like(vh)
    for b, segs in enumerate(segs_list):
        R = raw_len(segs)
        tau = visible_from(segs, we, mask_mode)
        L = len(tau)
        vis = tau[None, :] <= np.arange(R)[:, None]
        for h in range(Hq):
            g = h // G
            s = np.where(vis, scale * (q[b, :R, h] @ kh[b, :L, g].T), -np.inf)
            m = s.max(axis=1, initial=-np.inf)
            seen = np.isfinite(m)
            p = np.where(vis, np.exp(s - np.where(seen, m, 0.0)[:, None]), 0.0)
            l = p.sum(axis=1)
            p[seen] /= l[seen][:, None]
            dp = do[b, :R, h] @ vh[b, :L, g].T
            dz = p * (dp - (p * dp).sum(axis=1, keepdims=True))
            dv[b, :L, g] += p.T @ do[b, :R, h]
            dq[b, :R, h] = scale * (dz @ kh[b, :L, g])
            dk[b, :L, g] += scale * (dz.T @ q[b, :R, h])
    return dq, dk, dv


def pool_bwd(k_raw, v_raw, segs_list: List[Segs], w, layer, l0, u, dk_hat, dv_hat):
    """Gradients of pool() (the chain rule of Eq. 4): for a window with
    weights a = softmax(u . k_j), da_j = dK^ . k_j + dV^ . v_j and
    ds_j = a_j (da_j - sum_i a_i da_i); dk_j = a_j dK^ + ds_j u,
    dv_j = a_j dV^, du = sum over windows of ds_j k_j.  Returns
    (dk_raw, dv_raw [B, S, Hkv, D], du [Hkv, D])."""
    k = np.asarray(k_raw, np.float64)
    v = np.asarray(v_raw, np.float64)
    gk = np.asarray(dk_hat, np.float64)
    gv = np.asarray(dv_hat, np.float64)
    B, S, H, D = k.shape
    uu = np.zeros((H, D)) if u is None else np.asarray(u, np.float64)
    we = w_eff(w, layer, l0)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    du = np.zeros((H, D))
    for b, segs in enumerate(segs_list):
        slots, _ = layout(segs, we)
        for c, (first, n, _, _) in enumerate(slots):
            kw = k[b, first:first + n]
            vw = v[b, first:first + n]
            for g in range(H):
                logits = kw[:, g] @ uu[g]
                a = np.exp(logits - logits.max())
                a /= a.sum()
                da = kw[:, g] @ gk[b, c, g] + vw[:, g] @ gv[b, c, g]
                ds = a * (da - a @ da)
                dk[b, first:first + n, g] = a[:, None] * gk[b, c, g][None] + ds[:, None] * uu[g][None]
                dv[b, first:first + n, g] = a[:, None] * gv[b, c, g][None]
                du[g] += ds @ kw[:, g]
    return dk, dv, du
