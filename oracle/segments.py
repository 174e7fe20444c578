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
