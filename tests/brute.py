"""Brute-force SpeechKV on tiny inputs, in pure Python loops.

An independent second statement of arXiv 2607.06827 Sec. III-B (Eq. 4 and
Eq. 5 with its causal mask), used to pin the fp64 oracle.  It is written
differently on purpose: every compressed key carries the explicit list of
full-resolution frames it stands for, and a query at position p may attend to
it when the frames it needs are all at or before p (mask "end": every frame of
the window; mask "start": its first frame).  No window count formula, no
visibility-time formula and no vectorised code are shared with the oracle.
"""
from __future__ import annotations

import math


def frame_groups(P: int, T: int, N: int, w_eff: int):
    """List of (frames, is_speech) for the compressed sequence of one sequence."""
    groups = [([c], False) for c in range(P)]
    start = P
    while start < P + T:
        frames = []
        f = start
        while f < P + T and len(frames) < w_eff:
            frames.append(f)
            f += 1
        groups.append((frames, True))
        start = f
    groups += [([P + T + m], False) for m in range(N)]
    return groups


def pool_one(k, v, P, T, N, w_eff, u):
    """k, v: nested lists [S][H][D] of one sequence; u: [H][D] or None.

    Returns (k_hat, v_hat, groups) with k_hat, v_hat nested [L][H][D].
    """
    H = len(k[0])
    D = len(k[0][0])
    groups = frame_groups(P, T, N, w_eff)
    k_hat, v_hat = [], []
    for frames, is_speech in groups:
        krow, vrow = [], []
        for g in range(H):
            if not is_speech:
                krow.append(list(k[frames[0]][g]))
                vrow.append(list(v[frames[0]][g]))
                continue
            logits = []
            for f in frames:
                s = 0.0
                for e in range(D):
                    s += (u[g][e] if u is not None else 0.0) * k[f][g][e]
                logits.append(s)
            top = max(logits)
            weights = [math.exp(s - top) for s in logits]
            total = sum(weights)
            alphas = [x / total for x in weights]
            kk = [0.0] * D
            vv = [0.0] * D
            for a, f in zip(alphas, frames):
                for e in range(D):
                    kk[e] += a * k[f][g][e]
                    vv[e] += a * v[f][g][e]
            krow.append(kk)
            vrow.append(vv)
        k_hat.append(krow)
        v_hat.append(vrow)
    return k_hat, v_hat, groups


def attend_one(q, k_hat, v_hat, groups, mask, scale):
    """q: nested [Sq][Hq][D] of one sequence.  Returns out nested [rows][Hq][D]
    for rows = every full-resolution position, and lse [Hq][rows]."""
    Hq = len(q[0])
    Hkv = len(k_hat[0]) if k_hat else 1
    G = Hq // Hkv
    D = len(q[0][0])
    rows = 1 + max((max(fr) for fr, _ in groups), default=-1)
    out = [[[0.0] * D for _ in range(Hq)] for _ in range(rows)]
    lse = [[-math.inf] * rows for _ in range(Hq)]
    for p in range(rows):
        for h in range(Hq):
            g = h // G
            seen = []
            for c, (frames, _) in enumerate(groups):
                need = max(frames) if mask == "end" else min(frames)
                if need <= p:
                    s = 0.0
                    for e in range(D):
                        s += q[p][h][e] * k_hat[c][g][e]
                    seen.append((c, scale * s))
            if not seen:
                continue
            top = max(z for _, z in seen)
            total = sum(math.exp(z - top) for _, z in seen)
            for c, z in seen:
                pc = math.exp(z - top) / total
                for e in range(D):
                    out[p][h][e] += pc * v_hat[c][g][e]
            lse[h][p] = top + math.log(total)
    return out, lse
