"""Pins of the multi-run oracle (oracle/segments.py) to things other than
itself: the single-run C oracle (pinned on its own in test_oracle_pins.py),
invariances that Eq. 4 and the mask fix (a run split at a multiple of w from
its start, text runs that meet, the independence of one run's windows from
the other runs), and a brute-force visibility rule on tiny inputs."""
import itertools

import numpy as np
import pytest

import oracle
from oracle import segments as seg


def rand(shape, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


@pytest.mark.parametrize("P,T,N,w", [(8, 60, 5, 4), (0, 37, 3, 4), (5, 3, 4, 8), (7, 0, 6, 4),
                                     (4, 45, 0, 6), (3, 41, 2, 1), (0, 9, 0, 3), (2, 7, 5, 4)])
@pytest.mark.parametrize("mode", [0, 1])
def test_one_run_equals_single_span_oracle(P, T, N, w, mode):
    S, H, Hq, D = P + T + N, 2, 4, 16
    k, v = rand((1, S, H, D), 1), rand((1, S, H, D), 2)
    u, q = rand((H, D), 3, 0.5), rand((1, S, Hq, D), 4)
    segs = [[(P, T), (N, 0)]]
    kh, vh, clen = seg.pool(k, v, segs, w, 1, 0, u)
    rk, rv, rclen = oracle.pool(k, v, [P], [T], [N], w, 1, 0, u)
    assert clen.tolist() == rclen.tolist()
    L = int(clen[0])
    np.testing.assert_allclose(kh[0, :L], rk[0, :L], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(vh[0, :L], rv[0, :L], rtol=1e-12, atol=1e-12)
    out, lse = seg.attention(q, kh, vh, segs, w, 1, 0, mode)
    ro, rl = oracle.attention(q, rk, rv, [P], [T], [N], w, 1, 0, mode)
    np.testing.assert_allclose(out[0, :S], ro[0, :S], rtol=1e-10, atol=1e-12)
    assert np.array_equal(np.isneginf(lse[0, :, :S]), np.isneginf(rl[0, :, :S]))
    fin = np.isfinite(rl[0, :, :S])
    np.testing.assert_allclose(lse[0, :, :S][fin], rl[0, :, :S][fin], rtol=1e-12, atol=1e-12)


def test_identity_below_l0_keeps_every_row():
    segs = [[(3, 10), (2, 7), (4, 0)]]
    S = seg.raw_len(segs[0])
    k, v = rand((1, S, 2, 8), 5), rand((1, S, 2, 8), 6)
    kh, vh, clen = seg.pool(k, v, segs, 4, 2, 5, rand((2, 8), 7))
    assert int(clen[0]) == S
    np.testing.assert_array_equal(kh[0], k[0])
    np.testing.assert_array_equal(vh[0], v[0])


@pytest.mark.parametrize("mode", [0, 1])
def test_split_at_multiple_of_w_changes_nothing(mode):
    """Windows start at each run's first frame: a run cut where a window ends
    (with no text between the halves) pools and attends exactly as the whole."""
    whole = [[(5, 24), (3, 0)]]
    cut = [[(5, 8), (0, 16), (3, 0)]]
    S, w = 32, 4
    k, v, u = rand((1, S, 2, 8), 8), rand((1, S, 2, 8), 9), rand((2, 8), 10)
    q = rand((1, S, 4, 8), 11)
    a = seg.pool(k, v, whole, w, 0, 0, u)
    b = seg.pool(k, v, cut, w, 0, 0, u)
    np.testing.assert_array_equal(a[2], b[2])
    np.testing.assert_allclose(a[0], b[0], rtol=0, atol=0)
    oa, la = seg.attention(q, a[0], a[1], whole, w, 0, 0, mode)
    ob, lb = seg.attention(q, b[0], b[1], cut, w, 0, 0, mode)
    np.testing.assert_allclose(oa, ob, rtol=0, atol=0)


def test_split_off_a_window_boundary_realigns():
    """Cut where no window ends, the second run's windows start at the cut:
    the compressed lengths and rows differ from the whole run's."""
    S, w = 12, 4
    k, v, u = rand((1, S, 1, 8), 12), rand((1, S, 1, 8), 13), rand((1, 8), 14)
    a = seg.pool(k, v, [[(0, 12)]], w, 0, 0, u)
    b = seg.pool(k, v, [[(0, 6), (0, 6)]], w, 0, 0, u)
    assert int(a[2][0]) == 3 and int(b[2][0]) == 4
    # the second run's first window pools frames 6..9, not 4..7 or 8..11
    kw = k[0, 6:10, 0]
    lg = kw @ u[0]
    al = np.exp(lg - lg.max())
    al /= al.sum()
    np.testing.assert_allclose(b[0][0, 2, 0], al @ kw, rtol=1e-12)


def test_text_runs_merge():
    segs_a = [[(3, 0), (4, 10), (2, 0), (5, 6)]]
    segs_b = [[(7, 10), (7, 6)]]
    S = 31
    k, v, u = rand((1, S, 2, 8), 15), rand((1, S, 2, 8), 16), rand((2, 8), 17)
    q = rand((1, S, 4, 8), 18)
    a = seg.pool(k, v, segs_a, 4, 0, 0, u)
    b = seg.pool(k, v, segs_b, 4, 0, 0, u)
    np.testing.assert_array_equal(a[0], b[0])
    oa, _ = seg.attention(q, a[0], a[1], segs_a, 4, 0, 0)
    ob, _ = seg.attention(q, b[0], b[1], segs_b, 4, 0, 0)
    np.testing.assert_array_equal(oa, ob)


def test_runs_pool_independently():
    """A pooled row depends only on its own window's frames."""
    segs = [[(2, 9), (3, 11), (1, 0)]]
    S = seg.raw_len(segs[0])
    k, v, u = rand((1, S, 1, 8), 19), rand((1, S, 1, 8), 20), rand((1, 8), 21)
    kh, _, _ = seg.pool(k, v, segs, 4, 0, 0, u)
    k2 = k.copy()
    k2[0, 2:11] += 5.0  # the first run's frames
    kh2, _, _ = seg.pool(k2, v, segs, 4, 0, 0, u)
    L0 = 2 + 3  # text + first run's windows
    assert not np.allclose(kh[0, 2:L0], kh2[0, 2:L0])
    np.testing.assert_array_equal(kh[0, L0:], kh2[0, L0:])


@pytest.mark.parametrize("mode", [0, 1])
def test_visibility_brute_force(mode):
    """Every (row, key) pair on tiny sequences: a text key is visible from
    its own row on; a window in mode 0 once every one of its frames is at or
    before the row, in mode 1 once any is."""
    for segs in ([(0, 5), (2, 3)], [(1, 0), (0, 7)], [(2, 2), (0, 0), (1, 9), (3, 0)]):
        for w in (1, 2, 3, 4):
            slots, R = seg.layout(segs, w)
            tau = seg.visible_from(segs, w, mode)
            for p, (c, (first, n, _, _)) in itertools.product(range(R), enumerate(slots)):
                frames = range(first, first + n)
                want = all(f <= p for f in frames) if mode == 0 else any(f <= p for f in frames)
                assert (tau[c] <= p) == want, (segs, w, p, c)


def test_lengths():
    assert seg.compressed_len([(32, 375), (24, 250), (16, 500), (64, 0)], 4, 1, 0) == \
        32 + 94 + 24 + 63 + 16 + 125 + 64
    assert seg.compressed_len([(32, 375), (24, 250)], 4, 0, 1) == 32 + 375 + 24 + 250
    assert seg.compressed_len([], 4, 1, 0) == 0


_LAYOUT = seg.layout  # the layout under test, before any mutant replaces it


def _layout_global_windows(segs, w):
    """Mutant: windows aligned to multiples of w from the sequence start
    instead of each run's first frame."""
    slots, r = [], 0
    for t_len, s_len in segs:
        slots += [(r + i, 1, r + i, r + i) for i in range(t_len)]
        r += t_len
        frames = list(range(r, r + s_len))
        for _, grp in itertools.groupby(frames, key=lambda f: f // w):
            g = list(grp)
            slots.append((g[0], len(g), g[-1], g[0]))
        r += s_len
    return slots, r


def _layout_tau_first(segs, w):
    """Mutant: a window visible from its first frame in mode 0 as well."""
    slots, r = _LAYOUT(segs, w)
    return [(a, n, s, s) for a, n, _, s in slots], r


def _layout_last_window_full(segs, w):
    """Mutant: the short last window of a run takes w frames anyway."""
    slots, r = _LAYOUT(segs, w)
    return [(a, w if n > 1 else n, e, s) for a, n, e, s in slots], r


@pytest.mark.parametrize("mutant", [_layout_global_windows, _layout_tau_first,
                                    _layout_last_window_full])
def test_pins_catch_planted_mistakes(mutant, monkeypatch):
    monkeypatch.setattr(seg, "layout", mutant)
    checks = [
        lambda: test_one_run_equals_single_span_oracle(4, 45, 0, 6, 0),
        lambda: test_one_run_equals_single_span_oracle(2, 7, 5, 4, 0),
        lambda: test_split_at_multiple_of_w_changes_nothing(0),
        lambda: test_split_off_a_window_boundary_realigns(),
        lambda: test_visibility_brute_force(0),
        lambda: test_lengths(),
    ]
    caught = 0
    for check in checks:
        try:
            check()
        except (AssertionError, IndexError, ValueError):
            caught += 1
    assert caught > 0, f"{mutant.__name__} passed every pin"


# ------------------------------------------------------------------ backward

@pytest.mark.parametrize("P,T,N,w,mode", [(8, 30, 5, 4, 0), (0, 19, 3, 4, 1), (3, 11, 2, 1, 0),
                                          (2, 7, 5, 4, 0)])
def test_one_run_backward_equals_single_span_oracle(P, T, N, w, mode):
    S, H, Hq, D = P + T + N, 2, 4, 8
    k, v = rand((1, S, H, D), 31), rand((1, S, H, D), 32)
    u, q, do = rand((H, D), 33, 0.5), rand((1, S, Hq, D), 34), rand((1, S, Hq, D), 35)
    segs = [[(P, T), (N, 0)]]
    kh, vh, clen = seg.pool(k, v, segs, w, 1, 0, u)
    dq, dkh, dvh = seg.attention_bwd(q, kh, vh, segs, w, 1, 0, do, mode)
    rq, rk, rv = oracle.attention_bwd(q, kh, vh, [P], [T], [N], w, 1, 0, do, mode)
    L = int(clen[0])
    np.testing.assert_allclose(dq[0, :S], rq[0, :S], rtol=1e-9, atol=1e-12)
    np.testing.assert_allclose(dkh[0, :L], rk[0, :L], rtol=1e-9, atol=1e-12)
    np.testing.assert_allclose(dvh[0, :L], rv[0, :L], rtol=1e-9, atol=1e-12)
    dk, dv, du = seg.pool_bwd(k, v, segs, w, 1, 0, u, dkh, dvh)
    pk, pv, pu = oracle.pool_bwd(k, v, [P], [T], [N], w, 1, 0, u, dkh, dvh)
    np.testing.assert_allclose(dk[0, :S], pk[0, :S], rtol=1e-9, atol=1e-12)
    np.testing.assert_allclose(dv[0, :S], pv[0, :S], rtol=1e-9, atol=1e-12)
    np.testing.assert_allclose(du, pu, rtol=1e-9, atol=1e-12)


@pytest.mark.parametrize("mode", [0, 1])
def test_backward_finite_differences_several_runs(mode):
    """The chain pool -> attention over three runs: the gradients of
    L = sum(dout * out) match central differences of the pinned forward in
    random directions, for q, the raw keys and values, and the gate."""
    segs = [[(2, 9), (3, 6), (0, 5), (2, 0)], [(0, 7), (1, 2)]]
    S = max(seg.raw_len(s) for s in segs)
    B, H, Hq, D, w = 2, 2, 4, 8, 3
    k, v = rand((B, S, H, D), 41), rand((B, S, H, D), 42)
    u, q, do = rand((H, D), 43, 0.7), rand((B, S, Hq, D), 44), rand((B, S, Hq, D), 45)
    rows = [seg.raw_len(s) for s in segs]
    for b, R in enumerate(rows):  # rows past a sequence carry no gradient
        do[b, R:] = 0.0

    def loss(q_, k_, v_, u_):
        kh, vh, _ = seg.pool(k_, v_, segs, w, 1, 0, u_)
        out, _ = seg.attention(q_, kh, vh, segs, w, 1, 0, mode)
        return float((out * do).sum())

    kh, vh, _ = seg.pool(k, v, segs, w, 1, 0, u)
    dq, dkh, dvh = seg.attention_bwd(q, kh, vh, segs, w, 1, 0, do, mode)
    dk, dv, du = seg.pool_bwd(k, v, segs, w, 1, 0, u, dkh, dvh)
    eps = 1e-5
    for name, x, grad in (("q", q, dq), ("k", k, dk), ("v", v, dv), ("u", u, du)):
        dirn = rand(x.shape, 46 + len(name))
        args = dict(q_=q, k_=k, v_=v, u_=u)
        key = name + "_"
        args[key] = x + eps * dirn
        lp = loss(**args)
        args[key] = x - eps * dirn
        lm = loss(**args)
        fd = (lp - lm) / (2 * eps)
        an = float((grad * dirn).sum())
        assert abs(fd - an) <= 1e-6 * max(1.0, abs(fd)), (name, fd, an)
