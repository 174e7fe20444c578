"""ctypes front end of the fp64 C oracle (speechkv_oracle.c).

TEST INFRASTRUCTURE ONLY.  See the header of speechkv_oracle.c for what is
computed and which passages of arXiv 2607.06827 each function follows.  Inputs
are numpy arrays; everything is converted to float64 and passed as dense
row-major arrays.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "speechkv_oracle.c")
_LIB = os.path.join(_HERE, "libspeechkv_oracle.so")
_lib = None


def build() -> str:
    """Compile the oracle with gcc (-O2, OpenMP, no fast-math).  Returns the path."""
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99", "-Wall",
           "-o", _LIB + ".tmp", _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(_LIB + ".tmp", _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        build()
    lib = ctypes.CDLL(_LIB)
    dp = ctypes.POINTER(ctypes.c_double)
    ip = ctypes.POINTER(ctypes.c_int)
    i = ctypes.c_int
    lib.speechkv_oracle_pool.argtypes = [dp, dp, i, i, i, i, ip, ip, ip, i, i, i,
                                         dp, dp, dp, i, ip]
    lib.speechkv_oracle_pool.restype = None
    lib.speechkv_oracle_attention.argtypes = [dp, dp, dp, i, i, i, i, i, i, ip, ip,
                                              ip, i, i, i, i, ctypes.c_double, dp, dp]
    lib.speechkv_oracle_attention.restype = None
    lib.speechkv_oracle_decode.argtypes = [dp, dp, dp, ip, i, i, i, i, i,
                                           ctypes.c_double, dp, dp]
    lib.speechkv_oracle_decode.restype = None
    lib.speechkv_oracle_attention_bwd.argtypes = [dp, dp, dp, i, i, i, i, i, i, ip, ip, ip, i,
                                                  i, i, i, ctypes.c_double, dp, dp, dp, dp]
    lib.speechkv_oracle_attention_bwd.restype = None
    lib.speechkv_oracle_pool_bwd.argtypes = [dp, dp, i, i, i, i, ip, ip, ip, i, i, i, dp, dp, dp,
                                             i, dp, dp, dp]
    lib.speechkv_oracle_pool_bwd.restype = None
    lib.speechkv_oracle_compressed_len.argtypes = [i, i, i, i, i, i]
    lib.speechkv_oracle_compressed_len.restype = i
    lib.speechkv_oracle_num_threads.argtypes = []
    lib.speechkv_oracle_num_threads.restype = i
    _lib = lib
    return lib


def _f64(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _i32(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32).reshape(-1))


def _dp(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _ip(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int))


def num_threads() -> int:
    """OpenMP threads the oracle runs on."""
    return int(_load().speechkv_oracle_num_threads())


def compressed_len(P: int, T: int, N: int, w: int, layer: int, l0: int) -> int:
    """P + ceil(T / w_eff) + N with w_eff = w if layer >= l0 else 1."""
    return int(_load().speechkv_oracle_compressed_len(P, T, N, w, layer, l0))


def pool(k_raw, v_raw, P, T, N, w, layer, l0, u=None, Lc=None):
    """Eq. 4 on one layer.  k_raw, v_raw: [B, S, Hkv, D]; u: [Hkv, D] or None.

    Returns (k_hat, v_hat, clen) with k_hat, v_hat of shape [B, Lc, Hkv, D]
    (zero beyond each sequence's compressed length) and clen [B] int32.
    """
    lib = _load()
    k = _f64(k_raw)
    v = _f64(v_raw)
    B, S, H, D = k.shape
    assert v.shape == k.shape
    P, T, N = _i32(P), _i32(T), _i32(N)
    assert P.shape == T.shape == N.shape == (B,)
    assert np.all(P + T + N <= S) and np.all(P >= 0) and np.all(T >= 0) and np.all(N >= 0)
    lens = [compressed_len(int(P[b]), int(T[b]), int(N[b]), w, layer, l0) for b in range(B)]
    if Lc is None:
        Lc = max(max(lens), 1)
    assert Lc >= max(lens)
    uu = None if u is None else _f64(u)
    if uu is not None:
        assert uu.shape == (H, D)
    kh = np.zeros((B, Lc, H, D), np.float64)
    vh = np.zeros((B, Lc, H, D), np.float64)
    clen = np.zeros(B, np.int32)
    lib.speechkv_oracle_pool(_dp(k), _dp(v), B, S, H, D, _ip(P), _ip(T), _ip(N), w,
                             layer, l0, _dp(uu) if uu is not None else None,
                             _dp(kh), _dp(vh), Lc, _ip(clen))
    return kh, vh, clen


def attention(q, k_hat, v_hat, P, T, N, w, layer, l0, mask_mode=0, scale=None):
    """Eq. 5 with the causal mask over the compressed sequence, every row.

    q: [B, Sq, Hq, D]; k_hat, v_hat: [B, Lc, Hkv, D].
    Returns (out [B, Sq, Hq, D], lse [B, Hq, Sq]); rows p >= P+T+N are 0 / NaN.
    """
    lib = _load()
    q = _f64(q)
    kh = _f64(k_hat)
    vh = _f64(v_hat)
    B, Sq, Hq, D = q.shape
    _, Lc, Hkv, D2 = kh.shape
    assert D2 == D and vh.shape == kh.shape and Hq % Hkv == 0
    P, T, N = _i32(P), _i32(T), _i32(N)
    assert np.all(P + T + N <= Sq)
    if scale is None:
        scale = 1.0 / np.sqrt(D)
    out = np.zeros((B, Sq, Hq, D), np.float64)
    lse = np.zeros((B, Hq, Sq), np.float64)
    lib.speechkv_oracle_attention(_dp(q), _dp(kh), _dp(vh), B, Sq, Hq, Hkv, D, Lc,
                                  _ip(P), _ip(T), _ip(N), w, layer, l0, mask_mode,
                                  float(scale), _dp(out), _dp(lse))
    return out, lse


def decode(q, k_hat, v_hat, clen, scale=None):
    """One decode step: q [B, Hq, D] over every cached key c < clen[b].

    Returns (out [B, Hq, D], lse [B, Hq]).
    """
    lib = _load()
    q = _f64(q)
    kh = _f64(k_hat)
    vh = _f64(v_hat)
    B, Hq, D = q.shape
    _, Lc, Hkv, _ = kh.shape
    clen = _i32(clen)
    assert clen.shape == (B,) and np.all(clen <= Lc)
    if scale is None:
        scale = 1.0 / np.sqrt(D)
    out = np.zeros((B, Hq, D), np.float64)
    lse = np.zeros((B, Hq), np.float64)
    lib.speechkv_oracle_decode(_dp(q), _dp(kh), _dp(vh), _ip(clen), B, Hq, Hkv, D, Lc,
                               float(scale), _dp(out), _dp(lse))
    return out, lse


def attention_bwd(q, k_hat, v_hat, P, T, N, w, layer, l0, dout, mask_mode=0, scale=None):
    """Gradient of `attention`'s output against dout: (dq, dk_hat, dv_hat).

    q, dout: [B, Sq, Hq, D]; k_hat, v_hat: [B, Lc, Hkv, D].  Rows that see no
    key and rows p >= P+T+N get dq = 0; key rows past a compressed length 0.
    """
    lib = _load()
    q, kh, vh, go = _f64(q), _f64(k_hat), _f64(v_hat), _f64(dout)
    B, Sq, Hq, D = q.shape
    _, Lc, Hkv, D2 = kh.shape
    assert D2 == D and vh.shape == kh.shape and go.shape == q.shape and Hq % Hkv == 0
    P, T, N = _i32(P), _i32(T), _i32(N)
    assert np.all(P + T + N <= Sq)
    if scale is None:
        scale = 1.0 / np.sqrt(D)
    dq = np.zeros_like(q)
    dk = np.zeros_like(kh)
    dv = np.zeros_like(vh)
    lib.speechkv_oracle_attention_bwd(_dp(q), _dp(kh), _dp(vh), B, Sq, Hq, Hkv, D, Lc, _ip(P),
                                      _ip(T), _ip(N), w, layer, l0, mask_mode, float(scale),
                                      _dp(go), _dp(dq), _dp(dk), _dp(dv))
    return dq, dk, dv


def pool_bwd(k_raw, v_raw, P, T, N, w, layer, l0, u, dk_hat, dv_hat):
    """Gradient of `pool` against (dk_hat, dv_hat): (dk_raw, dv_raw, du).

    k_raw, v_raw: [B, S, Hkv, D]; u: [Hkv, D] or None (the zero gate, whose
    gradient du is still returned); dk_hat, dv_hat: [B, Lc, Hkv, D].
    """
    lib = _load()
    k, v, gk, gv = _f64(k_raw), _f64(v_raw), _f64(dk_hat), _f64(dv_hat)
    B, S, H, D = k.shape
    Lc = gk.shape[1]
    assert v.shape == k.shape and gk.shape == (B, Lc, H, D) and gv.shape == gk.shape
    P, T, N = _i32(P), _i32(T), _i32(N)
    assert np.all(P + T + N <= S)
    assert Lc >= max(compressed_len(int(P[b]), int(T[b]), int(N[b]), w, layer, l0)
                     for b in range(B))
    uu = None if u is None else _f64(u)
    if uu is not None:
        assert uu.shape == (H, D)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    du = np.zeros((H, D), np.float64)
    lib.speechkv_oracle_pool_bwd(_dp(k), _dp(v), B, S, H, D, _ip(P), _ip(T), _ip(N), w, layer,
                                 l0, _dp(uu) if uu is not None else None, _dp(gk), _dp(gv), Lc,
                                 _dp(dk), _dp(dv), _dp(du))
    return dk, dv, du
