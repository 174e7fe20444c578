"""ctypes binding of libspeechkv.so (include/speechkv.h), same names as the C ABI.

Argument marshalling only: tensors become device pointers, strides and sizes
become integers, and a non-zero status becomes a SpeechKVError.  Every step of
the hot path runs in the library's HIP kernels; nothing here computes.  The
module raises ImportError when the library has not been built.

Tensors are torch tensors on the current HIP device (PyTorch is used for
device memory and streams only).  `stream` defaults to torch's current stream.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Optional

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libspeechkv.so")
if not os.path.exists(_LIB_PATH):
    raise ImportError(f"{_LIB_PATH} is not built: run `python -m paper_2607_06827_amd.build`")
_lib = ctypes.CDLL(_LIB_PATH)

OK = 0
ERR_INVALID_ARG = -1
ERR_UNSUPPORTED = -2
ERR_WORKSPACE = -3
ERR_ALIAS = -4
ERR_HIP = -5
ERR_SCRATCH = -6
DTYPE_F32 = 0
DTYPE_BF16 = 1
MASK_WINDOW_END = 0
MASK_WINDOW_START = 1
MAX_WINDOW = 65536  # largest window size the pooling and attention calls take
MAX_SEGMENTS = 1024  # most segments one sequence of a segment table may have
NOALLOC_SCRATCH_BYTES = 16 << 20  # static split scratch of speechkv_decode_attn_noalloc, per GPU

LIBRARY_PATH = _LIB_PATH


class _PagedKV(ctypes.Structure):
    _fields_ = [("k_pages", ctypes.c_void_p), ("v_pages", ctypes.c_void_p),
                ("block_table", ctypes.c_void_p), ("num_pages", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("max_pages_per_seq", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("dtype", ctypes.c_int32)]


class _Spans(ctypes.Structure):
    _fields_ = [("prefix_len", ctypes.c_void_p), ("speech_len", ctypes.c_void_p),
                ("suffix_len", ctypes.c_void_p), ("max_speech_len", ctypes.c_int32),
                ("max_total_len", ctypes.c_int32)]


class _Segments(ctypes.Structure):
    _fields_ = [("seg_start", ctypes.c_void_p), ("text_len", ctypes.c_void_p),
                ("speech_len", ctypes.c_void_p), ("num_segments", ctypes.c_int32),
                ("max_segments", ctypes.c_int32), ("max_total_len", ctypes.c_int32)]


_vp, _i32, _i64, _f32, _sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_size_t
_lib.speechkv_pool_kv.argtypes = [_vp, _vp, _i64, _i64, _i64, _i32, _i32, ctypes.POINTER(_Spans),
                                  _i32, _vp, _i32, _i32, ctypes.POINTER(_PagedKV), _vp, _vp]
_lib.speechkv_pool_kv.restype = ctypes.c_int
_lib.speechkv_pool_kv_segments.argtypes = [_vp, _vp, _i64, _i64, _i64, _i32, _i32,
                                           ctypes.POINTER(_Segments), _i32, _vp, _i32, _i32,
                                           ctypes.POINTER(_PagedKV), _vp, _vp]
_lib.speechkv_pool_kv_segments.restype = ctypes.c_int
_lib.speechkv_prefill_attn_segments.argtypes = [_vp, _i32, _i32, _i32, ctypes.POINTER(_PagedKV),
                                                ctypes.POINTER(_Segments), _i32, _i32, _i32, _i32,
                                                ctypes.c_float, _vp, _vp, _vp]
_lib.speechkv_prefill_attn_segments.restype = ctypes.c_int
_lib.speechkv_compressed_len_segments.argtypes = [_vp, _vp, _i32, _i32, _i32, _i32]
_lib.speechkv_compressed_len_segments.restype = _i64
_lib.speechkv_pool_hidden.argtypes = [_vp, _i64, _i64, _i32, _i32, _i32, _i32, ctypes.POINTER(_Spans),
                                      _i32, _vp, _vp, _i64, _i64, _i32, _vp, _vp]
_lib.speechkv_pool_hidden.restype = ctypes.c_int
_lib.speechkv_decode_attn.argtypes = [_vp, _i32, _i32, ctypes.POINTER(_PagedKV), _vp, _i32, _vp,
                                      _vp, _f32, _i32, _vp, _vp, _sz, _vp]
_lib.speechkv_decode_attn.restype = ctypes.c_int
_lib.speechkv_decode_attn_noalloc.argtypes = [_vp, _i32, _i32, ctypes.POINTER(_PagedKV), _vp, _i32,
                                              _vp, _vp, _f32, _i32, _vp, _vp]
_lib.speechkv_decode_attn_noalloc.restype = ctypes.c_int
_lib.speechkv_prefill_attn.argtypes = [_vp, _i32, _i32, _i32, ctypes.POINTER(_PagedKV),
                                       ctypes.POINTER(_Spans), _i32, _i32, _i32, _i32, _f32, _vp,
                                       _vp, _vp]
_lib.speechkv_prefill_attn.restype = ctypes.c_int
_lib.speechkv_pool_prefill_attn.argtypes = [_vp, _i32, _i32, _i32, _vp, _vp, _i64, _i64, _i64, _i32,
                                            ctypes.POINTER(_Spans), _i32, _vp, _i32, _i32,
                                            ctypes.POINTER(_PagedKV), _vp, _i32, ctypes.c_float,
                                            _vp, _vp, _vp]
_lib.speechkv_pool_prefill_attn.restype = ctypes.c_int
_lib.speechkv_prefill_attn_bwd.argtypes = [_vp, _i32, _i32, _i32, ctypes.POINTER(_PagedKV),
                                           ctypes.POINTER(_Spans), _i32, _i32, _i32, _i32, _f32,
                                           _vp, _vp, _vp, _vp, _vp, _vp, _i32, _vp, _sz, _vp]
_lib.speechkv_prefill_attn_bwd.restype = ctypes.c_int
_lib.speechkv_prefill_attn_bwd_segments.argtypes = [_vp, _i32, _i32, _i32, ctypes.POINTER(_PagedKV),
                                                    ctypes.POINTER(_Segments), _i32, _i32, _i32,
                                                    _i32, _f32, _vp, _vp, _vp, _vp, _vp, _vp, _i32,
                                                    _vp, _sz, _vp]
_lib.speechkv_prefill_attn_bwd_segments.restype = ctypes.c_int
_lib.speechkv_prefill_attn_bwd_workspace_bytes.argtypes = [_i32, _i32, _i32]
_lib.speechkv_prefill_attn_bwd_workspace_bytes.restype = _sz
_lib.speechkv_pool_kv_bwd.argtypes = [_vp, _vp, _i64, _i64, _i64, _i32, _i32, _i32, _i32, _i32,
                                      ctypes.POINTER(_Spans), _i32, _vp, _i32, _i32, _vp, _vp, _i32,
                                      _vp, _vp, _vp, _vp, _sz, _vp]
_lib.speechkv_pool_kv_bwd.restype = ctypes.c_int
_lib.speechkv_pool_kv_bwd_segments.argtypes = [_vp, _vp, _i64, _i64, _i64, _i32, _i32, _i32, _i32,
                                               _i32, ctypes.POINTER(_Segments), _i32, _vp, _i32,
                                               _i32, _vp, _vp, _i32, _vp, _vp, _vp, _vp, _sz, _vp]
_lib.speechkv_pool_kv_bwd_segments.restype = ctypes.c_int
_lib.speechkv_pool_kv_bwd_workspace_bytes.argtypes = [_i32, _i32, _i32, _i32]
_lib.speechkv_pool_kv_bwd_workspace_bytes.restype = _sz
_lib.speechkv_compressed_len.argtypes = [_i32] * 6
_lib.speechkv_compressed_len.restype = _i64
_lib.speechkv_decode_num_splits.argtypes = [_i32, _i32, _i32]
_lib.speechkv_decode_num_splits.restype = _i32
_lib.speechkv_decode_workspace_bytes.argtypes = [_i32] * 6
_lib.speechkv_decode_workspace_bytes.restype = _sz
_lib.speechkv_status_string.argtypes = [ctypes.c_int]
_lib.speechkv_status_string.restype = ctypes.c_char_p
_lib.speechkv_version.argtypes = []
_lib.speechkv_version.restype = ctypes.c_char_p


class SpeechKVError(RuntimeError):
    def __init__(self, status: int, call: str):
        super().__init__(f"{call}: {speechkv_status_string(status)} (status {status})")
        self.status = status


@dataclasses.dataclass
class PagedKV:
    """One layer's paged cache: k_pages/v_pages [num_pages, Hkv, page_size, D]
    and block_table [B, max_pages_per_seq] int32, all on the device."""

    k_pages: torch.Tensor
    v_pages: torch.Tensor
    block_table: torch.Tensor

    def _c(self) -> _PagedKV:
        k, v, t = self.k_pages, self.v_pages, self.block_table
        for x in (k, v, t):
            if not x.is_contiguous():
                raise ValueError("paged cache tensors must be contiguous")
        if k.shape != v.shape or k.dim() != 4 or k.dtype != v.dtype:
            raise ValueError("k_pages and v_pages must share one [pages, heads, page, dim] shape")
        if t.dtype != torch.int32 or t.dim() != 2:
            raise ValueError("block_table must be int32 [batch, max_pages]")
        return _PagedKV(k.data_ptr(), v.data_ptr(), t.data_ptr(), k.shape[0], k.shape[2],
                        t.shape[1], k.shape[1], k.shape[3], _dtype_code(k.dtype))


@dataclasses.dataclass
class Spans:
    """Per-sequence text-prefix, speech and text-suffix lengths (device int32
    [B]) with host-side upper bounds."""

    prefix_len: torch.Tensor
    speech_len: torch.Tensor
    suffix_len: torch.Tensor
    max_speech_len: int
    max_total_len: int

    def _c(self) -> _Spans:
        for x in (self.prefix_len, self.speech_len, self.suffix_len):
            if x.dtype != torch.int32 or not x.is_contiguous():
                raise ValueError("span lengths must be contiguous int32 tensors")
        return _Spans(self.prefix_len.data_ptr(), self.speech_len.data_ptr(),
                      self.suffix_len.data_ptr(), self.max_speech_len, self.max_total_len)


@dataclasses.dataclass
class Segments:
    """Sequences with several speech runs: sequence b is its segments
    [seg_start[b], seg_start[b+1]), segment i being text_len[i] text rows then
    speech_len[i] speech frames (device int32 tensors), with host-side bounds
    on the segments of one sequence and on its rows."""

    seg_start: torch.Tensor
    text_len: torch.Tensor
    speech_len: torch.Tensor
    max_segments: int
    max_total_len: int

    def _c(self) -> _Segments:
        for x in (self.seg_start, self.text_len, self.speech_len):
            if x.dtype != torch.int32 or not x.is_contiguous():
                raise ValueError("segment tables must be contiguous int32 tensors")
        if self.text_len.shape != self.speech_len.shape:
            raise ValueError("text_len and speech_len must have one entry per segment")
        return _Segments(self.seg_start.data_ptr(), self.text_len.data_ptr(),
                         self.speech_len.data_ptr(), self.text_len.numel(), self.max_segments,
                         self.max_total_len)

    @staticmethod
    def from_lists(segs, device="cuda") -> "Segments":
        """Build the table from [[(text_len, speech_len), ...] per sequence]."""
        start = [0]
        for s in segs:
            start.append(start[-1] + len(s))
        flat = [x for s in segs for x in s]
        i32 = lambda v: torch.tensor(v, dtype=torch.int32, device=device)
        return Segments(i32(start), i32([t for t, _ in flat] or [0]),
                        i32([s for _, s in flat] or [0]), max([len(s) for s in segs] or [0]),
                        max([sum(t + s for t, s in x) for x in segs] or [0]))


def _dtype_code(dt: torch.dtype) -> int:
    if dt == torch.bfloat16:
        return DTYPE_BF16
    if dt == torch.float32:
        return DTYPE_F32
    return 99  # the library rejects it as unsupported


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(status: int, call: str):
    if status != OK:
        raise SpeechKVError(status, call)


def speechkv_pool_kv(k_raw: torch.Tensor, v_raw: torch.Tensor, spans: Spans, w: int,
                     gate_u: Optional[torch.Tensor], layer: int, l0: int, cache: PagedKV,
                     cache_len_out: Optional[torch.Tensor] = None, stream=None) -> None:
    """k_raw, v_raw: [B, S_raw, Hkv, D] views with a contiguous last axis."""
    if k_raw.shape != v_raw.shape or k_raw.stride() != v_raw.stride():
        raise ValueError("k_raw and v_raw must have one shape and one stride")
    if k_raw.dim() != 4 or k_raw.stride(3) != 1:
        raise ValueError("raw K/V must be [B, S, Hkv, D] with a contiguous last axis")
    sb, ss, sh, _ = k_raw.stride()
    c = cache._c()
    s = spans._c()
    st = _lib.speechkv_pool_kv(k_raw.data_ptr(), v_raw.data_ptr(), sb, ss, sh, k_raw.shape[0],
                               k_raw.shape[1], ctypes.byref(s), w, _ptr(gate_u), layer, l0,
                               ctypes.byref(c), _ptr(cache_len_out), _stream(stream))
    _check(st, "speechkv_pool_kv")


def speechkv_pool_kv_segments(k_raw: torch.Tensor, v_raw: torch.Tensor, segs: Segments, w: int,
                              gate_u: Optional[torch.Tensor], layer: int, l0: int, cache: PagedKV,
                              cache_len_out: Optional[torch.Tensor] = None, stream=None) -> None:
    """k_raw, v_raw: [B, S_raw, Hkv, D] views with a contiguous last axis."""
    if k_raw.shape != v_raw.shape or k_raw.stride() != v_raw.stride():
        raise ValueError("k_raw and v_raw must have one shape and one stride")
    if k_raw.dim() != 4 or k_raw.stride(3) != 1:
        raise ValueError("raw K/V must be [B, S, Hkv, D] with a contiguous last axis")
    sb, ss, sh, _ = k_raw.stride()
    c = cache._c()
    g = segs._c()
    st = _lib.speechkv_pool_kv_segments(k_raw.data_ptr(), v_raw.data_ptr(), sb, ss, sh,
                                        k_raw.shape[0], k_raw.shape[1], ctypes.byref(g), w,
                                        _ptr(gate_u), layer, l0, ctypes.byref(c),
                                        _ptr(cache_len_out), _stream(stream))
    _check(st, "speechkv_pool_kv_segments")


def speechkv_prefill_attn_segments(q: torch.Tensor, cache: PagedKV, segs: Segments, w: int,
                                   layer: int, l0: int, out: torch.Tensor,
                                   mask_mode: int = MASK_WINDOW_END, scale: Optional[float] = None,
                                   lse: Optional[torch.Tensor] = None, stream=None) -> None:
    """q, out: [B, q_len, Hq, D] contiguous; lse: [B, Hq, q_len] fp32 or None."""
    for x in (q, out) + ((lse,) if lse is not None else ()):
        if not x.is_contiguous():
            raise ValueError("prefill tensors must be contiguous")
    B, q_len, Hq, D = q.shape
    if scale is None:
        scale = D ** -0.5
    c = cache._c()
    g = segs._c()
    st = _lib.speechkv_prefill_attn_segments(q.data_ptr(), B, Hq, q_len, ctypes.byref(c),
                                             ctypes.byref(g), w, layer, l0, mask_mode, scale,
                                             out.data_ptr(), _ptr(lse), _stream(stream))
    _check(st, "speechkv_prefill_attn_segments")


def speechkv_compressed_len_segments(segs, w: int, layer: int, l0: int) -> int:
    """Compressed length of one sequence given as [(text_len, speech_len), ...]."""
    n = len(segs)
    t = (ctypes.c_int32 * max(n, 1))(*[x for x, _ in segs])
    s = (ctypes.c_int32 * max(n, 1))(*[y for _, y in segs])
    return int(_lib.speechkv_compressed_len_segments(ctypes.cast(t, _vp), ctypes.cast(s, _vp), n,
                                                     w, layer, l0))


def speechkv_pool_hidden(h: torch.Tensor, spans: Spans, w: int, gate_u: Optional[torch.Tensor],
                         out: torch.Tensor, out_len: Optional[torch.Tensor] = None,
                         stream=None) -> None:
    """h: [B, S_raw, hidden], out: [B, S_out, hidden], both with a contiguous last axis."""
    if h.dim() != 3 or out.dim() != 3 or h.stride(2) != 1 or out.stride(2) != 1:
        raise ValueError("h and out must be [B, S, hidden] with a contiguous last axis")
    if h.dtype != out.dtype or h.shape[0] != out.shape[0] or h.shape[2] != out.shape[2]:
        raise ValueError("h and out must agree in dtype, batch and hidden size")
    s = spans._c()
    st = _lib.speechkv_pool_hidden(h.data_ptr(), h.stride(0), h.stride(1), h.shape[0], h.shape[1],
                                   h.shape[2], _dtype_code(h.dtype), ctypes.byref(s), w,
                                   _ptr(gate_u), out.data_ptr(), out.stride(0), out.stride(1),
                                   out.shape[1], _ptr(out_len), _stream(stream))
    _check(st, "speechkv_pool_hidden")


def speechkv_decode_attn(q: torch.Tensor, cache: PagedKV, cache_len: torch.Tensor,
                         max_cache_len: int, out: torch.Tensor,
                         k_new: Optional[torch.Tensor] = None,
                         v_new: Optional[torch.Tensor] = None, scale: Optional[float] = None,
                         num_splits: int = 0, workspace: Optional[torch.Tensor] = None,
                         stream=None) -> None:
    """q, out: [B, Hq, D] contiguous; k_new, v_new: [B, Hkv, D] or None."""
    for x in (q, out, cache_len) + tuple(t for t in (k_new, v_new) if t is not None):
        if not x.is_contiguous():
            raise ValueError("decode tensors must be contiguous")
    B, Hq, D = q.shape
    if scale is None:
        scale = D ** -0.5
    c = cache._c()
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = _lib.speechkv_decode_attn(q.data_ptr(), B, Hq, ctypes.byref(c), cache_len.data_ptr(),
                                   max_cache_len, _ptr(k_new), _ptr(v_new), scale, num_splits,
                                   out.data_ptr(), _ptr(workspace), ws_bytes, _stream(stream))
    _check(st, "speechkv_decode_attn")


def speechkv_decode_attn_noalloc(q: torch.Tensor, cache: PagedKV, cache_len: torch.Tensor,
                                 max_cache_len: int, out: torch.Tensor,
                                 k_new: Optional[torch.Tensor] = None,
                                 v_new: Optional[torch.Tensor] = None,
                                 scale: Optional[float] = None, num_splits: int = 0,
                                 stream=None) -> None:
    """speechkv_decode_attn without a workspace: split partials go to the
    library's static per-GPU scratch.  Calls that overlap on one GPU race."""
    for x in (q, out, cache_len) + tuple(t for t in (k_new, v_new) if t is not None):
        if not x.is_contiguous():
            raise ValueError("decode tensors must be contiguous")
    B, Hq, D = q.shape
    if scale is None:
        scale = D ** -0.5
    c = cache._c()
    st = _lib.speechkv_decode_attn_noalloc(q.data_ptr(), B, Hq, ctypes.byref(c),
                                           cache_len.data_ptr(), max_cache_len, _ptr(k_new),
                                           _ptr(v_new), scale, num_splits, out.data_ptr(),
                                           _stream(stream))
    _check(st, "speechkv_decode_attn_noalloc")


def speechkv_prefill_attn(q: torch.Tensor, cache: PagedKV, spans: Spans, w: int, layer: int,
                          l0: int, out: torch.Tensor, mask_mode: int = MASK_WINDOW_END,
                          scale: Optional[float] = None, lse: Optional[torch.Tensor] = None,
                          stream=None) -> None:
    """q, out: [B, q_len, Hq, D] contiguous; lse: [B, Hq, q_len] fp32 or None."""
    for x in (q, out) + ((lse,) if lse is not None else ()):
        if not x.is_contiguous():
            raise ValueError("prefill tensors must be contiguous")
    B, q_len, Hq, D = q.shape
    if scale is None:
        scale = D ** -0.5
    c = cache._c()
    s = spans._c()
    st = _lib.speechkv_prefill_attn(q.data_ptr(), B, Hq, q_len, ctypes.byref(c), ctypes.byref(s),
                                    w, layer, l0, mask_mode, scale, out.data_ptr(), _ptr(lse),
                                    _stream(stream))
    _check(st, "speechkv_prefill_attn")


def speechkv_pool_prefill_attn(q: torch.Tensor, k_raw: torch.Tensor, v_raw: torch.Tensor,
                               spans: Spans, w: int, gate_u: Optional[torch.Tensor], layer: int,
                               l0: int, cache: PagedKV, out: torch.Tensor,
                               cache_len_out: Optional[torch.Tensor] = None,
                               mask_mode: int = MASK_WINDOW_END, scale: Optional[float] = None,
                               lse: Optional[torch.Tensor] = None, stream=None) -> None:
    """Pooling and prefill attention in one launch.  q, out: [B, q_len, Hq, D]
    contiguous; k_raw, v_raw: [B, S_raw, Hkv, D] views with a contiguous last
    axis; lse: [B, Hq, q_len] fp32 or None."""
    for x in (q, out) + ((lse,) if lse is not None else ()):
        if not x.is_contiguous():
            raise ValueError("prefill tensors must be contiguous")
    if k_raw.shape != v_raw.shape or k_raw.stride() != v_raw.stride():
        raise ValueError("k_raw and v_raw must have one shape and one stride")
    if k_raw.dim() != 4 or k_raw.stride(3) != 1:
        raise ValueError("raw K/V must be [B, S, Hkv, D] with a contiguous last axis")
    B, q_len, Hq, D = q.shape
    if scale is None:
        scale = D ** -0.5
    sb, ss, sh, _ = k_raw.stride()
    c = cache._c()
    s = spans._c()
    st = _lib.speechkv_pool_prefill_attn(q.data_ptr(), B, Hq, q_len, k_raw.data_ptr(),
                                         v_raw.data_ptr(), sb, ss, sh, k_raw.shape[1],
                                         ctypes.byref(s), w, _ptr(gate_u), layer, l0,
                                         ctypes.byref(c), _ptr(cache_len_out), mask_mode, scale,
                                         out.data_ptr(), _ptr(lse), _stream(stream))
    _check(st, "speechkv_pool_prefill_attn")


def speechkv_prefill_attn_bwd_workspace_bytes(batch: int, num_q_heads: int, q_len: int) -> int:
    return int(_lib.speechkv_prefill_attn_bwd_workspace_bytes(batch, num_q_heads, q_len))


def speechkv_prefill_attn_bwd(q: torch.Tensor, cache: PagedKV, spans: Spans, w: int, layer: int,
                              l0: int, out: torch.Tensor, lse: torch.Tensor, dout: torch.Tensor,
                              dq: torch.Tensor, dk_hat: torch.Tensor, dv_hat: torch.Tensor,
                              workspace: torch.Tensor, mask_mode: int = MASK_WINDOW_END,
                              scale: Optional[float] = None, stream=None) -> None:
    """q, out, dout, dq: [B, q_len, Hq, D]; lse: [B, Hq, q_len] fp32;
    dk_hat, dv_hat: [B, hat_capacity, Hkv, D] fp32; workspace: device bytes."""
    _prefill_attn_bwd(_lib.speechkv_prefill_attn_bwd, "speechkv_prefill_attn_bwd", q, cache,
                      spans, w, layer, l0, out, lse, dout, dq, dk_hat, dv_hat, workspace,
                      mask_mode, scale, stream)


def speechkv_prefill_attn_bwd_segments(q: torch.Tensor, cache: PagedKV, segs: Segments, w: int,
                                       layer: int, l0: int, out: torch.Tensor, lse: torch.Tensor,
                                       dout: torch.Tensor, dq: torch.Tensor, dk_hat: torch.Tensor,
                                       dv_hat: torch.Tensor, workspace: torch.Tensor,
                                       mask_mode: int = MASK_WINDOW_END,
                                       scale: Optional[float] = None, stream=None) -> None:
    """speechkv_prefill_attn_bwd for sequences given as segment tables."""
    _prefill_attn_bwd(_lib.speechkv_prefill_attn_bwd_segments, "speechkv_prefill_attn_bwd_segments",
                      q, cache, segs, w, layer, l0, out, lse, dout, dq, dk_hat, dv_hat, workspace,
                      mask_mode, scale, stream)


def _prefill_attn_bwd(fn, name, q, cache, spans, w, layer, l0, out, lse, dout, dq, dk_hat, dv_hat,
                      workspace, mask_mode, scale, stream):
    for x in (q, out, dout, dq, lse, dk_hat, dv_hat, workspace):
        if not x.is_contiguous():
            raise ValueError("backward tensors must be contiguous")
    if dk_hat.dtype != torch.float32 or dv_hat.dtype != torch.float32 or lse.dtype != torch.float32:
        raise ValueError("lse, dk_hat and dv_hat are fp32")
    if dk_hat.shape != dv_hat.shape or dk_hat.dim() != 4:
        raise ValueError("dk_hat and dv_hat must share one [B, capacity, Hkv, D] shape")
    B, q_len, Hq, D = q.shape
    if scale is None:
        scale = D ** -0.5
    c = cache._c()
    s = spans._c()
    st = fn(q.data_ptr(), B, Hq, q_len, ctypes.byref(c), ctypes.byref(s), w, layer, l0, mask_mode,
            scale, out.data_ptr(), lse.data_ptr(), dout.data_ptr(), dq.data_ptr(),
            dk_hat.data_ptr(), dv_hat.data_ptr(), dk_hat.shape[1], workspace.data_ptr(),
            workspace.numel() * workspace.element_size(), _stream(stream))
    _check(st, name)


def speechkv_pool_kv_bwd_workspace_bytes(batch: int, max_total_len: int, num_kv_heads: int,
                                         head_dim: int) -> int:
    return int(_lib.speechkv_pool_kv_bwd_workspace_bytes(batch, max_total_len, num_kv_heads,
                                                         head_dim))


def speechkv_pool_kv_bwd(k_raw: torch.Tensor, v_raw: torch.Tensor, spans: Spans, w: int,
                         gate_u: Optional[torch.Tensor], layer: int, l0: int,
                         dk_hat: torch.Tensor, dv_hat: torch.Tensor, dk_raw: torch.Tensor,
                         dv_raw: torch.Tensor, du: Optional[torch.Tensor] = None,
                         workspace: Optional[torch.Tensor] = None, stream=None) -> None:
    """k_raw, v_raw, dk_raw, dv_raw: [B, S_raw, Hkv, D] with one stride and a
    contiguous last axis; dk_hat, dv_hat: [B, capacity, Hkv, D] fp32; du:
    [Hkv, D] fp32 or None."""
    _pool_kv_bwd(_lib.speechkv_pool_kv_bwd, "speechkv_pool_kv_bwd", k_raw, v_raw, spans, w, gate_u,
                 layer, l0, dk_hat, dv_hat, dk_raw, dv_raw, du, workspace, stream)


def speechkv_pool_kv_bwd_segments(k_raw: torch.Tensor, v_raw: torch.Tensor, segs: Segments,
                                  w: int, gate_u: Optional[torch.Tensor], layer: int, l0: int,
                                  dk_hat: torch.Tensor, dv_hat: torch.Tensor,
                                  dk_raw: torch.Tensor, dv_raw: torch.Tensor,
                                  du: Optional[torch.Tensor] = None,
                                  workspace: Optional[torch.Tensor] = None, stream=None) -> None:
    """speechkv_pool_kv_bwd for sequences given as segment tables."""
    _pool_kv_bwd(_lib.speechkv_pool_kv_bwd_segments, "speechkv_pool_kv_bwd_segments", k_raw, v_raw,
                 segs, w, gate_u, layer, l0, dk_hat, dv_hat, dk_raw, dv_raw, du, workspace, stream)


def _pool_kv_bwd(fn, name, k_raw, v_raw, spans, w, gate_u, layer, l0, dk_hat, dv_hat, dk_raw,
                 dv_raw, du, workspace, stream):
    for x in (v_raw, dk_raw, dv_raw):
        if x.shape != k_raw.shape or x.stride() != k_raw.stride() or x.dtype != k_raw.dtype:
            raise ValueError("k_raw, v_raw, dk_raw and dv_raw must share shape, stride and dtype")
    if k_raw.dim() != 4 or k_raw.stride(3) != 1:
        raise ValueError("raw K/V must be [B, S, Hkv, D] with a contiguous last axis")
    for x in (dk_hat, dv_hat) + ((du,) if du is not None else ()):
        if x.dtype != torch.float32 or not x.is_contiguous():
            raise ValueError("dk_hat, dv_hat and du are contiguous fp32")
    B, S, H, D = k_raw.shape
    sb, ss, sh, _ = k_raw.stride()
    s = spans._c()
    ws = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = fn(k_raw.data_ptr(), v_raw.data_ptr(), sb, ss, sh, B, S, H, D, _dtype_code(k_raw.dtype),
            ctypes.byref(s), w, _ptr(gate_u), layer, l0, dk_hat.data_ptr(), dv_hat.data_ptr(),
            dk_hat.shape[1], dk_raw.data_ptr(), dv_raw.data_ptr(), _ptr(du), _ptr(workspace), ws,
            _stream(stream))
    _check(st, name)


def speechkv_compressed_len(prefix_len: int, speech_len: int, suffix_len: int, w: int,
                            layer: int, l0: int) -> int:
    return int(_lib.speechkv_compressed_len(prefix_len, speech_len, suffix_len, w, layer, l0))


def speechkv_decode_num_splits(batch: int, num_kv_heads: int, max_cache_len: int) -> int:
    return int(_lib.speechkv_decode_num_splits(batch, num_kv_heads, max_cache_len))


def speechkv_decode_workspace_bytes(batch: int, num_q_heads: int, num_kv_heads: int,
                                    head_dim: int, max_cache_len: int, num_splits: int = 0) -> int:
    return int(_lib.speechkv_decode_workspace_bytes(batch, num_q_heads, num_kv_heads, head_dim,
                                                    max_cache_len, num_splits))


def speechkv_status_string(status: int) -> str:
    return _lib.speechkv_status_string(status).decode()


def speechkv_version() -> str:
    return _lib.speechkv_version().decode()
