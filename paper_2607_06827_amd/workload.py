"""Device-resident SpeechKV jobs: every layer's inputs, caches and outputs.

A job is one batch of sequences through the whole hot path, layer by layer:
  prefill   pool the raw K/V of each layer into its paged cache (identity
            below l0), then attend with the full-resolution queries;
  decode    for each step and each layer, store the new token's K/V and
            attend over the cache (one query per sequence).
This module only allocates device memory, fills it from `inputs` and issues
the library calls in order; all computation happens in libspeechkv's kernels.
"""
from __future__ import annotations

from typing import List, Optional, Sequence

import torch

from . import inputs
from .speechkv import (PagedKV, Segments, Spans, speechkv_compressed_len,
                       speechkv_compressed_len_segments, speechkv_decode_attn,
                       speechkv_decode_num_splits, speechkv_decode_workspace_bytes,
                       speechkv_pool_hidden, speechkv_pool_kv, speechkv_pool_kv_bwd,
                       speechkv_pool_kv_bwd_workspace_bytes, speechkv_pool_kv_segments,
                       speechkv_pool_prefill_attn, speechkv_prefill_attn,
                       speechkv_prefill_attn_bwd, speechkv_prefill_attn_bwd_workspace_bytes,
                       speechkv_prefill_attn_segments)


def visible_pairs(P: int, T: int, N: int, w: int) -> int:
    """Sum over the P + T + N full-resolution rows of the number of compressed
    keys each row may attend to, under the causal mask over compressed
    positions (Sec. III-B, Eq. 5) with a pooled window visible from its last
    frame: prefix row p sees p + 1 keys, speech frame t sees the prefix and the
    windows that end at or before it, text row m after the speech sees all
    of those plus the text up to itself.  Used to count algorithmic FLOPs."""
    nW = -(-T // w)
    total = P * (P + 1) // 2
    total += sum((P + nW) if t == T - 1 else (P + (t + 1) // w) for t in range(T))
    total += sum(P + nW + m + 1 for m in range(N))
    return total


class Job:
    """All buffers of one workload on one device.

    layers        which layer indices to build (default: all); layer ids keep
                  their meaning with respect to l0.
    l0            first compressed layer (default wl.l0; num_layers or more
                  means no compression, the full-KV reference run).
    with_prefill  allocate prefill queries/outputs and run prefill attention.
    keep_decode   keep every decode output ([layers, steps, B, Hq, D]) rather
                  than reusing one buffer.
    share_inputs  another Job whose input tensors this one reuses.
    """

    def __init__(self, wl: inputs.Workload, device="cuda", layers: Optional[Sequence[int]] = None,
                 l0: Optional[int] = None, with_prefill: bool = True, keep_decode: bool = False,
                 share_inputs: Optional["Job"] = None, shuffle_pages: bool = True,
                 num_splits: int = 0):
        self.wl = wl
        self.device = torch.device(device)
        self.layers: List[int] = list(range(wl.num_layers)) if layers is None else list(layers)
        self.l0 = wl.l0 if l0 is None else l0
        self.with_prefill = with_prefill
        self.num_splits = num_splits
        B, Hq, Hkv, D = wl.batch, wl.num_q_heads, wl.num_kv_heads, wl.head_dim
        S = wl.prefill_len
        dev = self.device
        self.scale = D ** -0.5

        ints = lambda v: torch.full((B,), v, dtype=torch.int32, device=dev)
        self.spans = Spans(ints(wl.prefix_len), ints(wl.speech_len), ints(wl.suffix_len),
                           wl.speech_len, S)

        src = share_inputs
        self.k_raw, self.v_raw, self.gate, self.q_prefill = [], [], [], []
        self.q_dec, self.k_new, self.v_new = [], [], []
        for i, l in enumerate(self.layers):
            if src is not None:
                j = src.layers.index(l)
                self.k_raw.append(src.k_raw[j]); self.v_raw.append(src.v_raw[j])
                self.gate.append(src.gate[j])
                self.q_prefill.append(src.q_prefill[j] if with_prefill else None)
                self.q_dec.append(src.q_dec[j]); self.k_new.append(src.k_new[j])
                self.v_new.append(src.v_new[j])
                continue
            k, v = inputs.raw_kv(wl, l, device=dev)
            self.k_raw.append(k); self.v_raw.append(v)
            self.gate.append(inputs.gate(wl, l, device=dev))
            self.q_prefill.append(inputs.prefill_q(wl, l, device=dev) if with_prefill else None)
            steps = range(wl.decode_steps)
            self.q_dec.append(torch.stack([inputs.decode_q(wl, l, s, device=dev) for s in steps])
                              if wl.decode_steps else None)
            kn = [inputs.decode_kv_new(wl, l, s, device=dev) for s in steps]
            self.k_new.append(torch.stack([x[0] for x in kn]) if kn else None)
            self.v_new.append(torch.stack([x[1] for x in kn]) if kn else None)

        # caches sized for prefill plus every decoded token
        self.prefill_clen = [speechkv_compressed_len(wl.prefix_len, wl.speech_len, wl.suffix_len,
                                                     wl.window(l), l, self.l0) for l in self.layers]
        self.caches: List[PagedKV] = []
        self.cache_len_out = []
        for i, l in enumerate(self.layers):
            cap = self.prefill_clen[i] + wl.decode_steps
            pages = max(1, -(-cap // wl.page_size))
            table, total = inputs.block_table(B, pages, wl.seed, layer=l, shuffle=shuffle_pages)
            kp = torch.empty(total, Hkv, wl.page_size, D, dtype=wl.torch_dtype, device=dev)
            vp = torch.empty_like(kp)
            self.caches.append(PagedKV(kp, vp, table.to(dev)))
            self.cache_len_out.append(torch.zeros(B, dtype=torch.int32, device=dev))

        # decode cache lengths per (layer, step): prefill length + tokens so far
        self.dec_len = [torch.stack([ints(self.prefill_clen[i] + s + 1)
                                     for s in range(wl.decode_steps)]) if wl.decode_steps else None
                        for i in range(len(self.layers))]
        max_len = max(self.prefill_clen) + wl.decode_steps
        splits = [num_splits or speechkv_decode_num_splits(B, Hkv, c + wl.decode_steps)
                  for c in self.prefill_clen]
        ws = max(speechkv_decode_workspace_bytes(B, Hq, Hkv, D, max_len, s) for s in splits)
        self.workspace = torch.empty(max(ws, 16) // 4 + 4, dtype=torch.float32, device=dev)

        self.prefill_out = (torch.empty(B, S, Hq, D, dtype=wl.torch_dtype, device=dev)
                            if with_prefill else None)
        n_out = len(self.layers) * wl.decode_steps if keep_decode else 1
        self.keep_decode = keep_decode
        self.decode_out = torch.empty(max(n_out, 1), B, Hq, D, dtype=wl.torch_dtype, device=dev)

    # ------------------------------------------------------------------ steps
    def run_prefill(self, stream=None, layers: Optional[Sequence[int]] = None):
        wl = self.wl
        for i, l in enumerate(self.layers):
            if layers is not None and l not in layers:
                continue
            speechkv_pool_kv(self.k_raw[i], self.v_raw[i], self.spans, wl.window(l), self.gate[i],
                             l, self.l0, self.caches[i], self.cache_len_out[i], stream=stream)
            if self.with_prefill:
                speechkv_prefill_attn(self.q_prefill[i], self.caches[i], self.spans, wl.window(l), l,
                                      self.l0, self.prefill_out, scale=self.scale, stream=stream)

    def run_prefill_fused(self, stream=None, layers: Optional[Sequence[int]] = None):
        """The prefill of every layer as one launch each: the pooling runs on
        the fly inside the attention (speechkv_pool_prefill_attn), writing the
        same caches, lengths and outputs as run_prefill."""
        wl = self.wl
        for i, l in enumerate(self.layers):
            if layers is not None and l not in layers:
                continue
            speechkv_pool_prefill_attn(self.q_prefill[i], self.k_raw[i], self.v_raw[i], self.spans,
                                       wl.window(l), self.gate[i], l, self.l0, self.caches[i],
                                       self.prefill_out, cache_len_out=self.cache_len_out[i],
                                       scale=self.scale, stream=stream)

    def run_pool(self, stream=None):
        """Pooling of every layer (writes the caches)."""
        wl = self.wl
        for i, l in enumerate(self.layers):
            speechkv_pool_kv(self.k_raw[i], self.v_raw[i], self.spans, wl.window(l), self.gate[i],
                             l, self.l0, self.caches[i], self.cache_len_out[i], stream=stream)

    def run_prefill_attn(self, stream=None):
        """Prefill attention of every layer over caches already pooled."""
        wl = self.wl
        for i, l in enumerate(self.layers):
            speechkv_prefill_attn(self.q_prefill[i], self.caches[i], self.spans, wl.window(l), l,
                                  self.l0, self.prefill_out, scale=self.scale, stream=stream)

    def decode_out_at(self, i: int, step: int) -> torch.Tensor:
        return self.decode_out[i * self.wl.decode_steps + step if self.keep_decode else 0]

    def run_decode_step(self, step: int, stream=None):
        for i in range(len(self.layers)):
            self.decode_layer(i, step, stream)

    def decode_layer(self, i: int, step: int, stream=None):
        wl = self.wl
        speechkv_decode_attn(self.q_dec[i][step], self.caches[i], self.dec_len[i][step],
                             self.prefill_clen[i] + step + 1, self.decode_out_at(i, step),
                             k_new=self.k_new[i][step], v_new=self.v_new[i][step],
                             scale=self.scale, num_splits=self.num_splits,
                             workspace=self.workspace, stream=stream)

    def run(self, stream=None):
        """The whole job: prefill of every layer, then every decode step."""
        self.run_prefill(stream)
        for s in range(self.wl.decode_steps):
            self.run_decode_step(s, stream)

    # ------------------------------------------------------------- accounting
    def decode_bytes_layer(self, i: int, step: int) -> int:
        """Algorithmic HBM bytes of one decode launch (layer index i): every
        cached K and V row read once, q read, out written, and the new token's
        K/V read and written once."""
        wl = self.wl
        e = 2 if wl.dtype == "bf16" else 4
        row = wl.num_kv_heads * wl.head_dim * e
        L = self.prefill_clen[i] + step + 1
        return wl.batch * (2 * row * (L - 1) + 2 * wl.num_q_heads * wl.head_dim * e + 4 * row)

    def decode_bytes(self, step: int) -> int:
        """Algorithmic HBM bytes of one decode step over all layers."""
        return sum(self.decode_bytes_layer(i, step) for i in range(len(self.layers)))

    def pool_bytes_layer(self, i: int) -> int:
        """Algorithmic HBM bytes of one pooling launch (layer index i): every
        raw K and V row read once, every cache row written once (pooled
        windows and copied text alike), the gate vectors read."""
        wl = self.wl
        e = 2 if wl.dtype == "bf16" else 4
        row = wl.num_kv_heads * wl.head_dim * e
        return wl.batch * 2 * row * (wl.prefill_len + self.prefill_clen[i]) + row

    def prefill_visible_pairs(self, i: int) -> int:
        """(row, visible key) pairs of one sequence's prefill at layer index i."""
        wl = self.wl
        w = wl.window(self.layers[i]) if self.layers[i] >= self.l0 else 1
        return visible_pairs(wl.prefix_len, wl.speech_len, wl.suffix_len, w)

    def prefill_bytes_layer(self, i: int) -> int:
        """Algorithmic HBM bytes of one prefill attention launch: Q read and O
        written once, the compressed K and V read once."""
        wl = self.wl
        e = 2 if wl.dtype == "bf16" else 4
        q = wl.batch * wl.prefill_len * wl.num_q_heads * wl.head_dim * e
        kv = wl.batch * self.prefill_clen[i] * wl.num_kv_heads * wl.head_dim * e
        return 2 * q + 2 * kv

    def prefill_flops_layer(self, i: int) -> int:
        """Algorithmic FLOPs of one prefill attention launch: q.k and p.v for
        every (row, visible key) pair of every query head, 2 FLOPs per
        multiply-add (the masked-out pairs are not counted)."""
        wl = self.wl
        return 4 * wl.batch * wl.num_q_heads * wl.head_dim * self.prefill_visible_pairs(i)


class HiddenPoolJob:
    """HS Compression (Sec. IV-A, method (4)) of one workload: the hidden state
    entering layer l0 ([B, P + T + N, hidden], hidden = q_heads x head_dim,
    2048 for Qwen3-1.7B) pooled with the Eq. 4 window softmax into the
    shortened sequence every later layer runs on."""

    def __init__(self, wl: inputs.Workload, device="cuda"):
        self.wl = wl
        self.hidden = wl.num_q_heads * wl.head_dim
        B, S = wl.batch, wl.prefill_len
        self.h = inputs.normal((B, S, self.hidden), wl.seed * 100 + 71, device=device,
                               dtype=wl.torch_dtype)
        self.gate = inputs.normal((self.hidden,), wl.seed * 100 + 72, device=device,
                                  scale=self.hidden ** -0.5)
        self.out_rows = speechkv_compressed_len(wl.prefix_len, wl.speech_len, wl.suffix_len,
                                                wl.window(wl.l0), 1, 0)
        self.out = torch.empty(B, self.out_rows, self.hidden, dtype=wl.torch_dtype,
                               device=device)
        self.out_len = torch.empty(B, dtype=torch.int32, device=device)
        i32 = lambda v: torch.full((B,), v, dtype=torch.int32, device=device)
        self.spans = Spans(i32(wl.prefix_len), i32(wl.speech_len), i32(wl.suffix_len),
                           wl.speech_len, S)

    def run(self, stream=None):
        speechkv_pool_hidden(self.h, self.spans, self.wl.window(self.wl.l0), self.gate, self.out,
                             self.out_len, stream)

    def bytes(self) -> int:
        """Algorithmic HBM bytes of one launch: every input row read once,
        every output row written once, the gate read."""
        e = self.h.element_size()
        return self.wl.batch * self.hidden * e * (self.wl.prefill_len + self.out_rows) \
            + self.hidden * 4


class TrainJob:
    """One training-mode layer of a workload (Sec. III-C: the pooling runs in
    the forward pass and is optimised jointly): the forward (pool, then
    attention with its log-sum-exp) and the backward from a seeded output
    gradient (attention backward, then pooling backward down to the raw K/V
    and the gate).  Layer index `layer` of the workload, its first layer by
    default."""

    def __init__(self, wl: inputs.Workload, layer: Optional[int] = None, device="cuda"):
        layer = wl.l0 if layer is None else layer
        self.fwd = Job(wl, device=device, layers=[layer])
        self.wl = wl
        self.layer = layer
        self.w = wl.window(layer)
        f = self.fwd
        B, S, Hq, Hkv, D = wl.batch, wl.prefill_len, wl.num_q_heads, wl.num_kv_heads, wl.head_dim
        dev = f.device
        self.out = torch.empty(B, S, Hq, D, dtype=wl.torch_dtype, device=dev)
        self.lse = torch.empty(B, Hq, S, dtype=torch.float32, device=dev)
        self.dout = inputs.normal((B, S, Hq, D), wl.seed * 100 + 81, device=dev, dtype=wl.torch_dtype)
        self.clen = f.prefill_clen[0]
        self.dq = torch.empty_like(self.out)
        self.dk_hat = torch.empty(B, self.clen, Hkv, D, dtype=torch.float32, device=dev)
        self.dv_hat = torch.empty_like(self.dk_hat)
        self.dk_raw = torch.empty_like(f.k_raw[0])
        self.dv_raw = torch.empty_like(f.v_raw[0])
        self.du = torch.empty(Hkv, D, dtype=torch.float32, device=dev)
        n = max(speechkv_prefill_attn_bwd_workspace_bytes(B, Hq, S),
                speechkv_pool_kv_bwd_workspace_bytes(B, S, Hkv, D))
        self.workspace = torch.empty(n, dtype=torch.uint8, device=dev)

    def run_forward(self, stream=None):
        f, wl = self.fwd, self.wl
        speechkv_pool_kv(f.k_raw[0], f.v_raw[0], f.spans, self.w, f.gate[0], self.layer, f.l0,
                         f.caches[0], stream=stream)
        speechkv_prefill_attn(f.q_prefill[0], f.caches[0], f.spans, self.w, self.layer, f.l0,
                              self.out, scale=f.scale, lse=self.lse, stream=stream)

    def run_attn_bwd(self, stream=None):
        f, wl = self.fwd, self.wl
        speechkv_prefill_attn_bwd(f.q_prefill[0], f.caches[0], f.spans, self.w, self.layer, f.l0,
                                  self.out, self.lse, self.dout, self.dq, self.dk_hat, self.dv_hat,
                                  self.workspace, scale=f.scale, stream=stream)

    def run_pool_bwd(self, stream=None):
        f, wl = self.fwd, self.wl
        speechkv_pool_kv_bwd(f.k_raw[0], f.v_raw[0], f.spans, self.w, f.gate[0], self.layer, f.l0,
                             self.dk_hat, self.dv_hat, self.dk_raw, self.dv_raw, self.du,
                             self.workspace, stream=stream)

    def run_backward(self, stream=None):
        self.run_attn_bwd(stream)
        self.run_pool_bwd(stream)

    def attn_bwd_flops(self) -> int:
        """Algorithmic FLOPs of the attention backward: the four gradient
        products dP = dO V^T, dV^ = P^T dO, dK^ = dZ^T Q, dQ = dZ K^ over
        every (row, visible key) pair of every query head, 2 FLOPs per
        multiply-add (recomputing S is not counted)."""
        return 8 * self.wl.batch * self.wl.num_q_heads * self.wl.head_dim * \
            self.fwd.prefill_visible_pairs(0)

    def attn_bwd_bytes(self) -> int:
        """Algorithmic HBM bytes of the attention backward: Q, O, dO read and
        dQ written once, K^ and V^ read once, dK^ and dV^ (fp32) written once,
        LSE read once."""
        wl = self.wl
        e = 2 if wl.dtype == "bf16" else 4
        q = wl.batch * wl.prefill_len * wl.num_q_heads * wl.head_dim
        kv = wl.batch * self.clen * wl.num_kv_heads * wl.head_dim
        return 4 * q * e + 2 * kv * e + 2 * kv * 4 + wl.batch * wl.num_q_heads * wl.prefill_len * 4

    def pool_bwd_bytes(self) -> int:
        """Algorithmic HBM bytes of the pooling backward: raw K and V read once,
        their gradients written once, dK^ and dV^ (fp32) read once."""
        wl = self.wl
        e = 2 if wl.dtype == "bf16" else 4
        row = wl.num_kv_heads * wl.head_dim
        return wl.batch * (4 * wl.prefill_len * row * e + 2 * self.clen * row * 4)


# A multi-turn batch: three speech turns (30 s, 20 s and 40 s of 80 ms frames)
# between text prompts, 1261 rows per sequence, 418 after w = 4 pooling.
MULTI_TURN = [(32, 375), (24, 250), (16, 500), (64, 0)]


class SegmentJob:
    """One layer of a batch of sequences with several speech runs each
    (segment tables): pooling into a paged cache, then prefill attention.
    With one_run=True the same number of text rows and frames per sequence
    is laid out as a single run (all text before the speech but the last
    prompt), for comparison."""

    def __init__(self, segs, batch=16, q_heads=16, kv_heads=8, head_dim=128, w=4, seed=6,
                 page_size=16, one_run=False, device="cuda"):
        self.segs = [list(segs)] * batch
        self.w = w
        self.one_run = one_run
        rows = sum(t + s for t, s in segs)
        self.rows = rows
        self.clen = speechkv_compressed_len_segments(segs, w, 1, 0)
        dt = torch.bfloat16
        B, dev = batch, torch.device(device)
        self.k_raw = inputs.normal((B, rows, kv_heads, head_dim), seed * 100 + 1, device=dev, dtype=dt)
        self.v_raw = inputs.normal((B, rows, kv_heads, head_dim), seed * 100 + 2, device=dev, dtype=dt)
        self.gate = inputs.normal((kv_heads, head_dim), seed * 100 + 3, device=dev,
                                  scale=head_dim ** -0.5)
        self.q = inputs.normal((B, rows, q_heads, head_dim), seed * 100 + 4, device=dev, dtype=dt)
        self.out = torch.empty_like(self.q)
        self.scale = head_dim ** -0.5
        if one_run:
            P = sum(t for t, _ in segs[:-1])
            T = sum(s for _, s in segs)
            N = segs[-1][0]
            i32 = lambda v: torch.full((B,), v, dtype=torch.int32, device=dev)
            self.spans = Spans(i32(P), i32(T), i32(N), T, rows)
            self.clen = speechkv_compressed_len(P, T, N, w, 1, 0)
        else:
            self.table = Segments.from_lists(self.segs, device=dev)
        pages = -(-self.clen // page_size)
        table, total = inputs.block_table(B, pages, seed)
        kp = torch.empty(total, kv_heads, page_size, head_dim, dtype=dt, device=dev)
        self.cache = PagedKV(kp, torch.empty_like(kp), table.to(dev))

    def run(self, stream=None):
        if self.one_run:
            speechkv_pool_kv(self.k_raw, self.v_raw, self.spans, self.w, self.gate, 1, 0,
                             self.cache, stream=stream)
            speechkv_prefill_attn(self.q, self.cache, self.spans, self.w, 1, 0, self.out,
                                  scale=self.scale, stream=stream)
        else:
            speechkv_pool_kv_segments(self.k_raw, self.v_raw, self.table, self.w, self.gate, 1, 0,
                                      self.cache, stream=stream)
            speechkv_prefill_attn_segments(self.q, self.cache, self.table, self.w, 1, 0, self.out,
                                           scale=self.scale, stream=stream)
