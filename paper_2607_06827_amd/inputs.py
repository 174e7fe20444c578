"""Seeded synthetic inputs shaped like the paper's workloads.

This module only draws random numbers and arranges them; it holds none of
SpeechKV's arithmetic (no pooling, no attention, no window or cache-length
formula).  Both the GPU path and the fp64 oracle are fed from it, which is the
only thing the two share.

Workload shapes (arXiv 2607.06827):
  - speech frames every 80 ms (Sec. IV-A), so 30 s of audio is 375 frames,
    60 s is 750 and 10 minutes is 7500;
  - the backbone is Qwen3-1.7B with 28 decoder layers (Sec. IV-A); its
    attention uses 16 query heads, 8 KV heads and head_dim 128;
  - the speech representations of deeper layers are locally redundant
    (Sec. V-B, local similarity), which the generator imitates with a
    stationary AR(1) process along time per channel: x_0 ~ N(0, 1),
    x_t = rho * x_{t-1} + sqrt(1 - rho^2) * e_t, so adjacent frames have
    correlation rho and every frame is N(0, 1);
  - text keys and values are i.i.d. N(0, 1); queries are N(0, 1) and the
    attention scale 1/sqrt(head_dim) is applied once, by the kernels;
  - the gate vector of each layer and KV head is N(0, sigma^2) with
    sigma = 1/sqrt(head_dim), so gate logits over N(0, 1) keys have unit
    standard deviation.
No dataset, transcript or trained weight stands behind any of these numbers:
they replace OpenASR, the in-house test sets and the trained model, none of
which is available.

Every tensor is drawn in fp32 from its own torch.Generator, seeded from
(workload seed, layer, stream, step) through numpy's SeedSequence, then rounded
once (round-to-nearest-even) to the workload's element type.  The same call
gives the same tensor on the same device type; CPU and GPU generators differ,
so a test draws on one device and copies to the other.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional, Sequence, Tuple

import numpy as np
import torch

# stream ids of the independent random streams
_S_K_TEXT, _S_V_TEXT, _S_K_SPEECH, _S_V_SPEECH = 0, 1, 2, 3
_S_GATE, _S_Q_PREFILL, _S_Q_DECODE, _S_K_NEW, _S_V_NEW, _S_PAGES = 5, 6, 7, 8, 9, 10


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape of one synthetic workload (all layers share it)."""

    name: str
    batch: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    prefix_len: int      # text before the speech
    speech_len: int      # speech frames
    suffix_len: int      # text after the speech present at prefill
    decode_steps: int    # tokens decoded after prefill
    w: int               # window size R
    l0: int              # first compressed layer (0-indexed)
    num_layers: int
    rho: float           # AR(1) coefficient of the speech frames
    dtype: str           # "bf16" or "f32"
    seed: int
    page_size: int = 16
    # per-layer window sizes (one per layer, used from l0 on): the adaptive
    # compression ratio across layers that the paper leaves to future work
    # (Sec. VI); None gives every compressed layer the window w
    w_layers: Optional[Tuple[int, ...]] = None

    def __post_init__(self):
        if self.w_layers is not None:
            if len(self.w_layers) != self.num_layers or min(self.w_layers) < 1:
                raise ValueError("w_layers needs one window size >= 1 per layer")

    def window(self, layer: int) -> int:
        """Window size R of a layer (layers below l0 keep every frame
        whatever this returns)."""
        return self.w_layers[layer] if self.w_layers is not None else self.w

    @property
    def prefill_len(self) -> int:
        return self.prefix_len + self.speech_len + self.suffix_len

    @property
    def torch_dtype(self) -> torch.dtype:
        return torch.bfloat16 if self.dtype == "bf16" else torch.float32

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


def _wl(name, **kw):
    return Workload(name=name, **kw)


# The five workloads, named by what they are.
TINY_F32 = _wl("tiny-fp32-b1-h4kv2-d64-p8-t60-w4", batch=1, num_q_heads=4,
               num_kv_heads=2, head_dim=64, prefix_len=8, speech_len=60,
               suffix_len=0, decode_steps=16, w=4, l0=0, num_layers=1, rho=0.9,
               dtype="f32", seed=0)
LAYER_30S = _wl("qwen3-1.7b-layer-30s-b32", batch=32, num_q_heads=16,
                num_kv_heads=8, head_dim=128, prefix_len=32, speech_len=375,
                suffix_len=0, decode_steps=64, w=4, l0=0, num_layers=1, rho=0.9,
                dtype="bf16", seed=1)
STACK_60S = _wl("qwen3-1.7b-28L-60s-b64-w4-l0_14", batch=64, num_q_heads=16,
                num_kv_heads=8, head_dim=128, prefix_len=32, speech_len=750,
                suffix_len=0, decode_steps=128, w=4, l0=14, num_layers=28,
                rho=0.9, dtype="bf16", seed=2)
LONG_10MIN = _wl("qwen3-1.7b-28L-10min-b16-l0_14", batch=16, num_q_heads=16,
                 num_kv_heads=8, head_dim=128, prefix_len=32, speech_len=7500,
                 suffix_len=0, decode_steps=256, w=4, l0=14, num_layers=28,
                 rho=0.95, dtype="bf16", seed=3)
PREFILL_1500 = _wl("qwen3-1.7b-prefill-b8-1596q-471k", batch=8, num_q_heads=16,
                   num_kv_heads=8, head_dim=128, prefix_len=32, speech_len=1500,
                   suffix_len=64, decode_steps=0, w=4, l0=0, num_layers=1,
                   rho=0.9, dtype="bf16", seed=4)
WORKLOADS = [TINY_F32, LAYER_30S, STACK_60S, LONG_10MIN, PREFILL_1500]

# The 60 s stack with a window that grows with depth (2 for layers 14-17, 4 for
# 18-23, 8 for 24-27): an instance of per-layer adaptive compression ratios.
# The paper names them as future work and fixes no schedule; this one is
# illustrative.
ADAPTIVE_W_60S = STACK_60S.with_(name="qwen3-1.7b-28L-60s-b64-l0_14-w2_4_8",
                                 w_layers=(1,) * 14 + (2,) * 4 + (4,) * 6 + (8,) * 4)


def stream_seed(seed: int, layer: int, stream: int, step: int = 0) -> int:
    """63-bit seed of one random stream."""
    state = np.random.SeedSequence([seed, layer, stream, step]).generate_state(2, np.uint32)
    return int((int(state[0]) << 32 | int(state[1])) & ((1 << 63) - 1))


def _gen(device, seed: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def _normal(shape, device, seed) -> torch.Tensor:
    return torch.randn(*shape, generator=_gen(device, seed), device=device,
                       dtype=torch.float32)


def normal(shape, seed: int, device="cpu", scale: float = 1.0,
           dtype: torch.dtype = torch.float32) -> torch.Tensor:
    """Seeded N(0, scale^2) tensor drawn in fp32, rounded once to `dtype`."""
    return (_normal(tuple(shape), device, stream_seed(seed, 0, 99)) * scale).to(dtype)


def ar1(eps: torch.Tensor, rho: float, chunk: int = 64) -> torch.Tensor:
    """Stationary AR(1) along dim 1 of eps [B, T, F] (fp32, any device).

    x_0 = e_0 and x_t = rho x_{t-1} + sqrt(1 - rho^2) e_t.  Computed in blocks
    of `chunk` steps: inside a block the recursion is a lower-triangular
    Toeplitz product, and one carry per block links the blocks.
    """
    B, T, F = eps.shape
    if T == 0:
        return eps.clone()
    dev = eps.device
    c = math.sqrt(1.0 - rho * rho)
    e = eps.clone()
    e[:, 1:] *= c
    nc = -(-T // chunk)
    if nc * chunk != T:
        e = torch.cat([e, torch.zeros(B, nc * chunk - T, F, device=dev)], dim=1)
    e = e.view(B, nc, chunk, F)
    i = torch.arange(chunk, dtype=torch.float64)
    expo = i[:, None] - i[None, :]
    m = torch.where(expo >= 0, torch.pow(torch.tensor(rho, dtype=torch.float64),
                                         expo.clamp(min=0)), torch.zeros(()))
    m = m.to(torch.float32).to(dev)
    y = torch.matmul(m, e)                              # [B, nc, chunk, F]
    pw = torch.pow(torch.tensor(rho, dtype=torch.float64),
                   torch.arange(1, chunk + 1, dtype=torch.float64)).to(torch.float32).to(dev)
    x = torch.empty_like(y)
    carry = torch.zeros(B, F, device=dev)
    for n in range(nc):
        x[:, n] = y[:, n] + pw[None, :, None] * carry[:, None, :]
        carry = x[:, n, -1]
    return x.reshape(B, nc * chunk, F)[:, :T].contiguous()


def raw_kv(wl: Workload, layer: int, device="cpu", rows: Optional[int] = None):
    """Raw (unpooled) K and V of one layer, [B, rows, Hkv, D] in wl's dtype.

    Rows [0, P) and [P+T, P+T+N) are text, rows [P, P+T) are speech; rows
    beyond P+T+N (when rows > prefill_len) are zero.
    """
    B, H, D = wl.batch, wl.num_kv_heads, wl.head_dim
    P, T, N = wl.prefix_len, wl.speech_len, wl.suffix_len
    rows = wl.prefill_len if rows is None else rows
    assert rows >= P + T + N
    out = []
    for s_text, s_speech in ((_S_K_TEXT, _S_K_SPEECH), (_S_V_TEXT, _S_V_SPEECH)):
        x = torch.zeros(B, rows, H * D, device=device, dtype=torch.float32)
        text = _normal((B, P + N, H * D), device, stream_seed(wl.seed, layer, s_text))
        x[:, :P] = text[:, :P]
        x[:, P + T:P + T + N] = text[:, P:]
        if T:
            eps = _normal((B, T, H * D), device, stream_seed(wl.seed, layer, s_speech))
            x[:, P:P + T] = ar1(eps, wl.rho)
        out.append(x.view(B, rows, H, D).to(wl.torch_dtype))
    return out[0], out[1]


def gate(wl: Workload, layer: int, device="cpu", scale: float = 1.0) -> torch.Tensor:
    """Gate vectors u [Hkv, D] fp32 ~ N(0, 1/D), times `scale` (0 = zero gate)."""
    u = _normal((wl.num_kv_heads, wl.head_dim), device,
                stream_seed(wl.seed, layer, _S_GATE)) / math.sqrt(wl.head_dim)
    return (u * scale).contiguous()


def prefill_q(wl: Workload, layer: int, device="cpu", rows: Optional[int] = None):
    """Full-resolution queries [B, rows, Hq, D] ~ N(0, 1) in wl's dtype."""
    rows = wl.prefill_len if rows is None else rows
    q = _normal((wl.batch, rows, wl.num_q_heads, wl.head_dim), device,
                stream_seed(wl.seed, layer, _S_Q_PREFILL))
    return q.to(wl.torch_dtype)


def decode_q(wl: Workload, layer: int, step: int, device="cpu"):
    """Decode-step queries [B, Hq, D] ~ N(0, 1) in wl's dtype."""
    q = _normal((wl.batch, wl.num_q_heads, wl.head_dim), device,
                stream_seed(wl.seed, layer, _S_Q_DECODE, step))
    return q.to(wl.torch_dtype)


def decode_kv_new(wl: Workload, layer: int, step: int, device="cpu"):
    """Key and value of the token decoded at `step`, [B, Hkv, D] ~ N(0, 1)."""
    shape = (wl.batch, wl.num_kv_heads, wl.head_dim)
    k = _normal(shape, device, stream_seed(wl.seed, layer, _S_K_NEW, step))
    v = _normal(shape, device, stream_seed(wl.seed, layer, _S_V_NEW, step))
    return k.to(wl.torch_dtype), v.to(wl.torch_dtype)


def decode_q_all(wl: Workload, layer: int, steps: Sequence[int], device="cpu"):
    """decode_q for several steps stacked: [len(steps), B, Hq, D]."""
    return torch.stack([decode_q(wl, layer, s, device) for s in steps])


def block_table(batch: int, pages_per_seq: int, seed: int, layer: int = 0,
                shuffle: bool = True, spare_pages: int = 0):
    """Page ids [batch, pages_per_seq] int32 over a pool of
    batch * pages_per_seq + spare_pages pages: a random permutation of the pool
    (or the identity when shuffle is False), so that consecutive slots of a
    sequence land in scattered pages."""
    total = batch * pages_per_seq + spare_pages
    if shuffle:
        perm = torch.randperm(total, generator=_gen("cpu", stream_seed(seed, layer, _S_PAGES)))
    else:
        perm = torch.arange(total)
    return perm[:batch * pages_per_seq].view(batch, pages_per_seq).to(torch.int32).contiguous(), total
