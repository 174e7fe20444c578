// Learned window pooling of speech keys/values into the paged KV cache
// (arXiv 2607.06827, Sec. III-B, Eq. 4; Sec. III-C: done once, at prefill).
//
// Work unit: one (sequence b, compressed slot c, KV head g).  D/8 consecutive
// lanes own one unit, each lane 8 elements of the head dimension, so one wave
// covers 64/(D/8) heads of the same slot and reads their rows as one
// contiguous run when the raw tensor is [B][S][Hkv][D].
//   slot c < P                 copy raw row c                       (bitwise)
//   slot P + i, i < nW         softmax-of-gate-logits weighted sum over the
//                              window [P + i*w, min(P + (i+1)*w, P + T))
//   slot P + nW + m            copy raw row P + T + m                (bitwise)
// The gate logit u_g . k_j is a 16-lane (8-lane for D = 64) DPP reduction.
// The window softmax is computed online over groups of four frames so that
// eight loads are in flight per lane; a one-frame window is a copy.
// The kernel reads each raw row once and writes each cache row once: it is
// bound by HBM bandwidth.
#include "kernels.hpp"

namespace skv {

namespace {

template <typename T, int D>
__global__ __launch_bounds__(256) void pool_kv_kernel(PoolArgs a) {
  constexpr int kLanes = D / 8;          // lanes per unit
  constexpr int kUnits = 256 / kLanes;   // units per block
  constexpr float kLog2e = 1.4426950408889634f;

  const int b = blockIdx.y;
  const int tid = threadIdx.x;
  const int j = tid % kLanes;
  const int64_t unit = (int64_t)blockIdx.x * kUnits + tid / kLanes;
  const int heads = a.pv.kv_heads;
  const int g = (int)(unit % heads);
  const int64_t c64 = unit / heads;

  const int P = max(a.prefix_len[b], 0);
  const int S = max(a.speech_len[b], 0);  // speech frames
  const int N = max(a.suffix_len[b], 0);
  const int w = a.w_eff;
  const int nW = (S + w - 1) / w;
  const int len = P + nW + N;
  if (blockIdx.x == 0 && tid == 0 && a.cache_len_out) a.cache_len_out[b] = len;
  if (c64 >= len || c64 >= a.max_out) return;
  const int c = (int)c64;

  int src, frames;
  if (c < P) {
    src = c;
    frames = 1;
  } else if (c < P + nW) {
    src = P + (c - P) * w;
    frames = min(w, P + S - src);
  } else {
    src = P + S + (c - P - nW);
    frames = 1;
  }
  if (src + frames > a.raw_len) return;
  const int64_t page = page_of(a.table, b, c, a.pv);
  if (page < 0) return;
  const int64_t dst = page_row<D>(page, g, c & ((1 << a.pv.page_shift) - 1), a.pv) + 8 * j;

  const T* kr = static_cast<const T*>(a.k_raw) + b * a.stride_b + g * a.stride_h + 8 * j;
  const T* vr = static_cast<const T*>(a.v_raw) + b * a.stride_b + g * a.stride_h + 8 * j;
  T* kd = static_cast<T*>(a.k_pages) + dst;
  T* vd = static_cast<T*>(a.v_pages) + dst;

  if (frames == 1) {  // text row or one-frame window: weight exactly 1
    Chunk<T> kc, vc;
    kc.load(kr + src * a.stride_s);
    vc.load(vr + src * a.stride_s);
    kc.store(kd);
    vc.store(vd);
    return;
  }

  // gate slice of this lane, pre-multiplied by log2(e) so that exp2 gives the
  // natural-base softmax of the logits
  float u[8];
  if (a.gate) {
    const float4* gp = reinterpret_cast<const float4*>(a.gate + (int64_t)g * D + 8 * j);
    float4 u0 = gp[0], u1 = gp[1];
    u[0] = u0.x; u[1] = u0.y; u[2] = u0.z; u[3] = u0.w;
    u[4] = u1.x; u[5] = u1.y; u[6] = u1.z; u[7] = u1.w;
#pragma unroll
    for (int i = 0; i < 8; ++i) u[i] *= kLog2e;
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) u[i] = 0.f;
  }

  float m = neg_inf(), l = 0.f, ak[8], av[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) ak[i] = av[i] = 0.f;

  for (int f0 = 0; f0 < frames; f0 += 4) {
    Chunk<T> kc[4], vc[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      if (f0 + t < frames) {
        kc[t].load(kr + (int64_t)(src + f0 + t) * a.stride_s);
        vc[t].load(vr + (int64_t)(src + f0 + t) * a.stride_s);
      } else {
        kc[t].zero();
        vc[t].zero();
      }
    }
    float kf[4][8], s[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      kc[t].to_float(kf[t]);
      float part = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) part += u[i] * kf[t][i];
      s[t] = group_sum<kLanes>(part);
      if (f0 + t >= frames) s[t] = neg_inf();
    }
    const float mn = fmaxf(m, fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3])));
    const float corr = fast_exp2(m - mn);  // m = -inf on the first group gives 0
    l *= corr;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      ak[i] *= corr;
      av[i] *= corr;
    }
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const float p = fast_exp2(s[t] - mn);
      float vf[8];
      vc[t].to_float(vf);
      l += p;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        ak[i] += p * kf[t][i];
        av[i] += p * vf[i];
      }
    }
    m = mn;
  }
  const float inv = 1.f / l;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    ak[i] *= inv;
    av[i] *= inv;
  }
  Chunk<T> ko, vo;
  ko.from_float(ak);
  vo.from_float(av);
  ko.store(kd);
  vo.store(vd);
}

}  // namespace

hipError_t launch_pool(const PoolArgs& a, int dtype, int head_dim, int batch, hipStream_t s) {
  const int units_per_block = 256 / (head_dim / 8);
  const int64_t units = (int64_t)a.max_out * a.pv.kv_heads;
  // at least one block per sequence, which also writes cache_len_out
  const int64_t blocks = (units + units_per_block - 1) / units_per_block;
  const dim3 grid((unsigned)(blocks > 0 ? blocks : 1), batch);
  const dim3 block(256);
  if (dtype == 1) {
    if (head_dim == 128) return launch_struct(pool_kv_kernel<bf16_bits, 128>, grid, block, s, a);
    return launch_struct(pool_kv_kernel<bf16_bits, 64>, grid, block, s, a);
  }
  if (head_dim == 128) return launch_struct(pool_kv_kernel<float, 128>, grid, block, s, a);
  return launch_struct(pool_kv_kernel<float, 64>, grid, block, s, a);
}

}  // namespace skv
