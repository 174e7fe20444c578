// Learned window pooling of whole hidden states: the HS Compression variant
// of arXiv 2607.06827 (Sec. IV-A, method (4)), which applies the pooling of
// Eq. 4 to the entire hidden state at layer l0 so that every later layer,
// queries included, runs on the shortened sequence (plain causal attention
// over it is prefill/decode attention with a window of 1).
//
// One wave per output row.  Lane l holds elements [(v*64 + l)*8, +8) of the
// row for v < kVec, so every wave-wide load covers 1 KB (bf16) or 2 KB (fp32)
// of contiguous memory.  Text rows and one-frame windows are bitwise copies.
// A window's frames are pooled with an online softmax over their gate logits
// u . h_j (fp32 dots reduced over the whole wave), in passes of a few frames
// whose loads are all in flight together, so any w works.
// The kernel moves each input byte once and writes each output byte once: it
// is bound by HBM bandwidth.
#include "kernels.hpp"

namespace skv {

namespace {

constexpr float kLog2e = 1.4426950408889634f;

// Sum over all 64 lanes, the same in every lane.
__device__ __forceinline__ float wave_sum(float x) {
  x = group_sum<16>(x);
  const uint32_t u = __float_as_uint(x);
  auto p = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  x = __uint_as_float(p[0]) + __uint_as_float(p[1]);
  const uint32_t u2 = __float_as_uint(x);
  p = __builtin_amdgcn_permlane32_swap(u2, u2, false, false);
  return __uint_as_float(p[0]) + __uint_as_float(p[1]);
}

template <typename T, int kVec>
__global__ __launch_bounds__(256) void pool_hidden_kernel(PoolHiddenArgs a) {
  constexpr int kWavesPerBlock = 4;
  constexpr int kE = kVec * 8;  // elements per lane
  // frames loaded together per pass: about 16 KB of a bf16 wave in flight
  constexpr int kFrames = 16 / kVec < 8 ? 16 / kVec : 8;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int b = blockIdx.y;
  const int c = blockIdx.x * kWavesPerBlock + wave;  // output row

  const int P = max(a.prefix_len[b], 0);
  const int T_ = max(a.speech_len[b], 0);
  const int N = max(a.suffix_len[b], 0);
  const int w = a.w;
  const int nW = (T_ + w - 1) / w;
  const int L = P + nW + N;
  if (c == 0 && lane == 0 && a.out_len) a.out_len[b] = L;
  if (c >= L || c >= a.out_cap) return;

  const T* src = static_cast<const T*>(a.h) + (int64_t)b * a.stride_b;
  T* dst = static_cast<T*>(a.out) + (int64_t)b * a.out_stride_b + (int64_t)c * a.out_stride_s;
  auto row = [&](int s) { return src + (int64_t)min(s, a.raw_len - 1) * a.stride_s; };

  // source rows of output row c: a text row, or the frames of window c - P
  int f0, nf;
  if (c < P) {
    f0 = c;
    nf = 1;
  } else if (c >= P + nW) {
    f0 = P + T_ + (c - P - nW);
    nf = 1;
  } else {
    f0 = P + (c - P) * w;
    nf = min(w, P + T_ - f0);
  }
  if (nf == 1) {  // bitwise copy
    const T* s = row(f0);
#pragma unroll
    for (int v = 0; v < kVec; ++v) {
      Chunk<T> x;
      x.load(s + (v * 64 + lane) * 8);
      x.store(dst + (v * 64 + lane) * 8);
    }
    return;
  }

  float u[kE];
#pragma unroll
  for (int v = 0; v < kVec; ++v)
#pragma unroll
    for (int e = 0; e < 8; ++e) u[v * 8 + e] = a.gate ? a.gate[(v * 64 + lane) * 8 + e] : 0.f;

  float m = neg_inf(), l = 0.f, acc[kE];
#pragma unroll
  for (int e = 0; e < kE; ++e) acc[e] = 0.f;
  for (int base = 0; base < nf; base += kFrames) {
    Chunk<T> x[kFrames][kVec];
#pragma unroll
    for (int f = 0; f < kFrames; ++f) {
      const T* s = row(f0 + min(base + f, nf - 1));  // frames past the window repeat its last
#pragma unroll
      for (int v = 0; v < kVec; ++v) x[f][v].load(s + (v * 64 + lane) * 8);
    }
    float logit[kFrames];
#pragma unroll
    for (int f = 0; f < kFrames; ++f) {
      float d = 0.f;
#pragma unroll
      for (int v = 0; v < kVec; ++v) {
        float xf[8];
        x[f][v].to_float(xf);
#pragma unroll
        for (int e = 0; e < 8; ++e) d = __builtin_fmaf(u[v * 8 + e], xf[e], d);
      }
      logit[f] = base + f < nf ? wave_sum(d) * kLog2e : neg_inf();  // log2 units
    }
    float mx = m;
#pragma unroll
    for (int f = 0; f < kFrames; ++f) mx = fmaxf(mx, logit[f]);
    const float corr = fast_exp2(m - mx);  // 0 on the first pass (m = -inf)
    l *= corr;
#pragma unroll
    for (int e = 0; e < kE; ++e) acc[e] *= corr;
    m = mx;
#pragma unroll
    for (int f = 0; f < kFrames; ++f) {
      const float p = fast_exp2(logit[f] - m);  // 0 for frames past the window
      l += p;
#pragma unroll
      for (int v = 0; v < kVec; ++v) {
        float xf[8];
        x[f][v].to_float(xf);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[v * 8 + e] = __builtin_fmaf(p, xf[e], acc[v * 8 + e]);
      }
    }
  }
  const float inv = 1.f / l;
#pragma unroll
  for (int v = 0; v < kVec; ++v) {
    float y[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) y[e] = acc[v * 8 + e] * inv;
    Chunk<T> out;
    out.from_float(y);
    out.store(dst + (v * 64 + lane) * 8);
  }
}

template <typename T>
hipError_t launch_pool_hidden_t(const PoolHiddenArgs& a, int hidden, int batch, hipStream_t s) {
  // at least one block per sequence: block 0 writes out_len even when every span is empty
  const int blocks = (a.max_out + 3) / 4;
  const dim3 grid((unsigned)(blocks > 0 ? blocks : 1), batch);
  switch (hidden / 512) {
    case 1: return launch_struct(pool_hidden_kernel<T, 1>, grid, dim3(256), s, a);
    case 2: return launch_struct(pool_hidden_kernel<T, 2>, grid, dim3(256), s, a);
    case 4: return launch_struct(pool_hidden_kernel<T, 4>, grid, dim3(256), s, a);
    default: return launch_struct(pool_hidden_kernel<T, 8>, grid, dim3(256), s, a);
  }
}

}  // namespace

bool pool_hidden_supported(int hidden) {
  return hidden == 512 || hidden == 1024 || hidden == 2048 || hidden == 4096;
}

hipError_t launch_pool_hidden(const PoolHiddenArgs& a, int dtype, int hidden, int batch,
                              hipStream_t s) {
  if (dtype == 1) return launch_pool_hidden_t<bf16_bits>(a, hidden, batch, s);
  return launch_pool_hidden_t<float>(a, hidden, batch, s);
}

}  // namespace skv
