// Learned window pooling of whole hidden states: the HS Compression variant
// of arXiv 2607.06827 (Sec. IV-A, method (4)), which applies the pooling of
// Eq. 4 to the entire hidden state at layer l0 so that every later layer,
// queries included, runs on the shortened sequence (plain causal attention
// over it is prefill/decode attention with a window of 1).
//
// Layout: each thread owns 8 consecutive elements (one 16-byte piece for
// bf16) of a row for each of kVec slices, kTpr threads cover one row, and a
// 256-thread block handles 256 / kTpr output rows (one row for hidden 2048
// and 4096, so a row is spread over four waves).  Text rows and one-frame
// windows are bitwise copies.  A window's frames are pooled with an online
// softmax over the gate logits u . h_j in passes of four frames: every load
// of a pass (the gate and all four frames) is issued before the first one is
// used, each wave reduces its share of the dot products with cross-lane
// operations, and the per-wave partial logits meet in LDS behind one barrier
// per pass.  The loads are unconditional (row indices are clamped instead),
// so no branch forces an early wait for outstanding loads.
// The kernel moves each input byte once and writes each output byte once: it
// is bound by HBM bandwidth.  bf16 rows are read with non-temporal loads
// (streamed once, they need not stay in the caches).
#include "kernels.hpp"

namespace skv {

namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kFrames = 4;  // frames per pass
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

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

// One streamed 8-element piece of a hidden-state row.
template <typename T>
__device__ __forceinline__ void load_piece(Chunk<T>& x, const T* p) {
  if constexpr (sizeof(T) == 2) {
    const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
    x.raw = make_uint4(v[0], v[1], v[2], v[3]);
  } else {
    x.load(p);
  }
}

template <typename T, int kTpr, int kVec, bool kGate>
__global__ __launch_bounds__(256) void pool_hidden_kernel(PoolHiddenArgs a) {
  constexpr int kRows = 256 / kTpr;  // output rows per block
  constexpr int kWavesPerRow = kTpr / 64;
  constexpr int kE = kVec * 8;       // elements per thread
  __shared__ float s_part[2][4][kFrames];  // [pass parity][wave][frame]
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int lr = tid % kTpr;   // thread within its row
  const int rib = tid / kTpr;  // row within the block
  const int b = blockIdx.y;
  const int cb = blockIdx.x * kRows;
  const int c = cb + rib;      // output row

  const OneRun run = one_run_now(a.prefix_len, a.speech_len, a.suffix_len, b, a.w);
  const int P = run.P, T_ = run.T, N = run.N, w = run.w, nW = run.nW;
  const int L = P + nW + N;
  if (blockIdx.x == 0 && tid == 0 && a.out_len) a.out_len[b] = L;
  const int lim = min(L, a.out_cap);
  if (cb >= lim) return;  // block-uniform

  const T* src = static_cast<const T*>(a.h) + (int64_t)b * a.stride_b;
  T* dst = static_cast<T*>(a.out) + (int64_t)b * a.out_stride_b + (int64_t)c * a.out_stride_s;
  auto row = [&](int s) { return src + (int64_t)min(s, a.raw_len - 1) * a.stride_s; };
  auto elt = [&](int v) { return (v * kTpr + lr) * 8; };

  // source rows of output row c: nf = 1 for a text row or a one-frame window
  // (a copy), nf = 0 past the sequence's end or the buffer's capacity
  const bool text_before = c < P, text_after = c >= P + nW;
  const int f0 = text_before ? c : text_after ? P + T_ + (c - P - nW) : P + (c - P) * w;
  const int nf = c >= lim ? 0 : (text_before || text_after) ? 1 : min(w, P + T_ - f0);

  // block-uniform: does any row of this block pool a window of several frames?
  const bool block_pools = w > 1 && cb < min(P + nW, lim) && cb + kRows > P;
  if (!block_pools) {
    Chunk<T> x[kVec];
#pragma unroll
    for (int v = 0; v < kVec; ++v) load_piece(x[v], row(f0) + elt(v));
    if (nf == 1)
#pragma unroll
      for (int v = 0; v < kVec; ++v) x[v].store(dst + elt(v));
    return;
  }

  float u[kE];
  if constexpr (kGate) {
#pragma unroll
    for (int v = 0; v < kVec; ++v) {
      const float4* g = reinterpret_cast<const float4*>(a.gate + elt(v));
      const float4 g0 = g[0], g1 = g[1];
      u[v * 8 + 0] = g0.x; u[v * 8 + 1] = g0.y; u[v * 8 + 2] = g0.z; u[v * 8 + 3] = g0.w;
      u[v * 8 + 4] = g1.x; u[v * 8 + 5] = g1.y; u[v * 8 + 6] = g1.z; u[v * 8 + 7] = g1.w;
    }
  }

  float m = neg_inf(), l = 0.f, acc[kE];
#pragma unroll
  for (int e = 0; e < kE; ++e) acc[e] = 0.f;
  Chunk<T> first[kVec];  // frame 0: the output of a copy row
  const int passes = (w + kFrames - 1) / kFrames;  // block-uniform
  for (int p = 0; p < passes; ++p) {
    const int base = p * kFrames;
    Chunk<T> x[kFrames][kVec];
#pragma unroll
    for (int f = 0; f < kFrames; ++f) {
      // frames past the window repeat its last one; copy and dead rows re-read their own row
      const T* s = row(f0 + min(base + f, max(nf, 1) - 1));
#pragma unroll
      for (int v = 0; v < kVec; ++v) load_piece(x[f][v], s + elt(v));
    }
    if (p == 0)
#pragma unroll
      for (int v = 0; v < kVec; ++v) first[v] = x[0][v];
    if constexpr (kGate) {
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
        d = wave_sum(d);
        if (lane == 0) s_part[p & 1][wave][f] = d;
      }
      // two parity buffers: a wave that runs ahead writes the other one, and it
      // cannot come back to this one before every wave has passed the next barrier
      __syncthreads();
    }
    float logit[kFrames];
#pragma unroll
    for (int f = 0; f < kFrames; ++f) {
      float d = 0.f;  // the zero gate: every frame weighs the same
      if constexpr (kGate)
#pragma unroll
        for (int k = 0; k < kWavesPerRow; ++k) d += s_part[p & 1][rib * kWavesPerRow + k][f];
      logit[f] = base + f < nf ? d * kLog2e : neg_inf();  // log2 units
    }
    float mx = m;
#pragma unroll
    for (int f = 0; f < kFrames; ++f) mx = fmaxf(mx, logit[f]);
    mx = fmaxf(mx, -1e30f);  // a row without frames keeps finite weights (it is never stored)
    const float corr = fast_exp2(m - mx);  // 0 on the first pass (m = -inf)
    l *= corr;
#pragma unroll
    for (int e = 0; e < kE; ++e) acc[e] *= corr;
    m = mx;
#pragma unroll
    for (int f = 0; f < kFrames; ++f) {
      const float pw = fast_exp2(logit[f] - mx);  // 0 for frames past the window
      l += pw;
#pragma unroll
      for (int v = 0; v < kVec; ++v) {
        float xf[8];
        x[f][v].to_float(xf);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[v * 8 + e] = __builtin_fmaf(pw, xf[e], acc[v * 8 + e]);
      }
    }
  }
  const float inv = 1.f / l;
#pragma unroll
  for (int v = 0; v < kVec; ++v) {
    float y[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) y[e] = acc[v * 8 + e] * inv;
    Chunk<T> o;
    o.from_float(y);
    if (nf == 1) o = first[v];
    if (nf >= 1) o.store(dst + elt(v));
  }
}

template <typename T, bool kGate>
hipError_t launch_pool_hidden_t(const PoolHiddenArgs& a, int hidden, int batch, hipStream_t s) {
  auto grid = [&](int rows_per_block) {
    const int blocks = (a.max_out + rows_per_block - 1) / rows_per_block;
    // at least one block per sequence: block 0 writes out_len even when every span is empty
    return dim3((unsigned)(blocks > 0 ? blocks : 1), batch);
  };
  switch (hidden) {
    case 512: return launch_struct(pool_hidden_kernel<T, 64, 1, kGate>, grid(4), dim3(256), s, a);
    case 1024: return launch_struct(pool_hidden_kernel<T, 128, 1, kGate>, grid(2), dim3(256), s, a);
    case 2048: return launch_struct(pool_hidden_kernel<T, 256, 1, kGate>, grid(1), dim3(256), s, a);
    default: return launch_struct(pool_hidden_kernel<T, 256, 2, kGate>, grid(1), dim3(256), s, a);
  }
}

template <typename T>
hipError_t launch_pool_hidden_g(const PoolHiddenArgs& a, int hidden, int batch, hipStream_t s) {
  return a.gate ? launch_pool_hidden_t<T, true>(a, hidden, batch, s)
                : launch_pool_hidden_t<T, false>(a, hidden, batch, s);
}

}  // namespace

bool pool_hidden_supported(int hidden) {
  return hidden == 512 || hidden == 1024 || hidden == 2048 || hidden == 4096;
}

hipError_t launch_pool_hidden(const PoolHiddenArgs& a, int dtype, int hidden, int batch,
                              hipStream_t s) {
  if (dtype == 1) return launch_pool_hidden_g<bf16_bits>(a, hidden, batch, s);
  return launch_pool_hidden_g<float>(a, hidden, batch, s);
}

}  // namespace skv
