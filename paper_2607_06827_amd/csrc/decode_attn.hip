// One decoding step of attention over the compressed paged cache
// (arXiv 2607.06827, Sec. III-B, Eq. 5; Sec. III-C: the cache already holds the
// pooled speech, so each step reads R times fewer speech entries).
//
// Grid (split, kv head g, sequence b); 4 waves per block.  A block handles
// the key range [split*chunk, min(L, (split+1)*chunk)) of one (b, g) for all
// G query heads of the group, so each K/V row is read from HBM once per step
// and used G times from registers.
//
// Lane layout: D/8 lanes per key row, 8 elements per lane, so a wave-wide
// 16-byte load covers 64/(D/8) consecutive keys = one contiguous 1 KB run of
// a (page, head) block.  Each wave streams U such loads of K and U of V per
// iteration before touching them (2U KB in flight per wave at bf16) and keeps
// an online softmax per lane row; the q.k dot is a DPP reduction over the
// row's lanes.  Row states are merged with cross-row shuffles, wave states
// through LDS, and split states either directly into `out` (one split) or
// into the workspace for decode_merge_kernel, which combines them with a
// log-sum-exp reduction in fixed split order.
//
// If k_new/v_new are given, the block whose range holds slot L-1 stores them
// there, and every block reads that key from k_new/v_new directly.
// The kernel moves each K/V byte once: it is bound by HBM bandwidth.
#include "kernels.hpp"

namespace skv {

namespace {

constexpr int kDecodeWaves = 4;

// Merge two online-softmax states (log2 units).  Empty states have m = -inf.
__device__ __forceinline__ void merge_state(float& m, float& l, float* acc, float mo, float lo,
                                            const float* acco) {
  const float M = fmaxf(m, mo);
  const float fa = (m == neg_inf()) ? 0.f : fast_exp2(m - M);
  const float fb = (mo == neg_inf()) ? 0.f : fast_exp2(mo - M);
  l = l * fa + lo * fb;
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = acc[i] * fa + acco[i] * fb;
  m = M;
}

template <typename T, int D, int G, int U>
__global__ __launch_bounds__(256) void decode_kernel(DecodeArgs a) {
  constexpr int kLanes = D / 8;            // lanes per key row
  constexpr int kRows = 64 / kLanes;       // keys per wave-wide load
  constexpr int kKeysPerWave = U * kRows;  // keys per wave iteration
  constexpr int kStride = kDecodeWaves * kKeysPerWave;

  __shared__ float s_acc[kDecodeWaves][G][D];
  __shared__ float s_m[kDecodeWaves][G];
  __shared__ float s_l[kDecodeWaves][G];

  const int split = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r = lane / kLanes, j = lane % kLanes;
  const int heads = a.pv.kv_heads;
  const int hq = heads * G;
  const int slot_mask = (1 << a.pv.page_shift) - 1;

  const int cap = min(a.max_len, a.pv.max_pages << a.pv.page_shift);
  const int L = min(max(a.cache_len[b], 0), cap);
  int chunk = (L + a.num_splits - 1) / a.num_splits;
  chunk = (chunk + kKeysPerWave - 1) / kKeysPerWave * kKeysPerWave;
  const int c_begin = split * chunk;
  const int c_end = min(L, c_begin + chunk);

  T* kpool = static_cast<T*>(a.k_pages);
  T* vpool = static_cast<T*>(a.v_pages);
  const bool has_new = a.k_new != nullptr;
  const int last = L - 1;
  const T* k_new = has_new ? static_cast<const T*>(a.k_new) + ((int64_t)b * heads + g) * D + 8 * j : nullptr;
  const T* v_new = has_new ? static_cast<const T*>(a.v_new) + ((int64_t)b * heads + g) * D + 8 * j : nullptr;

  // store the newest token's K/V into its slot (once per (b, g))
  if (has_new && L > 0 && c_begin <= last && last < c_end && wave == 0 && r == 0) {
    const int64_t page = page_of(a.table, b, last, a.pv);
    if (page >= 0) {
      const int64_t off = page_row<D>(page, g, last & slot_mask, a.pv) + 8 * j;
      Chunk<T> kc, vc;
      kc.load(k_new);
      vc.load(v_new);
      kc.store(kpool + off);
      vc.store(vpool + off);
    }
  }

  // queries of the G heads, pre-scaled so that exp2 gives softmax(scale q.k)
  float qf[G][8];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    Chunk<T> qc;
    qc.load(static_cast<const T*>(a.q) + ((int64_t)b * hq + g * G + h) * D + 8 * j);
    qc.to_float(qf[h]);
#pragma unroll
    for (int i = 0; i < 8; ++i) qf[h][i] *= a.scale_log2;
  }

  float m[G], l[G], acc[G][8];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    m[h] = neg_inf();
    l[h] = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[h][i] = 0.f;
  }

  for (int base = c_begin + wave * kKeysPerWave; base < c_end; base += kStride) {
    Chunk<T> kc[U], vc[U];
    bool valid[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int c = base + u * kRows + r;
      valid[u] = c < c_end;
      const T* kp = nullptr;
      const T* vp = nullptr;
      if (valid[u]) {
        if (has_new && c == last) {
          kp = k_new;
          vp = v_new;
        } else {
          const int64_t page = page_of(a.table, b, c, a.pv);
          if (page >= 0) {
            const int64_t off = page_row<D>(page, g, c & slot_mask, a.pv) + 8 * j;
            kp = kpool + off;
            vp = vpool + off;
          } else {
            valid[u] = false;
          }
        }
      }
      if (valid[u]) {
        kc[u].load(kp);
        vc[u].load(vp);
      } else {
        kc[u].zero();
        vc[u].zero();
      }
    }
    float s[U][G];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float kf[8];
      kc[u].to_float(kf);
#pragma unroll
      for (int h = 0; h < G; ++h) {
        float part = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) part += qf[h][i] * kf[i];
        s[u][h] = group_sum<kLanes>(part);
        if (!valid[u]) s[u][h] = neg_inf();
      }
    }
    float mn[G], corr[G];
#pragma unroll
    for (int h = 0; h < G; ++h) {
      float mx = s[0][h];
#pragma unroll
      for (int u = 1; u < U; ++u) mx = fmaxf(mx, s[u][h]);
      mn[h] = fmaxf(m[h], mx);
      // a lane row that has seen no valid key yet keeps m = -inf
      corr[h] = (mn[h] == neg_inf()) ? 1.f : fast_exp2(m[h] - mn[h]);
      l[h] *= corr[h];
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[h][i] *= corr[h];
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float vf[8];
      vc[u].to_float(vf);
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float p = (mn[h] == neg_inf()) ? 0.f : fast_exp2(s[u][h] - mn[h]);
        l[h] += p;
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[h][i] += p * vf[i];
      }
    }
#pragma unroll
    for (int h = 0; h < G; ++h) m[h] = mn[h];
  }

  // merge the kRows lane rows of the wave (lanes with the same j)
#pragma unroll
  for (int off = kLanes; off < 64; off <<= 1) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      float acco[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) acco[i] = xor_shuffle(acc[h][i], off);
      const float mo = xor_shuffle(m[h], off);
      const float lo = xor_shuffle(l[h], off);
      merge_state(m[h], l[h], acc[h], mo, lo, acco);
    }
  }
  if (r == 0) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
#pragma unroll
      for (int i = 0; i < 8; ++i) s_acc[wave][h][8 * j + i] = acc[h][i];
      if (j == 0) {
        s_m[wave][h] = m[h];
        s_l[wave][h] = l[h];
      }
    }
  }
  __syncthreads();

  // merge the waves; one thread per (head, element)
  for (int idx = tid; idx < G * D; idx += 256) {
    const int h = idx / D, e = idx % D;
    float M = neg_inf();
#pragma unroll
    for (int w = 0; w < kDecodeWaves; ++w) M = fmaxf(M, s_m[w][h]);
    float num = 0.f, den = 0.f;
    if (M != neg_inf()) {
#pragma unroll
      for (int w = 0; w < kDecodeWaves; ++w) {
        const float mw = s_m[w][h];
        if (mw == neg_inf()) continue;
        const float f = fast_exp2(mw - M);
        num += f * s_acc[w][h][e];
        den += f * s_l[w][h];
      }
    }
    const int64_t row = (int64_t)b * hq + g * G + h;
    if (a.num_splits == 1) {
      const float o = den > 0.f ? num / den : 0.f;
      if (sizeof(T) == 2)
        static_cast<bf16_bits*>(a.out)[row * D + e] = (bf16_bits)f32_to_bf16(o);
      else
        static_cast<float*>(a.out)[row * D + e] = o;
    } else {
      const int64_t ws = row * a.num_splits + split;
      a.ws_o[ws * D + e] = num;
      if (e == 0) {
        a.ws_ml[ws * 2] = M;
        a.ws_ml[ws * 2 + 1] = den;
      }
    }
  }
}

// Log-sum-exp merge of the split partials of one (b, h); fixed split order.
template <typename T, int D>
__global__ __launch_bounds__(D) void decode_merge_kernel(DecodeArgs a) {
  const int h = blockIdx.x, b = blockIdx.y, e = threadIdx.x;
  const int hq = gridDim.x;
  const int S = a.num_splits;
  const int64_t row = (int64_t)b * hq + h;
  const float* ml = a.ws_ml + row * S * 2;
  const float* po = a.ws_o + row * S * D + e;
  float M = neg_inf();
  for (int s = 0; s < S; ++s) M = fmaxf(M, ml[2 * s]);
  float num = 0.f, den = 0.f;
  if (M != neg_inf()) {
    for (int s = 0; s < S; ++s) {
      const float ms = ml[2 * s];
      if (ms == neg_inf()) continue;
      const float f = fast_exp2(ms - M);
      num += f * po[(int64_t)s * D];
      den += f * ml[2 * s + 1];
    }
  }
  const float o = den > 0.f ? num / den : 0.f;
  if (sizeof(T) == 2)
    static_cast<bf16_bits*>(a.out)[row * D + e] = (bf16_bits)f32_to_bf16(o);
  else
    static_cast<float*>(a.out)[row * D + e] = o;
}

template <typename T, int D>
hipError_t launch_decode_d(const DecodeArgs& a, int group, dim3 grid, hipStream_t s) {
  const dim3 block(256);
  // fp32 rows are twice as wide: halve the unroll to bound registers
  constexpr int U = sizeof(T) == 2 ? 8 : 4;
  switch (group) {
    case 1: return launch_struct(decode_kernel<T, D, 1, U>, grid, block, s, a);
    case 2: return launch_struct(decode_kernel<T, D, 2, U>, grid, block, s, a);
    case 4: return launch_struct(decode_kernel<T, D, 4, U>, grid, block, s, a);
    default: return launch_struct(decode_kernel<T, D, 8, U / 2>, grid, block, s, a);
  }
}

}  // namespace

hipError_t launch_decode(const DecodeArgs& a, int dtype, int head_dim, int group, int batch,
                         hipStream_t s) {
  const dim3 grid(a.num_splits, a.pv.kv_heads, batch);
  if (dtype == 1) {
    if (head_dim == 128) return launch_decode_d<bf16_bits, 128>(a, group, grid, s);
    return launch_decode_d<bf16_bits, 64>(a, group, grid, s);
  }
  if (head_dim == 128) return launch_decode_d<float, 128>(a, group, grid, s);
  return launch_decode_d<float, 64>(a, group, grid, s);
}

hipError_t launch_decode_merge(const DecodeArgs& a, int dtype, int head_dim, int num_q_heads,
                               int batch, hipStream_t s) {
  const dim3 grid(num_q_heads, batch);
  const dim3 block(head_dim);
  if (dtype == 1) {
    if (head_dim == 128) return launch_struct(decode_merge_kernel<bf16_bits, 128>, grid, block, s, a);
    return launch_struct(decode_merge_kernel<bf16_bits, 64>, grid, block, s, a);
  }
  if (head_dim == 128) return launch_struct(decode_merge_kernel<float, 128>, grid, block, s, a);
  return launch_struct(decode_merge_kernel<float, 64>, grid, block, s, a);
}

}  // namespace skv
