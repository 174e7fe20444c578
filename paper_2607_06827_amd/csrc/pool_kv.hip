// Learned window pooling of speech keys/values into the paged KV cache
// (arXiv 2607.06827, Sec. III-B, Eq. 4; Sec. III-C: done once, at prefill).
//
// Work unit: one (sequence b, compressed slot c, KV head g).  D/8 consecutive
// lanes own one unit, each lane 8 elements of the head dimension, so one wave
// covers 64/(D/8) heads of the same slot and reads their rows as one
// contiguous run when the raw tensor is [B][S][Hkv][D].  A block is one
// wave: the blocks are short-lived (a few loads, a few stores), and one-wave
// blocks measured 1.2% faster than four-wave blocks on the 60 s stack (1.9%
// with the sequence lengths requested together, one_run_now).
//   slot c < P                 copy raw row c                       (bitwise)
//   slot P + i, i < nW         softmax-of-gate-logits weighted sum over the
//                              window [P + i*w, min(P + (i+1)*w, P + T))
//   slot P + nW + m            copy raw row P + T + m                (bitwise)
// For sequences with several speech runs (kRuns, a segment table) the slots
// follow the segments in order, each run with its own windows; the span view
// (spans.hpp) gives every slot's source rows either way.
// The gate logit u_g . k_j is a 16-lane (8-lane for D = 64) DPP reduction.
// The window softmax is computed online over groups of four frames so that
// eight loads are in flight per lane; a one-frame window is a copy.  The
// loads are unconditional (frame indices are clamped, frames past the window
// get weight 0) and the block-table entry is checked only before the stores,
// so no branch makes a lane wait for one load before issuing the next.
// The kernel reads each raw row once and writes each cache row once: it is
// bound by HBM bandwidth.  Cache rows are written with non-temporal stores
// (measured 2.6% faster than cached stores on the 60 s stack).
#include "kernels.hpp"
#include "pool_window.hpp"

namespace skv {

namespace {

constexpr int kPoolThreads = 64;
typedef unsigned int nt_u32x4 __attribute__((ext_vector_type(4)));

// Raw rows are read once: bf16 rows come in with non-temporal loads (with
// one-wave blocks 2% faster over the 60 s stack; with four-wave blocks they
// had been slower).
template <typename T>
__device__ __forceinline__ void load_nt(Chunk<T>& c, const T* p) {
  if constexpr (sizeof(T) == 2) {
    const nt_u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const nt_u32x4*>(p));
    c.raw = make_uint4(v[0], v[1], v[2], v[3]);
  } else {
    c.load(p);
  }
}

template <typename T, int D, bool kGate, bool kRuns>
__global__ __launch_bounds__(kPoolThreads) void pool_kv_kernel(PoolArgs a) {
  constexpr int kLanes = D / 8;                   // lanes per unit
  constexpr int kUnits = kPoolThreads / kLanes;   // units per block

  const int b = blockIdx.y;
  const int tid = threadIdx.x;
  const int j = tid % kLanes;
  const int64_t unit = (int64_t)blockIdx.x * kUnits + tid / kLanes;
  const int heads = a.pv.kv_heads;
  const int g = (int)(unit % heads);
  const int64_t c64 = unit / heads;

  const auto sp = span_view<kRuns>(a, b, a.w_eff);
  const int len = sp.clen();
  if (blockIdx.x == 0 && tid == 0 && a.cache_len_out) a.cache_len_out[b] = len;
  if (c64 >= len || c64 >= a.max_out) return;
  const int c = (int)c64;

  const SlotSource sl = sp.slot(c);
  const int src = sl.first, frames = sl.frames;
  // page of slot c: the entry is loaded now and checked only before the stores
  const int idx = c >> a.pv.page_shift;
  const int32_t entry = a.table[(int64_t)b * a.pv.max_pages + min(idx, a.pv.max_pages - 1)];

  const T* kr = static_cast<const T*>(a.k_raw) + b * a.stride_b + g * a.stride_h + 8 * j;
  const T* vr = static_cast<const T*>(a.v_raw) + b * a.stride_b + g * a.stride_h + 8 * j;
  auto at = [&](int s) { return (int64_t)min(s, a.raw_len - 1) * a.stride_s; };
  auto dst = [&]() {
    return page_row<D>(entry, g, c & ((1 << a.pv.page_shift) - 1), a.pv) + 8 * j;
  };
  // rows past the raw tensor (a broken caller obligation) or without a page are skipped
  auto writable = [&]() {
    return src + frames <= a.raw_len && idx < a.pv.max_pages && entry >= 0 &&
           entry < a.pv.num_pages;
  };

  if (frames == 1) {  // text row or one-frame window: weight exactly 1
    Chunk<T> kc, vc;
    load_nt(kc, kr + at(src));
    load_nt(vc, vr + at(src));
    if (writable()) {
      kc.store_nt(static_cast<T*>(a.k_pages) + dst());
      vc.store_nt(static_cast<T*>(a.v_pages) + dst());
    }
    return;
  }

  float u[8];
  if constexpr (kGate) {
    const float4* gp = reinterpret_cast<const float4*>(a.gate + (int64_t)g * D + 8 * j);
    const float4 u0 = gp[0], u1 = gp[1];
    u[0] = u0.x; u[1] = u0.y; u[2] = u0.z; u[3] = u0.w;
    u[4] = u1.x; u[5] = u1.y; u[6] = u1.z; u[7] = u1.w;
  }

  WindowPool<T, kLanes> wp;
  wp.init();
  for (int f0 = 0; f0 < frames; f0 += 4) {
    // all eight loads in flight; frames past the window repeat its last one
    Chunk<T> kc[4], vc[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int64_t o = at(src + min(f0 + t, frames - 1));
      load_nt(kc[t], kr + o);
      load_nt(vc[t], vr + o);
    }
    wp.template add4<kGate>(kc, vc, u, f0, frames);
  }
  Chunk<T> ko, vo;
  wp.finish(ko, vo);
  if (writable()) {
    ko.store_nt(static_cast<T*>(a.k_pages) + dst());
    vo.store_nt(static_cast<T*>(a.v_pages) + dst());
  }
}

template <typename T, int D, bool kRuns>
hipError_t launch_pool_t(const PoolArgs& a, dim3 grid, hipStream_t s) {
  return a.gate ? launch_struct(pool_kv_kernel<T, D, true, kRuns>, grid, dim3(kPoolThreads), s, a)
                : launch_struct(pool_kv_kernel<T, D, false, kRuns>, grid, dim3(kPoolThreads), s, a);
}

template <typename T, int D>
hipError_t launch_pool_d(const PoolArgs& a, dim3 grid, hipStream_t s) {
  return a.segs.seg_start ? launch_pool_t<T, D, true>(a, grid, s) : launch_pool_t<T, D, false>(a, grid, s);
}

}  // namespace

int64_t pool_grid_blocks(int max_out, int kv_heads, int head_dim) {
  const int units_per_block = kPoolThreads / (head_dim / 8);
  const int64_t units = (int64_t)max_out * kv_heads;
  // at least one block per sequence, which also writes cache_len_out
  const int64_t blocks = (units + units_per_block - 1) / units_per_block;
  return blocks > 0 ? blocks : 1;
}

hipError_t launch_pool(const PoolArgs& a, int dtype, int head_dim, int batch, hipStream_t s) {
  const int64_t blocks = pool_grid_blocks(a.max_out, a.pv.kv_heads, head_dim);
  if (blocks > INT32_MAX) return hipErrorInvalidConfiguration;  // the host layer rejects these first
  const dim3 grid((unsigned)blocks, batch);
  if (dtype == 1)
    return head_dim == 128 ? launch_pool_d<bf16_bits, 128>(a, grid, s) : launch_pool_d<bf16_bits, 64>(a, grid, s);
  return head_dim == 128 ? launch_pool_d<float, 128>(a, grid, s) : launch_pool_d<float, 64>(a, grid, s);
}

}  // namespace skv
