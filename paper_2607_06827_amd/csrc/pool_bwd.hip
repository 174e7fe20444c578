// Backward of the window pooling (arXiv 2607.06827, Sec. III-B, Eq. 4; Sec.
// III-C: the gate is trained jointly with the model).
//
// For window i with frames j, logits s_j = u_g . k_j, alpha = softmax(s) and
// the gradients dK^_i, dV^_i of its pooled row:
//   dalpha_j = dK^_i . k_j + dV^_i . v_j
//   ds_j     = alpha_j (dalpha_j - sum_j' alpha_j' dalpha_j')
//   dk_j     = alpha_j dK^_i + ds_j u_g,    dv_j = alpha_j dV^_i
//   du_g    += ds_j k_j                    (over every sequence and window)
// A text row (or a one-frame window) was copied, so its gradient is that of
// the row it became.  The slots' source rows come from the span view
// (spans.hpp): one run per sequence, or the runs of a segment table (kRuns).
//
// Layout: each thread owns 8 consecutive elements of one KV head; D/8
// threads cover a (slot, head) unit, and a 256-thread block covers
// 256 / (D/8) consecutive slots of one head of one sequence per pass, `iters`
// passes (iters chosen so that the launch has a few thousand blocks).  Every
// raw row is read at most twice (once more for windows longer than four
// frames) and every gradient row written once: the kernel is bound by HBM
// bandwidth.  The gate gradient is kept per thread, summed over the block
// (lanes with the same elements by a butterfly within the wave, then the
// waves in LDS) into one D-float partial per block, and the partials are
// summed by a second kernel in a fixed order, so the result does not depend
// on scheduling.
#include "kernels.hpp"
#include "kernels_bwd.hpp"

namespace skv {

namespace {

constexpr float kLog2e = 1.4426950408889634f;
typedef unsigned int nt_u32x4 __attribute__((ext_vector_type(4)));

// Raw K/V rows come in with non-temporal loads (29.3 -> 27.2 us at 1596 x 471,
// b=8); the dK^/dV^ rows, written by the attention backward just before,
// were 8% slower that way and keep cached loads.
template <typename T>
__device__ __forceinline__ void load_nt(Chunk<T>& c, const T* p) {
  if constexpr (sizeof(T) == 2) {
    const nt_u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const nt_u32x4*>(p));
    c.raw = make_uint4(v[0], v[1], v[2], v[3]);
  } else {
    c.load(p);
  }
}
constexpr int kTargetBlocks = 4096;  // ~16 blocks per CU; more are taken one pass each

template <int D>
constexpr int lanes_per_head() { return D / 8; }

// Four waves per SIMD (a bound of 128 registers: below it the kernel spills),
// and the raw gradients written with non-temporal stores (no later access of
// this kernel reads them; -5% at 1596 x 471, b=8).
#ifndef SKV_POOLBWD_OCC
#define SKV_POOLBWD_OCC 4
#endif
#ifndef SKV_POOLBWD_NT
#define SKV_POOLBWD_NT 1
#endif

template <typename T, int D, bool kGate, bool kRuns>
__global__ __launch_bounds__(256, SKV_POOLBWD_OCC) void pool_bwd_kernel(PoolBwdArgs a) {
  constexpr int kLanes = lanes_per_head<D>();
  constexpr int kSlotLanes = 256 / kLanes;  // slots per pass
  const int heads = a.kv_heads;
  const int tid = threadIdx.x;
  const int sl = tid / kLanes, j = tid % kLanes;
  const int g = blockIdx.y, b = blockIdx.z;

  const int64_t base = (int64_t)b * a.stride_b + (int64_t)g * a.stride_h + 8 * j;
  const T* kr = static_cast<const T*>(a.k_raw) + base;
  const T* vr = static_cast<const T*>(a.v_raw) + base;
  T* dkr = static_cast<T*>(a.dk_raw) + base;
  T* dvr = static_cast<T*>(a.dv_raw) + base;
  auto at = [&](int s) { return (int64_t)min(s, a.raw_len - 1) * a.stride_s; };

  float uu[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) uu[e] = 0.f;
  float du[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) du[e] = 0.f;

  // one pass: slot c of this block, its gradient rows k0, k1 (dK^) and v0,
  // v1 (dV^) already loaded
  auto pass = [&](int c, const auto& sp, int len, float4 k0, float4 k1, float4 v0, float4 v1)
                  __attribute__((always_inline)) {
    if (c >= len) return;
    const SlotSource slot = sp.slot(c);
    const int src = slot.first, n = slot.frames;
    if (src + n > a.raw_len) return;  // a broken caller obligation: rows left alone

    // gradient of pooled row c (fp32)
    float gk[8], gv[8];
    {
      gk[0] = k0.x; gk[1] = k0.y; gk[2] = k0.z; gk[3] = k0.w; gk[4] = k1.x; gk[5] = k1.y; gk[6] = k1.z; gk[7] = k1.w;
      gv[0] = v0.x; gv[1] = v0.y; gv[2] = v0.z; gv[3] = v0.w; gv[4] = v1.x; gv[5] = v1.y; gv[6] = v1.z; gv[7] = v1.w;
    }
    if (n == 1) {  // a copied row: weight exactly 1, no logit path
      Chunk<T> ok, ov;
      ok.from_float(gk);
      ov.from_float(gv);
      if (SKV_POOLBWD_NT) {
        ok.store_nt(dkr + at(src));
        ov.store_nt(dvr + at(src));
      } else {
        ok.store(dkr + at(src));
        ov.store(dvr + at(src));
      }
      return;
    }

    // the gate row, requested behind this slot's gradient rows (a load at the
    // top of the kernel would make the first slot's loads wait for it)
    if constexpr (kGate) {
      asm volatile("" ::: "memory");
      const float4* gp = reinterpret_cast<const float4*>(a.gate + (int64_t)g * D + 8 * j);
      const float4 u0 = gp[0], u1 = gp[1];
      uu[0] = u0.x; uu[1] = u0.y; uu[2] = u0.z; uu[3] = u0.w;
      uu[4] = u1.x; uu[5] = u1.y; uu[6] = u1.z; uu[7] = u1.w;
    }
    // frames f0..f0+3 (past the window: its last frame, weight 0), their log2
    // logits and dalpha
    Chunk<T> kc[4], vc[4];
    float ls[4], da[4];
    auto group = [&](int f0) __attribute__((always_inline)) {
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int64_t o = at(src + min(f0 + t, n - 1));
        load_nt(kc[t], kr + o);
        load_nt(vc[t], vr + o);
      }
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        float kf[8], vf[8];
        kc[t].to_float(kf);
        vc[t].to_float(vf);
        float s = 0.f, d = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          s = __builtin_fmaf(uu[e], kf[e], s);
          d = __builtin_fmaf(gk[e], kf[e], __builtin_fmaf(gv[e], vf[e], d));
        }
        ls[t] = f0 + t < n ? group_sum<kLanes>(s) * kLog2e : neg_inf();
        da[t] = group_sum<kLanes>(d);
      }
    };
    // pass 1: the window's softmax normaliser Z and sum_j alpha_j dalpha_j
    float m = neg_inf(), z = 0.f, y = 0.f;
    for (int f0 = 0; f0 < n; f0 += 4) {
      group(f0);
      const float mx = fmaxf(m, fmaxf(fmaxf(ls[0], ls[1]), fmaxf(ls[2], ls[3])));
      const float corr = fast_exp2(m - mx);  // 0 on the first group
      z *= corr;
      y *= corr;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const float p = fast_exp2(ls[t] - mx);  // 0 past the window
        z += p;
        y = __builtin_fmaf(p, da[t], y);
      }
      m = mx;
    }
    const float inv = 1.f / z, mean = y * inv;
    // pass 2: the frame gradients (a window of at most four frames is still
    // in registers from pass 1)
    for (int f0 = 0; f0 < n; f0 += 4) {
      if (n > 4) group(f0);
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const float al = fast_exp2(ls[t] - m) * inv;
        const float ds = al * (da[t] - mean);
        float kf[8], gkf[8], gvf[8];
        kc[t].to_float(kf);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          gkf[e] = __builtin_fmaf(ds, uu[e], al * gk[e]);
          gvf[e] = al * gv[e];
          du[e] = __builtin_fmaf(ds, kf[e], du[e]);  // ds = 0 past the window
        }
        if (f0 + t < n) {
          Chunk<T> ok, ov;
          ok.from_float(gkf);
          ov.from_float(gvf);
          const int64_t o = at(src + f0 + t);
          if (SKV_POOLBWD_NT) {
            ok.store_nt(dkr + o);
            ov.store_nt(dvr + o);
          } else {
            ok.store(dkr + o);
            ov.store(dvr + o);
          }
        }
      }
    }
  };
  // the gradient rows of slot c (clamped to the dK^ capacity: a slot past the
  // sequence is never used)
  auto hat_rows = [&](int c, float4& k0, float4& k1, float4& v0, float4& v1) __attribute__((always_inline)) {
    const int64_t row = (((int64_t)b * a.hat_cap + min(c, a.hat_cap - 1)) * heads + g) * D + 8 * j;
    const float4* hk = reinterpret_cast<const float4*>(a.dk_hat + row);
    const float4* hv = reinterpret_cast<const float4*>(a.dv_hat + row);
    k0 = hk[0]; k1 = hk[1];
    v0 = hv[0]; v1 = hv[1];
  };
  const int iters = a.slots_per_block / kSlotLanes;
  auto slot_of = [&](int k) { return (blockIdx.x * iters + k) * kSlotLanes + sl; };
  // the first pass's gradient rows do not depend on the span lengths (the slot
  // comes from the block index): requested before them
  float4 f0k, f1k, f0v, f1v;
  hat_rows(slot_of(0), f0k, f1k, f0v, f1v);
  const auto sp = span_view<kRuns>(a, b, a.w_eff);
  const int len = min(min(sp.clen(), a.max_out), a.hat_cap);
  if (iters > 0) pass(slot_of(0), sp, len, f0k, f1k, f0v, f1v);
  for (int k = 1; k < iters; ++k) {
    float4 k0, k1, v0, v1;
    hat_rows(slot_of(k), k0, k1, v0, v1);
    pass(slot_of(k), sp, len, k0, k1, v0, v1);
  }

  if (!a.du_part) return;
  // this block's gate gradient: the slots of each wave by a butterfly over
  // the lanes that hold the same elements (lane bits above the unit's), then
  // the four waves in LDS, in a fixed order
#pragma unroll
  for (int m = kLanes; m < 64; m <<= 1)
#pragma unroll
    for (int e = 0; e < 8; ++e) du[e] += xor_shuffle(du[e], m);
  __shared__ float s_du[4][D];
  const int wave = tid >> 6, lane = tid & 63;
  if (lane < kLanes) {
#pragma unroll
    for (int e = 0; e < 8; ++e) s_du[wave][8 * lane + e] = du[e];
  }
  __syncthreads();
  if (tid < D) {
    const float sum = (s_du[0][tid] + s_du[1][tid]) + (s_du[2][tid] + s_du[3][tid]);
    a.du_part[(((int64_t)b * a.blocks_per_seq + blockIdx.x) * heads + g) * D + tid] = sum;
  }
}

// du[i] = sum over the per-block partials (a block that saw no slot of its
// head wrote zeros).  One 256-thread block per four consecutive outputs:
// thread t adds the 16-byte loads of partials t, t + 256, ... (four in
// flight), then the block's 256 sums are added in a fixed order, a butterfly
// within each wave and the four waves in LDS.  Blocks go to the XCDs in turn
// (block i to XCD i mod 8), so the output quads are dealt out in eight runs,
// one per XCD: the eight quads of a 128-byte line of a partial are read by
// one XCD's L2, not by eight.  The grid is n / 4 blocks, a multiple of 8.
constexpr int kReduceThreads = 256;
__global__ __launch_bounds__(kReduceThreads) void du_reduce_kernel(const float* part, int parts, int n, float* du) {
  const int i = ((blockIdx.x & 7) * (gridDim.x >> 3) + (blockIdx.x >> 3)) * 4;
  const int t = threadIdx.x;
  float4 acc[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) acc[u] = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int p0 = 0; p0 < parts; p0 += 4 * kReduceThreads) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int p = p0 + u * kReduceThreads + t;
      if (p < parts) {
        const float4 v = *reinterpret_cast<const float4*>(part + (int64_t)p * n + i);
        acc[u].x += v.x; acc[u].y += v.y; acc[u].z += v.z; acc[u].w += v.w;
      }
    }
  }
  float4 s4;
  s4.x = (acc[0].x + acc[1].x) + (acc[2].x + acc[3].x);
  s4.y = (acc[0].y + acc[1].y) + (acc[2].y + acc[3].y);
  s4.z = (acc[0].z + acc[1].z) + (acc[2].z + acc[3].z);
  s4.w = (acc[0].w + acc[1].w) + (acc[2].w + acc[3].w);
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) {
    s4.x += xor_shuffle(s4.x, m); s4.y += xor_shuffle(s4.y, m);
    s4.z += xor_shuffle(s4.z, m); s4.w += xor_shuffle(s4.w, m);
  }
  __shared__ float4 s_sum[kReduceThreads / 64];
  if ((t & 63) == 0) s_sum[t >> 6] = s4;
  __syncthreads();
  if (t == 0) {
    float4 r;
    r.x = (s_sum[0].x + s_sum[1].x) + (s_sum[2].x + s_sum[3].x);
    r.y = (s_sum[0].y + s_sum[1].y) + (s_sum[2].y + s_sum[3].y);
    r.z = (s_sum[0].z + s_sum[1].z) + (s_sum[2].z + s_sum[3].z);
    r.w = (s_sum[0].w + s_sum[1].w) + (s_sum[2].w + s_sum[3].w);
    *reinterpret_cast<float4*>(du + i) = r;
  }
}

template <typename T, int D>
hipError_t launch_t(const PoolBwdArgs& a, int batch, hipStream_t s) {
  const dim3 grid((unsigned)a.blocks_per_seq, (unsigned)a.kv_heads, (unsigned)batch);
  hipError_t e;
  if (a.segs.seg_start)
    e = a.gate ? launch_struct(pool_bwd_kernel<T, D, true, true>, grid, dim3(256), s, a)
               : launch_struct(pool_bwd_kernel<T, D, false, true>, grid, dim3(256), s, a);
  else
    e = a.gate ? launch_struct(pool_bwd_kernel<T, D, true, false>, grid, dim3(256), s, a)
               : launch_struct(pool_bwd_kernel<T, D, false, false>, grid, dim3(256), s, a);
  if (e != hipSuccess || !a.du) return e;
  const int n = a.kv_heads * D;  // a multiple of 64, so n / 4 blocks are a multiple of 8
  hipLaunchKernelGGL(du_reduce_kernel, dim3(n / 4), dim3(kReduceThreads), 0, s, a.du_part,
                     batch * a.blocks_per_seq, n, a.du);
  return hipGetLastError();
}

}  // namespace

int pool_bwd_slots_per_block(int batch, int max_out, int kv_heads, int head_dim) {
  if (head_dim != 64 && head_dim != 128) return 0;
  if (batch < 1 || kv_heads < 1) return 0;
  const int lanes = 256 / (head_dim / 8);                                 // slots per pass
  const int64_t groups = max_out > 0 ? (max_out + lanes - 1) / lanes : 1;  // passes per (sequence, head)
  const int64_t pairs = (int64_t)batch * kv_heads;
  const int64_t blocks = pairs >= kTargetBlocks ? 1 : (kTargetBlocks + pairs - 1) / pairs;  // per pair
  return (int)((groups + blocks - 1) / blocks) * lanes;
}

void pool_bwd_grid(int batch, int max_out, int hat_cap, int kv_heads, int head_dim, int* spb, int* blocks) {
  const int lanes = 256 / (head_dim / 8);
  const int spb_ws = pool_bwd_slots_per_block(batch, max_out, kv_heads, head_dim);
  const int cap = max_out > 0 ? (max_out + spb_ws - 1) / spb_ws : 1;  // blocks the workspace holds
  const int bound = max(min(max_out, hat_cap), 1);                     // slots that can hold work
  const int groups = (bound + lanes - 1) / lanes;
  const int use = min(cap, groups);
  *spb = ((groups + use - 1) / use) * lanes;
  *blocks = (bound + *spb - 1) / *spb;
}

hipError_t launch_pool_bwd(const PoolBwdArgs& a, int dtype, int head_dim, int batch,
                           hipStream_t s) {
  if (dtype == 1)
    return head_dim == 128 ? launch_t<bf16_bits, 128>(a, batch, s) : launch_t<bf16_bits, 64>(a, batch, s);
  return head_dim == 128 ? launch_t<float, 128>(a, batch, s) : launch_t<float, 64>(a, batch, s);
}

}  // namespace skv
