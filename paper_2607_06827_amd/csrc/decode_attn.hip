// One decoding step of attention over the compressed paged cache
// (arXiv 2607.06827, Sec. III-B, Eq. 5; Sec. III-C: the cache already holds the
// pooled speech, so each step reads R times fewer speech entries).
//
// Grid (split, kv head g, sequence b); kWaves waves per block.  A block owns
// the key range of one split of one (b, g) for all G query heads of the
// group, so each K/V row is read from HBM once per step and used G times from
// registers.  With enough (b, g) pairs to fill the GPU there is one split and
// the block writes the output directly: one launch per layer.  Otherwise the
// splits write (o, m, l) partials that decode_merge_kernel combines by a
// log-sum-exp reduction in fixed split order.
//
// Key ranges are cut from the host-known bound on the cache length, so the
// first K/V loads wait only on the block-table entries: the first batches
// are requested from the bound before the device cache length arrives, and
// the queries and the masked tail (with the new token's K/V) go out behind
// them.  The wave's table entries sit one per lane and are read back with
// readlane, so every load address is a wave-uniform page base (SGPRs) plus
// a fixed 32-bit per-lane offset.
//
// Lane layout: kLanes = D/8 lanes per key row, 8 elements (16 bytes of bf16,
// 32 of fp32) per lane, so kRows = 64 / kLanes consecutive keys of one page
// form a "group" that the wave reads with one wave-wide load per 16 bytes,
// each covering whole 128-byte lines of one (page, head) block.  A wave
// streams its groups in batches of U groups of K and of V, kDepth batches in
// flight, branch-free, with non-temporal loads (the cache is read once per
// step).  The masked tail of the range (at most one batch: the leftover
// groups and the group holding key L-1) is requested beside the first full
// batch, so no round trip follows the stream.
//
// bf16 rows of 128 (16 lanes) take pairs of groups at a time: the 2G partial
// q.k sums of a lane (v_dot2_f32_bf16 over bf16 pairs) are reduced over the
// row "transposed", so that each lane ends with one full logit and the
// exponent, the growth test and the weight cost one operation per lane; the
// weights of the two keys a lane row holds are rounded to bf16 as a pair (as
// in an MFMA P.V) and every accumulator takes both products with one
// v_dot2_f32_bf16.  Other shapes and the masked tail reduce each logit over
// its row with DPP and accumulate P.V in fp32.  Each lane row keeps its own
// online-softmax sums against a reference max shared by the whole wave
// (moved, with a rescale, only when a ballot shows some logit exceeding it by
// 2^8), so the rows' states add up at the end (DPP / permlane swaps) and the
// waves' states merge through LDS in one step.
//
// If k_new/v_new are given, key L-1 is read from k_new/v_new directly (in the
// masked tail of the wave whose range holds it), and the lanes holding it
// store it into slot L-1 after the stream.  The kernel moves each K/V byte once: it is bound by HBM
// bandwidth.
#include "kernels.hpp"

namespace skv {

namespace {

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

// 16-byte load that does not keep the line in the caches.
__device__ __forceinline__ uint4 stream_load(const void* p) {
  const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
  return make_uint4(v[0], v[1], v[2], v[3]);
}


// E elements of one key row held by one lane, as kVec 16-byte pieces.  With
// kLanes lanes per row, piece i of lane j is bytes [16 (i kLanes + j), +16)
// of the row, so each wave-wide load instruction reads whole 128-byte lines
// (one piece of every lane of kRows consecutive rows).
template <typename T, int E, int kLanes>
struct Row {
  static constexpr int kVec = E * (int)sizeof(T) / 16;
  static constexpr int kElems = 16 / (int)sizeof(T);  // elements per piece
  uint4 v[kVec];
  // element index inside the row of element k of piece i for lane j
  static __device__ __forceinline__ int elem(int i, int j, int k) { return (i * kLanes + j) * kElems + k; }
  // base is wave-uniform, lane_off a 32-bit per-lane offset
  __device__ __forceinline__ void stream(const char* base, uint32_t lane_off) {
#pragma unroll
    for (int i = 0; i < kVec; ++i) v[i] = stream_load(base + lane_off + 16 * kLanes * i);
  }
  __device__ __forceinline__ void load(const T* row, int j) {
#pragma unroll
    for (int i = 0; i < kVec; ++i) v[i] = *reinterpret_cast<const uint4*>(row + elem(i, j, 0));
  }
  __device__ __forceinline__ void store(T* row, int j) const {
#pragma unroll
    for (int i = 0; i < kVec; ++i) *reinterpret_cast<uint4*>(row + elem(i, j, 0)) = v[i];
  }
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int i = 0; i < kVec; ++i) v[i] = make_uint4(0, 0, 0, 0);
  }
  __device__ __forceinline__ uint32_t word(int w) const {
    const uint4& x = v[w / 4];
    return (w & 3) == 0 ? x.x : (w & 3) == 1 ? x.y : (w & 3) == 2 ? x.z : x.w;
  }
  // f[i * kElems + k] = element k of piece i
  __device__ __forceinline__ void to_float(float* f) const {
    if (sizeof(T) == 2) {
#pragma unroll
      for (int w = 0; w < E / 2; ++w) {
        f[2 * w] = __uint_as_float(word(w) << 16);
        f[2 * w + 1] = __uint_as_float(word(w) & 0xffff0000u);
      }
    } else {
#pragma unroll
      for (int w = 0; w < E; ++w) f[w] = __uint_as_float(word(w));
    }
  }
};

// q.k partial dot of one lane's E elements.  bf16 takes the products of the
// raw bf16 pairs with v_dot2_f32_bf16 (exact products, fp32 sums); fp32 uses
// fused multiply-adds.  The logit scale is applied in the exponent.
template <typename T, int E, int kLanes>
struct QSlice {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  Row<T, E, kLanes> q;
  __device__ __forceinline__ float dot(const Row<T, E, kLanes>& k) const {
    float acc = 0.f;
    if (sizeof(T) == 2) {
#pragma unroll
      for (int w = 0; w < E / 2; ++w)
        acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, k.word(w)),
                                              __builtin_bit_cast(bf16x2_t, q.word(w)), acc, false);
    } else {
#pragma unroll
      for (int w = 0; w < E; ++w) acc += __uint_as_float(q.word(w)) * __uint_as_float(k.word(w));
    }
    return acc;
  }
};

// Row sums of n independent values (rows of kLanes lanes), step by step.
template <int kLanes, int n>
__device__ __forceinline__ void row_sums(float* x) {
  static_assert(kLanes == 8 || kLanes == 16, "rows of 8 or 16 lanes");
#pragma unroll
  for (int i = 0; i < n; ++i) x[i] += dpp<kDppQuadXor1>(x[i]);
#pragma unroll
  for (int i = 0; i < n; ++i) x[i] += dpp<kDppQuadXor2>(x[i]);
#pragma unroll
  for (int i = 0; i < n; ++i) x[i] += dpp<kDppHalfMirror>(x[i]);
  if (kLanes == 16) {
#pragma unroll
    for (int i = 0; i < n; ++i) x[i] += dpp<kDppMirror>(x[i]);
  }
}

// Transposed row sums over rows of 16 lanes: n partial sums per lane in, one
// full row sum per lane out, in about n + log2(16/n) + ... steps instead of
// 4 n.  Each level halves the values a lane carries: the lane keeps the half
// picked by one bit of its lane index and adds the partner's copy of that
// half (the partner differs in that bit, so it kept the other half).  The
// levels pair lanes i^8 (row_ror:8), i^7 (row_half_mirror), i^2 and i^1
// (quad permutes); together they cover all 16 lanes of the row.  Lane i ends
// with value number  b3 n/2 + b2 n/4 + b1 n/8 + b0 n/16  (bits of i within
// its row, terms below 1 dropped).
template <int kCtrl, int kBit, int c>
__device__ __forceinline__ void halve_values(float* x, int lane) {
  const bool up = (lane >> kBit) & 1;
#pragma unroll
  for (int t = 0; t < c / 2; ++t) {
    const float keep = up ? x[t + c / 2] : x[t];
    const float send = up ? x[t] : x[t + c / 2];
    x[t] = keep + dpp<kCtrl>(send);
  }
}

template <int n>
__device__ __forceinline__ float transpose_sum16(float* x, int lane) {
  static_assert(n == 1 || n == 2 || n == 4 || n == 8 || n == 16, "power of two up to 16");
  if constexpr (n >= 2) halve_values<kDppRowRor8, 3, n>(x, lane);
  else x[0] += dpp<kDppRowRor8>(x[0]);
  if constexpr (n >= 4) halve_values<kDppHalfMirror, 2, n / 2>(x, lane);
  else x[0] += dpp<kDppHalfMirror>(x[0]);
  if constexpr (n >= 8) halve_values<kDppQuadXor2, 1, n / 4>(x, lane);
  else x[0] += dpp<kDppQuadXor2>(x[0]);
  if constexpr (n >= 16) halve_values<kDppQuadXor1, 0, n / 8>(x, lane);
  else x[0] += dpp<kDppQuadXor1>(x[0]);
  return x[0];
}

// Lane k of each 16-lane row, to every lane of that row (k a constant once
// the caller's loop is unrolled).
__device__ __forceinline__ uint32_t row_bcast(uint32_t x, int k) {
  const int v = (int)x;
  switch (k) {
    case 0: return (uint32_t)__builtin_amdgcn_mov_dpp(v, kDppRowBcast0 + 0, 0xf, 0xf, true);
    case 2: return (uint32_t)__builtin_amdgcn_mov_dpp(v, kDppRowBcast0 + 2, 0xf, 0xf, true);
    case 4: return (uint32_t)__builtin_amdgcn_mov_dpp(v, kDppRowBcast0 + 4, 0xf, 0xf, true);
    default: return (uint32_t)__builtin_amdgcn_mov_dpp(v, kDppRowBcast0 + 6, 0xf, 0xf, true);
  }
}

// Maximum over all 64 lanes (any values), the same in every lane.
__device__ __forceinline__ float full_wave_max(float x) {
  x = fmaxf(x, dpp<kDppQuadXor1>(x));
  x = fmaxf(x, dpp<kDppQuadXor2>(x));
  x = fmaxf(x, dpp<kDppHalfMirror>(x));
  x = fmaxf(x, dpp<kDppMirror>(x));
  auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
  p = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
}

// Running maxima may lag the true maximum by up to 2^kSlack in the exponent
// before the accumulators are rescaled: every weight stays below 2^kSlack, far
// from fp32 overflow, and the final division by the weight sum makes the
// choice of reference exact.  It makes rescaling rare after the first keys.
constexpr float kSlack = 8.f;

template <typename T, int D, int G, int E>
struct DecodeWave {
  static constexpr int kLanes = D / E;       // lanes per key row
  static constexpr int kRows = 64 / kLanes;  // keys per wave-wide load (one group)

  typedef Row<T, E, kLanes> R;
  QSlice<T, E, kLanes> qs[G];
  float scale_log2;
  int lane;
  float m[G], l[G], acc[G][E];  // online softmax state of this lane row (log2 units)

  __device__ __forceinline__ void init() {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      m[h] = neg_inf();
      l[h] = 0.f;
#pragma unroll
      for (int i = 0; i < E; ++i) acc[h][i] = 0.f;
    }
  }

  // Maximum of a row-uniform value over all rows of the wave (lanes with the
  // same j hold the same value within a row after the row reduction).
  static __device__ __forceinline__ float wave_max(float x) {
    if (kLanes == 8) x = fmaxf(x, dpp<kDppRowRor8>(x));
    {
      const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
      x = fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
    }
    const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
  }

  // Consume N loaded groups.  kMasked: some keys may be invalid (valid[u]
  // false, possibly every key of this lane row).  The reference maxima m[h]
  // are the same in every lane of the wave; they move (and the accumulators
  // are rescaled) only when some row's logits exceed them by more than
  // kSlack, decided by a wave-wide ballot.
  // bf16 rows of 16 lanes, pairs of groups, up to 4 heads: the unmasked
  // batches take consume_paired
  static constexpr bool kPaired = sizeof(T) == 2 && kLanes == 16 && G <= 4;

  template <int N, bool kMasked>
  __device__ __forceinline__ void consume(const R* kc, const R* vc, const bool* valid) {
    if constexpr (kPaired && !kMasked && N == 2) {
      consume_paired(kc, vc);
      return;
    }
    float s[N][G];  // unscaled logits; the scale is > 0
#pragma unroll
    for (int u = 0; u < N; ++u)
#pragma unroll
      for (int h = 0; h < G; ++h) s[u][h] = qs[h].dot(kc[u]);
    // row sums, one DPP step at a time over all N*G independent chains so that
    // no step waits on the step just before it
    row_sums<kLanes, N * G>(&s[0][0]);
    if (kMasked) {
#pragma unroll
      for (int u = 0; u < N; ++u)
#pragma unroll
        for (int h = 0; h < G; ++h)
          if (!valid[u]) s[u][h] = neg_inf();
    }
    float mx[G];
    bool grow = false;
#pragma unroll
    for (int h = 0; h < G; ++h) {
      mx[h] = s[0][h];
#pragma unroll
      for (int u = 1; u < N; ++u) mx[h] = fmaxf(mx[h], s[u][h]);
      mx[h] *= scale_log2;
      grow = grow || mx[h] > m[h] + kSlack;
    }
    if (__builtin_amdgcn_ballot_w64(grow)) {
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float M = wave_max(mx[h]);
        if (M > m[h] + kSlack) {
          const float corr = fast_exp2(m[h] - M);
          l[h] *= corr;
#pragma unroll
          for (int i = 0; i < E; ++i) acc[h][i] *= corr;
          m[h] = M;
        }
      }
    }
#pragma unroll
    for (int u = 0; u < N; ++u) {
      float vf[E];
      vc[u].to_float(vf);
#pragma unroll
      for (int h = 0; h < G; ++h) {
        float p = fast_exp2(__builtin_fmaf(s[u][h], scale_log2, -m[h]));
        if (kMasked) p = (m[h] == neg_inf()) ? 0.f : p;  // nothing valid yet
        l[h] += p;
#pragma unroll
        for (int i = 0; i < E; ++i) acc[h][i] += p * vf[i];
      }
    }
  }

  // Two unmasked bf16 groups (keys r of groups u = 0, 1 in lane row r).
  // The 2 G partial q.k sums of a lane are reduced transposed, so that lane
  // (bits b3 b2 b1 b0 of its index in the row) holds the logit of key u = b3
  // for head h = (b2 b1 b0) / (8 / G): the exponent, the growth test and the
  // weight are then one operation per lane for the whole batch.  The weight
  // pair (key 0, key 1) of each head is rounded to bf16 as one pair (as in an
  // MFMA P.V), broadcast over the row, and every accumulator takes both
  // products with one v_dot2_f32_bf16 on the element pair (key 0, key 1) of
  // the row; the weight sum uses the same rounded pair.
  __device__ __forceinline__ void consume_paired(const R* kc, const R* vc) {
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    constexpr int kHeadStride = 8 / G;  // lanes between heads within a half row
    float x[2 * G];
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int h = 0; h < G; ++h) x[u * G + h] = qs[h].dot(kc[u]);
    const float sl = transpose_sum16<2 * G>(x, lane);
    const int hl = (lane & 7) / kHeadStride;  // this lane's head
    float ml = m[0];
#pragma unroll
    for (int h = 1; h < G; ++h) ml = hl == h ? m[h] : ml;
    float t = __builtin_fmaf(sl, scale_log2, -ml);
    if (__builtin_amdgcn_ballot_w64(t > kSlack)) {
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float M = full_wave_max(hl == h ? sl * scale_log2 : neg_inf());
        if (M > m[h] + kSlack) {
          const float corr = fast_exp2(m[h] - M);
          l[h] *= corr;
#pragma unroll
          for (int i = 0; i < E; ++i) acc[h][i] *= corr;
          m[h] = M;
        }
      }
      ml = m[0];
#pragma unroll
      for (int h = 1; h < G; ++h) ml = hl == h ? m[h] : ml;
      t = __builtin_fmaf(sl, scale_log2, -ml);
    }
    const float pw = fast_exp2(t);
    // lanes of key 0 pack (own, key-1 partner); row_newbcast spreads head h's
    // pair from lane h * kHeadStride to its row
    const uint32_t pk = pack_bf16x2(pw, dpp<kDppRowRor8>(pw));
    uint32_t lo[E / 2], hi[E / 2];  // (key 0, key 1) of elements 2w and 2w+1
#pragma unroll
    for (int w = 0; w < E / 2; ++w) {
      const uint32_t a = vc[0].word(w), b = vc[1].word(w);
      lo[w] = __builtin_amdgcn_perm(b, a, 0x05040100u);
      hi[w] = __builtin_amdgcn_perm(b, a, 0x07060302u);
    }
    const bf16x2_t ones = __builtin_bit_cast(bf16x2_t, 0x3f803f80u);  // (1, 1)
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const bf16x2_t pp = __builtin_bit_cast(bf16x2_t, row_bcast(pk, h * kHeadStride));
      l[h] = __builtin_amdgcn_fdot2_f32_bf16(pp, ones, l[h], false);
#pragma unroll
      for (int w = 0; w < E / 2; ++w) {
        acc[h][2 * w] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, lo[w]), pp,
                                                        acc[h][2 * w], false);
        acc[h][2 * w + 1] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, hi[w]), pp,
                                                            acc[h][2 * w + 1], false);
      }
    }
  }
};

// Sum a value over the lane rows of the wave (lane ^ K for K = 8, 16, 32).
// K = 8 reads the partner with DPP row_ror:8; K = 16 and 32 with the gfx950
// permlane swaps, which hand each lane the pair (own, partner) or (partner,
// own): addition is commutative, so both lanes get the same bits.
template <int K>
__device__ __forceinline__ float add_partner(float v) {
  if (K == 8) return v + dpp<kDppRowRor8>(v);
  const uint32_t u = __float_as_uint(v);
  if (K == 16) {
    const auto p = __builtin_amdgcn_permlane16_swap(u, u, false, false);
    return __uint_as_float(p[0]) + __uint_as_float(p[1]);
  }
  const auto p = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return __uint_as_float(p[0]) + __uint_as_float(p[1]);
}

template <int K, int G, int E>
__device__ __forceinline__ void sum_rows(float* l, float (*acc)[E]) {
#pragma unroll
  for (int h = 0; h < G; ++h) {
    l[h] = add_partner<K>(l[h]);
#pragma unroll
    for (int i = 0; i < E; ++i) acc[h][i] = add_partner<K>(acc[h][i]);
  }
}

#ifndef SKV_DECODE_DEPTH
#define SKV_DECODE_DEPTH 2
#endif
constexpr int kDepth = SKV_DECODE_DEPTH;  // load batches in flight per wave
static_assert(kDepth >= 2, "the stream keeps at least one batch in flight");

template <typename T, int D, int G, int NW, int U, int E>
__global__ __launch_bounds__(NW * 64, (G <= 2 ? 4 : 2)) void decode_kernel(DecodeArgs a) {
  typedef DecodeWave<T, D, G, E> W;
  typedef typename W::R R;
  constexpr int kLanes = W::kLanes;
  constexpr int kRows = W::kRows;

  __shared__ float s_acc[NW][G][D];
  __shared__ float s_m[NW][G];
  __shared__ float s_l[NW][G];

  const int split = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r = lane / kLanes, j = lane % kLanes;
  const int heads = a.pv.kv_heads;
  const int hq = heads * G;
  const int shift = a.pv.page_shift;
  const int slot_mask = (1 << shift) - 1;

  // this wave's key groups, cut from the host bound (no device value needed)
  const int cap = min(a.max_len, a.pv.max_pages << shift);
  const int groups = (cap + kRows - 1) / kRows;
  const int per_split = (groups + a.num_splits - 1) / a.num_splits;
  const int s_begin = min(split * per_split, groups);
  const int s_end = min(groups, s_begin + per_split);
  const int per_wave = (s_end - s_begin + NW - 1) / NW;
  const int g_begin = min(s_begin + wave * per_wave, s_end);
  const int g_end = min(s_end, g_begin + per_wave);

  // Prologue.  Only the block-table entries gate the first K/V loads: the
  // first kDepth - 1 batches are requested from the host bound before the
  // cache length arrives (when the length is below the bound, those that turn
  // out to lie past the unmasked range are simply never reduced), and the
  // queries and the masked tail (which reads the new token's K/V) follow.
  const int first_page = (g_begin * kRows) >> shift;
  const int32_t* table = a.table + (int64_t)b * a.pv.max_pages;
  int tbl = -1;
  if (g_begin < g_end && first_page + lane < a.pv.max_pages) tbl = table[first_page + lane];
  const int L = min(max(a.cache_len[b], 0), cap);
  const int64_t num_pages = a.pv.num_pages;
  auto checked = [num_pages](int page) { return (page >= 0 && page < num_pages) ? page : -1; };

  W st;
  st.scale_log2 = a.scale_log2;
  st.lane = lane;
  st.init();

  T* kpool = static_cast<T*>(a.k_pages);
  T* vpool = static_cast<T*>(a.v_pages);
  const bool has_new = a.k_new != nullptr;
  const int64_t new_row = ((int64_t)b * heads + g) * D;
  // byte offset of this lane's first piece inside a group (consecutive rows)
  uint32_t lane_off = (uint32_t)((r * D + R::elem(0, j, 0)) * sizeof(T));

  // page of group grp (wave-uniform), or -1 when the table entry is bad
  auto group_page = [&](int grp) -> int {
    const int pg = (grp * kRows) >> shift;
    const int idx = pg - first_page;
    if (idx < 64) return __builtin_amdgcn_readlane(tbl, idx);  // checked when loaded
    return checked(table[min(pg, a.pv.max_pages - 1)]);
  };
  auto group_base = [&](int page, int grp) -> int64_t {
    return ((((int64_t)page * heads + g) << shift) + ((grp * kRows) & slot_mask)) * D;
  };

  auto issue_full = [&](int gs, R* kc, R* vc) -> bool {
    bool ok = true;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int page = group_page(gs + u);
      ok = ok && page >= 0;
      const int64_t base = group_base(page >= 0 ? page : 0, gs + u) * (int64_t)sizeof(T);
      // An empty asm that "redefines" the 32-bit lane offset in place, next
      // to the loads, keeps the compiler from hoisting a 64-bit per-lane
      // address out of the loop: the loads take the uniform-base +
      // 32-bit-offset (saddr) form with no per-lane address arithmetic.
      asm volatile("" : "+v"(lane_off));
      kc[u].stream(reinterpret_cast<const char*>(kpool) + base, lane_off);
      vc[u].stream(reinterpret_cast<const char*>(vpool) + base, lane_off);
    }
    return ok;
  };

  // Software pipeline over the nbatch unmasked batches, kDepth buffers deep:
  // while batch k is reduced, batches k+1 .. k+kDepth-1 are in flight.  The
  // steady-state loop issues unconditionally (so the wait before each
  // reduction covers only the batch being reduced); buffer indices are
  // compile-time constants throughout, so the buffers stay in registers.
  R kb[kDepth][U], vb[kDepth][U];
  tbl = checked(tbl);
  // The block-table entries are needed before the first batch anyway;
  // waiting for them here once keeps the compiler from re-waiting on them,
  // conservatively, at the head of every loop iteration.  (The cache length
  // is a scalar load with a counter of its own: it stays in flight.)
  __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);

  // The first batches, from the host bound: groups wholly below its last
  // unmasked key.  With the device length L <= bound, every batch the stream
  // below reduces among them is one of these.
  const int bound_unmasked = has_new ? max(cap - 1, 0) : cap;
  const int nbatch_bound = (max(g_begin, min(g_end, bound_unmasked / kRows)) - g_begin) / U;
  bool ok_first[kDepth - 1];
#pragma unroll
  for (int d = 0; d < kDepth - 1; ++d)
    ok_first[d] = d < nbatch_bound ? issue_full(g_begin + d * U, kb[d], vb[d]) : true;

#pragma unroll
  for (int h = 0; h < G; ++h)
    st.qs[h].q.load(static_cast<const T*>(a.q) + ((int64_t)b * hq + g * G + h) * D, j);

  // keys [0, Lc) come from the cache; with k_new, key L-1 comes from k_new
  const int last = L - 1;
  const int Lc = has_new ? max(L - 1, 0) : L;
  // groups wholly inside [0, Lc) take the unmasked path, U at a time
  const int g_full = max(g_begin, min(g_end, Lc / kRows));
  const int nbatch = (g_full - g_begin) / U;
  bool all_ok = true;
#pragma unroll
  for (int d = 0; d < kDepth - 1; ++d)
    if (d < nbatch) all_ok = all_ok && ok_first[d];

  // Masked batch starting at group gs: keys >= L (and groups past the tail)
  // are invalid; key L-1 comes from k_new when given.
  const int g_tail_end = min(g_end, (L + kRows - 1) / kRows);
  auto load_masked = [&](int gs, R* kc, R* vc, bool* valid) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int grp = gs + u;
      const int c = grp * kRows + r;
      valid[u] = grp < g_tail_end && c < L;
      const T* kp = nullptr;  // start of this lane's key row
      const T* vp = nullptr;
      if (valid[u]) {
        if (has_new && c == last) {
          kp = static_cast<const T*>(a.k_new) + new_row;
          vp = static_cast<const T*>(a.v_new) + new_row;
        } else {
          const int page = group_page(grp);
          if (page >= 0) {
            const int64_t base = group_base(page, grp) + (int64_t)r * D;
            kp = kpool + base;
            vp = vpool + base;
          } else {
            valid[u] = false;
          }
        }
      }
      if (valid[u]) {
        kc[u].load(kp, j);
        vc[u].load(vp, j);
      } else {
        kc[u].zero();
        vc[u].zero();
      }
    }
  };

  // The lanes that read key L-1 from k_new/v_new (a masked batch holds it)
  // store that row into slot L-1 of the cache.  No load of this launch reads
  // the slot from the cache, so the store can wait until after the stream.
  auto store_new = [&](int gs, const R* kc, const R* vc, const bool* valid) {
    if (!has_new || last < gs * kRows || last >= (gs + U) * kRows) return;  // wave-uniform
    const int u = last / kRows - gs, grp = gs + u;
    const int page = group_page(grp);
#pragma unroll
    for (int v = 0; v < U; ++v)  // (compile-time register indices)
      if (v == u && valid[v] && r == last % kRows && page >= 0) {
        const int64_t off = group_base(page, grp) + (int64_t)r * D;
        kc[v].store(kpool + off, j);
        vc[v].store(vpool + off, j);
      }
  };

  // The masked tail (at most U groups: the leftover full groups of the
  // batching plus the one group holding key L-1) is requested now, so that
  // its round trip is not added after the stream.
  const int tail_begin = g_begin + nbatch * U;
  R kt[U], vt[U];
  bool tvalid[U];
  load_masked(tail_begin, kt, vt, tvalid);
  int bi = 0;
  for (; bi + 2 * kDepth - 2 < nbatch; bi += kDepth) {
#pragma unroll
    for (int d = 0; d < kDepth; ++d) {
      constexpr int kAhead = kDepth - 1;
      all_ok = issue_full(g_begin + (bi + d + kAhead) * U, kb[(d + kAhead) % kDepth],
                          vb[(d + kAhead) % kDepth]) && all_ok;
      st.template consume<U, false>(kb[d], vb[d], nullptr);
    }
  }
  // drain: fewer than 2 kDepth - 1 batches are left, the first kDepth - 1 of
  // them already in flight
#pragma unroll
  for (int d = 0; d < 2 * kDepth - 2; ++d) {
    if (bi + d < nbatch) {
      if (bi + d + kDepth - 1 < nbatch)
        all_ok = issue_full(g_begin + (bi + d + kDepth - 1) * U, kb[(d + kDepth - 1) % kDepth],
                            vb[(d + kDepth - 1) % kDepth]) && all_ok;
      st.template consume<U, false>(kb[d % kDepth], vb[d % kDepth], nullptr);
    }
  }
  store_new(tail_begin, kt, vt, tvalid);
  // A block-table entry out of range (a caller error) was read as page 0:
  // drop what the unmasked path accumulated rather than mix in that page.
  if (!all_ok) st.init();

  // masked tail: its first batch was loaded up front; any further batches
  // (none with the group accounting above, kept for safety) load here
  st.template consume<U, true>(kt, vt, tvalid);
  for (int gs = tail_begin + U; gs < g_tail_end; gs += U) {
    load_masked(gs, kt, vt, tvalid);
    store_new(gs, kt, vt, tvalid);
    st.template consume<U, true>(kt, vt, tvalid);
  }

  // the lane rows share the reference maxima: their states simply add up
  if (kLanes == 8) sum_rows<8, G, E>(st.l, st.acc);
  sum_rows<16, G, E>(st.l, st.acc);
  sum_rows<32, G, E>(st.l, st.acc);

  if (r == 0) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
#pragma unroll
      for (int i = 0; i < E; ++i) s_acc[wave][h][R::elem(i / R::kElems, j, i % R::kElems)] = st.acc[h][i];
      if (j == 0) {
        s_m[wave][h] = st.m[h];
        s_l[wave][h] = st.l[h];
      }
    }
  }
  __syncthreads();

  // One thread per (head, element) merges the waves: each derives its head's
  // weights from the waves' maxima itself, so one barrier suffices.
  for (int idx = tid; idx < G * D; idx += NW * 64) {
    const int h = idx / D, e = idx % D;
    float M = neg_inf();
#pragma unroll
    for (int w = 0; w < NW; ++w) M = fmaxf(M, s_m[w][h]);
    float num = 0.f, den = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const float mw = s_m[w][h];
      const float f = (mw == neg_inf()) ? 0.f : fast_exp2(mw - M);
      num += f * s_acc[w][h][e];
      den += f * s_l[w][h];
    }
    const int64_t row = (int64_t)b * hq + g * G + h;
    if (a.num_splits == 1) {
      const float o = den > 0.f ? num / den : 0.f;
      if (sizeof(T) == 2)
        static_cast<bf16_bits*>(a.out)[row * D + e] = (bf16_bits)f32_to_bf16(o);
      else
        static_cast<float*>(a.out)[row * D + e] = o;
    } else {
      a.ws_o[(row * a.num_splits + split) * D + e] = num;
      if (e == 0) {
        const int64_t ws = row * a.num_splits + split;
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
  // Every split wrote its partial (an empty one: m = -inf, o = l = 0), so
  // the loads are unconditional and issued eight splits at a time; an empty
  // split gets weight 0.
  float M = neg_inf();
#pragma unroll 8
  for (int s = 0; s < S; ++s) M = fmaxf(M, ml[2 * s]);
  float num = 0.f, den = 0.f;
  if (M != neg_inf()) {
#pragma unroll 8
    for (int s = 0; s < S; ++s) {
      const float ms = ml[2 * s];
      const float f = ms == neg_inf() ? 0.f : fast_exp2(ms - M);
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

// Waves per block and key groups per load batch (tuning knobs; the split
// heuristic of the host layer assumes 4 waves).  Four waves per block beat
// eight at every shape measured but one: 512 (b, kv head) blocks on 256 CUs
// stream 1-2% faster, smaller batches up to 8% faster; a long pooled layer
// of a small batch (16 x 8 heads, ~1900 keys, 4 splits) 2% slower.
#ifndef SKV_DECODE_WAVES
#define SKV_DECODE_WAVES 4
#endif
#ifndef SKV_DECODE_BATCH
#define SKV_DECODE_BATCH 2
#endif
constexpr int kDecodeWaves = SKV_DECODE_WAVES;

// Elements per lane: 8 (one 16-byte piece of bf16, two of fp32).  Wider
// rows per lane cut the per-key reduction but cost more in the final row
// merge than they save on the short caches of pooled layers.
template <typename T, int D, int G>
constexpr int elems_per_lane() { return 8; }

template <typename T, int D, int G>
hipError_t launch_decode_g(const DecodeArgs& a, dim3 grid, hipStream_t s) {
  constexpr int E = elems_per_lane<T, D, G>();
  constexpr int kBytes = E * (int)sizeof(T);  // per lane per key row
  // about 32 bytes of K (and of V) per lane per batch, fewer for wide G
  constexpr int U0 = SKV_DECODE_BATCH * 16 / kBytes;
  constexpr int U = (G >= 8 ? U0 / 2 : U0) > 0 ? (G >= 8 ? U0 / 2 : U0) : 1;
  return launch_struct(decode_kernel<T, D, G, kDecodeWaves, U, E>, grid, dim3(kDecodeWaves * 64), s, a);
}

template <typename T, int D>
hipError_t launch_decode_d(const DecodeArgs& a, int group, dim3 grid, hipStream_t s) {
  switch (group) {
    case 1: return launch_decode_g<T, D, 1>(a, grid, s);
    case 2: return launch_decode_g<T, D, 2>(a, grid, s);
    case 4: return launch_decode_g<T, D, 4>(a, grid, s);
    default: return launch_decode_g<T, D, 8>(a, grid, s);
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
