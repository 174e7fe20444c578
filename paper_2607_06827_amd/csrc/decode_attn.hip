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
// block-table entries, the queries and the cache length are all requested at
// once and the first K/V loads wait on a single memory round trip.  The wave's
// table entries sit one per lane and are read back with readlane, so every
// load address is a wave-uniform page base plus a fixed per-lane offset.
//
// Lane layout: kLanes lanes per key row, E elements per lane in 16-byte
// pieces (bf16 rows of 128 with G <= 2: 8 lanes x 16 elements, otherwise
// D/8 lanes x 8), so kRows = 64 / kLanes consecutive keys of one page form a
// "group" that the wave reads with E*elt/16 wave-wide loads, each covering
// whole 128-byte lines of one (page, head) block.  A wave streams its
// groups in batches of U loads of K and of V, double-buffered so that the next
// batch is in flight while the current one is reduced.  Batches of groups that
// lie wholly inside the cache take a branch-free path with non-temporal loads
// (the cache is read once per step); the last partial group and the newest
// token go through a masked tail.  q.k is a v_dot2_f32_bf16 partial (fma for
// fp32) reduced over the row's lanes with DPP; each lane row keeps its own
// online-softmax sum against a reference max shared by the whole wave (moved,
// with a rescale, only when a ballot shows some row exceeding it by 2^8), so
// the rows' states add up at the end (DPP / permlane swaps) and the waves'
// states merge through LDS.
//
// If k_new/v_new are given, the wave whose range holds slot L-1 stores them
// there, and that key is read from k_new/v_new directly.
// The kernel moves each K/V byte once: it is bound by HBM bandwidth.
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

template <int kLanes>
__device__ __forceinline__ float row_sum(float x) {
  static_assert(kLanes == 8 || kLanes == 16, "rows of 8 or 16 lanes");
  return group_sum<kLanes>(x);
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
  template <int N, bool kMasked>
  __device__ __forceinline__ void consume(const R* kc, const R* vc, const bool* valid) {
    float s[N][G];  // unscaled logits; the scale is > 0
#pragma unroll
    for (int u = 0; u < N; ++u) {
#pragma unroll
      for (int h = 0; h < G; ++h) {
        s[u][h] = row_sum<kLanes>(qs[h].dot(kc[u]));
        if (kMasked && !valid[u]) s[u][h] = neg_inf();
      }
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

template <typename T, int D, int G, int NW, int U, int E>
__global__ __launch_bounds__(NW * 64, (G <= 2 ? 4 : 2)) void decode_kernel(DecodeArgs a) {
  typedef DecodeWave<T, D, G, E> W;
  typedef typename W::R R;
  constexpr int kLanes = W::kLanes;
  constexpr int kRows = W::kRows;

  __shared__ float s_acc[NW][G][D];
  __shared__ float s_m[NW][G];
  __shared__ float s_l[NW][G];
  __shared__ float s_w[NW][G];  // per-wave merge weights
  __shared__ float s_den[G];

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

  // independent prologue loads: cache length, queries, block-table entries
  const int L = min(max(a.cache_len[b], 0), cap);
  const int first_page = (g_begin * kRows) >> shift;
  const int32_t* table = a.table + (int64_t)b * a.pv.max_pages;
  int tbl = -1;
  if (g_begin < g_end && first_page + lane < a.pv.max_pages) tbl = table[first_page + lane];

  W st;
#pragma unroll
  for (int h = 0; h < G; ++h)
    st.qs[h].q.load(static_cast<const T*>(a.q) + ((int64_t)b * hq + g * G + h) * D, j);
  st.scale_log2 = a.scale_log2;
  st.init();

  T* kpool = static_cast<T*>(a.k_pages);
  T* vpool = static_cast<T*>(a.v_pages);
  const bool has_new = a.k_new != nullptr;
  const int last = L - 1;
  const int64_t new_row = ((int64_t)b * heads + g) * D;
  // byte offset of this lane's first piece inside a group (consecutive rows)
  const uint32_t lane_off = (uint32_t)((r * D + R::elem(0, j, 0)) * sizeof(T));

  // the wave holding slot L-1 stores the newest token's K/V there
  if (has_new && L > 0 && g_begin * kRows <= last && last < g_end * kRows && r == 0) {
    const int64_t page = page_of(a.table, b, last, a.pv);
    if (page >= 0) {
      const int64_t off = page_row<D>(page, g, last & slot_mask, a.pv);
      R kc, vc;
      kc.load(static_cast<const T*>(a.k_new) + new_row, j);
      vc.load(static_cast<const T*>(a.v_new) + new_row, j);
      kc.store(kpool + off, j);
      vc.store(vpool + off, j);
    }
  }

  // page of group grp (wave-uniform), or -1 when the table entry is bad
  auto group_page = [&](int grp) -> int {
    const int pg = (grp * kRows) >> shift;
    const int idx = pg - first_page;
    const int page = idx < 64 ? __builtin_amdgcn_readlane(tbl, idx) : table[min(pg, a.pv.max_pages - 1)];
    return (page >= 0 && page < a.pv.num_pages) ? page : -1;
  };
  auto group_base = [&](int page, int grp) -> int64_t {
    return ((((int64_t)page * heads + g) << shift) + ((grp * kRows) & slot_mask)) * D;
  };

  // keys [0, Lc) come from the cache; with k_new, key L-1 comes from k_new
  const int Lc = has_new ? max(L - 1, 0) : L;
  // groups wholly inside [0, Lc) take the unmasked path, U at a time
  const int g_full = max(g_begin, min(g_end, Lc / kRows));
  const int nbatch = (g_full - g_begin) / U;

  auto issue_full = [&](int gs, R* kc, R* vc) -> bool {
    bool ok = true;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int page = group_page(gs + u);
      ok = ok && page >= 0;
      const int64_t base = group_base(page >= 0 ? page : 0, gs + u) * (int64_t)sizeof(T);
      kc[u].stream(reinterpret_cast<const char*>(kpool) + base, lane_off);
      vc[u].stream(reinterpret_cast<const char*>(vpool) + base, lane_off);
    }
    return ok;
  };

  R k0[U], v0[U], k1[U], v1[U];
  bool all_ok = true;
  if (nbatch > 0) all_ok = issue_full(g_begin, k0, v0);
  for (int bi = 0; bi < nbatch; bi += 2) {
    const int gs = g_begin + bi * U;
    const bool more = bi + 1 < nbatch;
    if (more) all_ok = issue_full(gs + U, k1, v1) && all_ok;
    st.template consume<U, false>(k0, v0, nullptr);
    if (more) {
      if (bi + 2 < nbatch) all_ok = issue_full(gs + 2 * U, k0, v0) && all_ok;
      st.template consume<U, false>(k1, v1, nullptr);
    }
  }
  // A block-table entry out of range (a caller error) was read as page 0:
  // drop what the unmasked path accumulated rather than mix in that page.
  if (!all_ok) st.init();

  // masked tail: the remaining groups of the range that hold keys < L
  const int g_tail_end = min(g_end, (L + kRows - 1) / kRows);
  for (int gs = g_begin + nbatch * U; gs < g_tail_end; gs += U) {
    R kc[U], vc[U];
    bool valid[U];
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
    st.template consume<U, true>(kc, vc, valid);
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
  // per-head merge weights of the waves, once
  if (tid < G) {
    const int h = tid;
    float M = neg_inf();
#pragma unroll
    for (int w = 0; w < NW; ++w) M = fmaxf(M, s_m[w][h]);
    float den = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const float mw = s_m[w][h];
      const float f = (mw == neg_inf()) ? 0.f : fast_exp2(mw - M);
      s_w[w][h] = f;
      den += f * s_l[w][h];
    }
    s_den[h] = den;
    if (a.num_splits > 1) {
      const int64_t ws = ((int64_t)b * hq + g * G + h) * a.num_splits + split;
      a.ws_ml[ws * 2] = M;
      a.ws_ml[ws * 2 + 1] = den;
    }
  }
  __syncthreads();

  // one thread per (head, element)
  for (int idx = tid; idx < G * D; idx += NW * 64) {
    const int h = idx / D, e = idx % D;
    float num = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) num += s_w[w][h] * s_acc[w][h][e];
    const int64_t row = (int64_t)b * hq + g * G + h;
    if (a.num_splits == 1) {
      const float den = s_den[h];
      const float o = den > 0.f ? num / den : 0.f;
      if (sizeof(T) == 2)
        static_cast<bf16_bits*>(a.out)[row * D + e] = (bf16_bits)f32_to_bf16(o);
      else
        static_cast<float*>(a.out)[row * D + e] = o;
    } else {
      a.ws_o[(row * a.num_splits + split) * D + e] = num;
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

// Waves per block and key groups per load batch (tuning knobs; the split
// heuristic of the host layer assumes 8 waves).
#ifndef SKV_DECODE_WAVES
#define SKV_DECODE_WAVES 8
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
