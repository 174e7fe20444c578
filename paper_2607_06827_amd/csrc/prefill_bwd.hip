// Backward of the attention over the compressed cache (arXiv 2607.06827,
// Sec. III-B, Eq. 5 under the causal mask over compressed positions; Sec.
// III-C: training runs the pooling inside the forward pass and optimises it
// jointly, so the gradient reaches Q, the pooled K^/V^ and, through them, the
// raw K/V and the gate).
//
// With P = softmax(scale Q K^T) under the mask, O = P V and the gradient dO:
//   dP      = dO V^T,   Delta_p = sum_c P_pc dP_pc  (= dO_p . O_p exactly)
//   dZ      = P o (dP - Delta)
//   dQ      = scale dZ K^,   dK^ = scale dZ^T Q,   dV^ = P^T dO
// Delta is formed from P and dP in fp32, not from the stored output: a row
// that sees few keys has dZ = P (dP - Delta) nearly cancelling, and the bf16
// rounding of O would otherwise dominate its dQ.
// P is recomputed from the forward's log-sum-exp, so nothing of size
// queries x keys is stored.  Two kernels, each owning its output so that
// nothing is accumulated across blocks:
//
// dQ kernel - the forward's tiling: a block owns one (sequence, KV head) and
//   32*RB query rows for the G query heads; per 32-key tile
//     S^T = K Q^T,  dP^T = V dO^T          (keys x queries, one query per lane)
//     dQ^T += K^T dZ0^T,  Kbar^T += K^T P^T (K^T read transposed from the K tile)
//   in one pass, with dZ0 = P o (dP - Delta0) for Delta0 = dO . O from the
//   stored output; the exact Delta accumulates beside it, and at the end
//   dQ = scale (dZ0 K^ + (Delta0 - Delta) Kbar), Kbar = P K^.  It saves
//   Delta for:
// dK/dV kernel - a block owns 32 keys per wave (128 keys) of one (sequence,
//   KV head) and walks the (query head, 32-row query tile) pairs that see
//   them; each pair's Q / dO tile is staged once in LDS for all the waves
//   (direct loads, three steps ahead), and each wave computes on its own keys,
//   K and V held in registers
//     S = Q K^T,  dP = dO V^T               (queries x keys, one key per lane)
//     dV^T += dO^T P,  dK^T += Q^T dZ        (dO^T, Q^T read transposed)
//   starting S and dP from -LSE/scale and -Delta of their rows.
// The fp32 kernels below run every product on the 32x32x2 fp32 MFMA.  The
// bf16 kernels (further down) keep this split and these formulas on the
// 16x16x32 bf16 MFMA with smaller per-wave tiles (16 query rows, or 16 keys, a
// wave), so that three waves share each SIMD; P and dZ are rounded to bf16 as
// MFMA operands, every product accumulates in fp32, and dK^ and dV^ are
// written in fp32.
// The mask's visibility rule comes from the span view (spans.hpp): one run
// per sequence, or the runs of a segment table (kRuns).
#include <climits>
#include <type_traits>

#include "attn_mfma.hpp"
#include "kernels.hpp"
#include "kernels_bwd.hpp"

namespace skv {

namespace {

constexpr float kLog2eF = 1.4426950408889634f;

// s_waitcnt immediate that waits until at most n vector-memory operations of
// the wave are outstanding (vmcnt in bits 3:0 and 15:14; expcnt and lgkmcnt
// at their maxima, so they are not waited for)
constexpr int wait_vmcnt(int n) { return 0x0F70 | (n & 15) | ((n >> 4) << 14); }
static_assert(wait_vmcnt(0) == kWaitVmcnt0, "vmcnt(0) encoding");

__device__ __forceinline__ float frag_dot(bf16x8_t x, bf16x8_t y) {
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) s = __builtin_fmaf((float)x[i], (float)y[i], s);
  return s;
}
__device__ __forceinline__ float frag_dot(float x, float y) { return x * y; }

// ------------------------------------------------------------------ dQ

template <typename T, int D, int G, bool kRuns>
__global__ __launch_bounds__(PrefillShape<G>::kThreads) void prefill_bwd_dq_kernel(PrefillBwdArgs a) {
  typedef Mfma<T> M;
  typedef typename M::Frag Frag;
  constexpr int kThreads = PrefillShape<G>::kThreads;
  constexpr int kRows = PrefillShape<G>::kRows;
  constexpr int kKeys = 32;                       // keys per tile
  constexpr int kPack = M::kPack;
  constexpr int kStep = 2 * kPack;                // head-dim elements per MFMA
  constexpr int kQChunks = D / kStep;
  constexpr int kElems16 = 16 / (int)sizeof(T);   // elements per 16-byte chunk
  constexpr int kChunksPerRow = D / kElems16;
  constexpr int kRowK = D + kElems16;             // padded K and V rows (elements)
  constexpr int kItems = kKeys * kChunksPerRow;   // staging work: (key, 16-byte chunk)
  constexpr int kItemsPerThread = (kItems + kThreads - 1) / kThreads;
  constexpr int kTile = kKeys * kRowK;

  __shared__ __attribute__((aligned(16))) T s_buf[2 * 2 * kTile];  // [buffer][K, V]

  // XCD-aware, heaviest-first item order (as in the forward)
  int pair, tile;
  query_tile_item(blockIdx.x, gridDim.x, a.num_q_tiles, pair, tile);
  const int heads = a.pv.kv_heads;
  const int g = pair % heads;
  const int b = pair / heads;

  const auto sp = span_view<kRuns>(a, b, a.w_eff);
  const int rows = min(sp.rows(), a.q_len);
  const int clen = min(sp.clen(), a.pv.max_pages << a.pv.page_shift);
  const int p0 = tile * kRows;
  if (p0 >= rows) return;
  const int kmax = min(sp.visible(min(p0 + kRows, rows) - 1, a.mask_mode), clen);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = g * G + wave % G;
  const int col = lane & 31, hg = lane >> 5;
  const int wrow0 = p0 + (wave / G) * 32;
  const int p = wrow0 + col;
  const bool qvalid = p < rows;
  const int nvis = qvalid ? min(sp.visible(p, a.mask_mode), clen) : 0;
  const int hq = a.num_q_heads;
  const int slot_mask = (1 << a.pv.page_shift) - 1;

  f32x16_t acc[D / 32], kbar[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[db][i] = kbar[db][i] = 0.f;
  float dsum = 0.f;  // sum over this lane's keys of P dP (half of Delta)

  const T* kpool = static_cast<const T*>(a.k_pages);
  const T* vpool = static_cast<const T*>(a.v_pages);
  const int ntiles = (kmax + kKeys - 1) / kKeys;

  // K/V staging: the forward's branch-free pipeline (table entries three tiles
  // ahead, rows two tiles ahead in registers, LDS one tile ahead), both tiles
  // row-major; rows past the visible range are zero.
  const int32_t* table_row = a.table + (int64_t)b * a.pv.max_pages;
  const int64_t num_pages = a.pv.num_pages;
  const int shift = a.pv.page_shift;
  int pg[2][kItemsPerThread];
  uint4 rk[2][kItemsPerThread], rv[2][kItemsPerThread];
  uint32_t okm[2];
  auto item_key = [&](int it) { return (tid + it * kThreads) / kChunksPerRow; };
  auto item_chunk = [&](int it) { return (tid + it * kThreads) % kChunksPerRow; };
  auto table_load = [&](int kt, int* pgs) {
#pragma unroll
    for (int it = 0; it < kItemsPerThread; ++it)
      pgs[it] = table_row[min((kt * kKeys + item_key(it)) >> shift, a.pv.max_pages - 1)];
  };
  auto fetch = [&](int kt, const int* pgs, uint4* rks, uint4* rvs, uint32_t& oks) {
    oks = 0;
#pragma unroll
    for (int it = 0; it < kItemsPerThread; ++it) {
      const int key = kt * kKeys + item_key(it);
      const int page = pgs[it];
      const bool ok = key < kmax && page >= 0 && page < num_pages;
      oks |= ok ? 1u << it : 0u;
      const int64_t off = page_row<D>(ok ? page : 0, g, key & slot_mask, a.pv) + item_chunk(it) * kElems16;
      rks[it] = *reinterpret_cast<const uint4*>(kpool + off);
      rvs[it] = *reinterpret_cast<const uint4*>(vpool + off);
    }
  };
  auto stage = [&](int buf, const uint4* rks, const uint4* rvs, uint32_t oks) {
    T* sk = s_buf + buf * 2 * kTile;
    T* sv = sk + kTile;
#pragma unroll
    for (int it = 0; it < kItemsPerThread; ++it) {
      if (tid + it * kThreads >= kItems) continue;
      const int key = item_key(it), ch = item_chunk(it);
      const uint32_t m = 0u - ((oks >> it) & 1u);
      const uint4 kv = rks[it], vv = rvs[it];
      *reinterpret_cast<uint4*>(&sk[key * kRowK + ch * kElems16]) = make_uint4(kv.x & m, kv.y & m, kv.z & m, kv.w & m);
      *reinterpret_cast<uint4*>(&sv[key * kRowK + ch * kElems16]) = make_uint4(vv.x & m, vv.y & m, vv.z & m, vv.w & m);
    }
  };

  table_load(0, pg[0]);
  table_load(1, pg[1]);
  fetch(0, pg[0], rk[0], rv[0], okm[0]);
  table_load(2, pg[0]);
  fetch(1, pg[1], rk[1], rv[1], okm[1]);
  __builtin_amdgcn_sched_barrier(0);
  // this lane's query, output and output-gradient row (B operands; rows past
  // the end read row 0 of the sequence: finite, never stored)
  Frag qf[kQChunks], gf[kQChunks];
  const int64_t row_off = (((int64_t)b * a.q_len + (qvalid ? p : 0)) * hq + h) * D + hg * kPack;
  const T* qrow = static_cast<const T*>(a.q) + row_off;
  const T* grow = static_cast<const T*>(a.dout) + row_off;
  const T* orow = static_cast<const T*>(a.out) + row_off;
  float delta0 = 0.f;  // dO . O from the stored output: the pivot of dZ0
#pragma unroll
  for (int kc = 0; kc < kQChunks; ++kc) {
    qf[kc] = M::load(qrow + kc * kStep);
    gf[kc] = M::load(grow + kc * kStep);
    delta0 += frag_dot(gf[kc], M::load(orow + kc * kStep));
  }
  const int64_t stat = ((int64_t)b * hq + h) * a.q_len + (qvalid ? p : 0);
  const float lse2 = a.lse[stat] * kLog2eF;
  __builtin_amdgcn_sched_barrier(0);
  stage(0, rk[0], rv[0], okm[0]);
  __syncthreads();
  __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
  delta0 = partner_sum(delta0);  // the partner lane holds the other half of the row

  auto tile_step = [&](int kt, auto par) {
    constexpr int kPar = decltype(par)::value;
    constexpr int kOther = 1 - kPar;
    table_load(kt + 3, pg[kOther]);
    fetch(kt + 2, pg[kPar], rk[kPar], rv[kPar], okm[kPar]);
    const int kb = kt * kKeys;
    const T* sk = s_buf + kPar * 2 * kTile;
    const T* sv = sk + kTile;
    if (kt < ntiles) {
      // S^T and dP^T: row = key (8*(i/4) + 4*hg + i%4), column = this lane's query
      f32x16_t st, dpt;
#pragma unroll
      for (int i = 0; i < 16; ++i) st[i] = dpt[i] = 0.f;
      const T* krow = &sk[col * kRowK + hg * kPack];
      const T* vrow = &sv[col * kRowK + hg * kPack];
#pragma unroll
      for (int kc = 0; kc < kQChunks; ++kc) {
        st = M::mma(M::load(krow + kc * kStep), qf[kc], st);
        dpt = M::mma(M::load(vrow + kc * kStep), gf[kc], dpt);
      }
      float pr[16], dz[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int key = kb + 8 * (i / 4) + 4 * hg + (i % 4);
        const float e = fast_exp2(__builtin_fmaf(st[i], a.scale_log2, -lse2));
        pr[i] = key < nvis ? e : 0.f;
        dz[i] = pr[i] * (dpt[i] - delta0);
        dsum = __builtin_fmaf(pr[i], dpt[i], dsum);
      }
      // dQ^T += K^T dZ0^T and Kbar^T += K^T P^T over the 32 keys of the tile
#pragma unroll
      for (int kk = 0; kk < kKeys / kStep; ++kk) {
        const Frag zf = M::pack_p(dz + kk * kPack);
        const Frag pf = M::pack_p(pr + kk * kPack);
#pragma unroll
        for (int db = 0; db < D / 32; ++db) {
          const Frag kt = M::template load_v<kRowK>(sk, kk, db, lane);
          acc[db] = M::mma(kt, zf, acc[db]);
          kbar[db] = M::mma(kt, pf, kbar[db]);
        }
      }
    }
    stage(kOther, rk[kOther], rv[kOther], okm[kOther]);
    __syncthreads();
  };
  for (int kt = 0; kt < ntiles; kt += 2) {
    tile_step(kt, std::integral_constant<int, 0>());
    tile_step(kt + 1, std::integral_constant<int, 1>());
  }

  const float delta = partner_sum(dsum);  // sum over all the row's keys of P dP
  if (!qvalid) return;
  if (hg == 0) a.delta[stat] = delta;
  T* drow = static_cast<T*>(a.dq) + (((int64_t)b * a.q_len + p) * hq + h) * D;
  const float sc = a.scale, fix = delta0 - delta;
  auto dq_at = [&](int db, int i) { return sc * __builtin_fmaf(fix, kbar[db][i], acc[db][i]); };
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int ig = 0; ig < 4; ++ig)
      M::store4(drow + db * 32 + 8 * ig + 4 * hg, dq_at(db, 4 * ig), dq_at(db, 4 * ig + 1),
                dq_at(db, 4 * ig + 2), dq_at(db, 4 * ig + 3));
}

// --------------------------------------------------------------- dK / dV

// Q / dO tiles of the dK/dV kernel: 32 unpadded rows in LDS, filled by
// direct loads (global_load_lds: a wave-wide load writes 64 x 16 bytes in
// lane order), 16-byte chunks XOR-swizzled within a row: chunk c of row r sits
// at position c ^ swz(r), so the operand reads of 16 rows at one chunk hit
// distinct banks.
template <typename T, int D>
struct QTile {
  static constexpr int kElems16 = 16 / (int)sizeof(T);
  static constexpr int kChunks = D / kElems16;              // 16-byte chunks per row
  static constexpr int kRowsPerLoad = 64 / kChunks;         // rows per wave-wide load
  static constexpr int kLoads = 32 / kRowsPerLoad;          // wave-wide loads per tile
  static constexpr int kElems = 32 * D;
  // XOR swizzle of the 16-byte chunks of row r.  With 16 chunks per row
  // (bf16, D = 128: a row spans the 64 banks once) the tile is read both
  // row-wise (16x16x32 A operands: 16 consecutive rows at one chunk per 16
  // lanes) and transposed (ds_read_b64_tr_b16: 8 consecutive rows x 2
  // neighbouring chunks per 32 lanes).  ((r & 7) << 1) | ((r >> 3) & 1) is a
  // permutation of 16 consecutive rows (the row-wise reads hit 16 distinct
  // chunk positions) whose bits 1-3 differ over 8 consecutive rows (the
  // transposed reads hit 16 distinct positions).  (The 32x32 layout's
  // ((r & 3) << 2) | ((r >> 2) & 3) gives rows r and r + 4 the same pair of
  // positions in the transposed reads: a 2-way bank conflict on each.)
  static __device__ __forceinline__ int swz(int r) {
    if constexpr (kChunks == 16) return ((r & 7) << 1) | ((r >> 3) & 1);
    return r & (kChunks >= 16 ? 15 : kChunks - 1);
  }
  // element e of row r
  static __device__ __forceinline__ int at(int r, int e) {
    return r * D + (((e / kElems16) ^ swz(r)) * kElems16) + (e % kElems16);
  }
};

// A operand (kPack elements from element e) of row r of a swizzled tile
__device__ __forceinline__ bf16x8_t tile_a(const bf16_bits* t, int off) {
  return __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u16x8_t*>(t + off));
}
__device__ __forceinline__ float tile_a(const float* t, int off) { return t[off]; }

// Transposed A operand of a swizzled 32-row tile: what Mfma<T>::load_v
// returns for a padded row-major tile (rows 16kk + 4(g/2) + j/4 (+8) for
// bf16, row 8(kk/4) + 4hg + kk%4 for fp32; columns of head-dim block db).
template <int D>
__device__ __forceinline__ bf16x8_t tile_t(const bf16_bits* t, int kk, int db, int lane) {
  typedef QTile<bf16_bits, D> Q;
  const int g = lane >> 4, j = lane & 15;
  const int r = 16 * kk + 4 * (g >> 1) + (j >> 2);
  const int e = 32 * db + 16 * (g & 1) + 4 * (j & 3);
  const s16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_ptr)(t + Q::at(r, e)));
  const s16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_ptr)(t + Q::at(r + 8, e)));
  const u16x8_t v = {(unsigned short)lo[0], (unsigned short)lo[1], (unsigned short)lo[2], (unsigned short)lo[3],
                     (unsigned short)hi[0], (unsigned short)hi[1], (unsigned short)hi[2], (unsigned short)hi[3]};
  return __builtin_bit_cast(bf16x8_t, v);
}
template <int D>
__device__ __forceinline__ float tile_t(const float* t, int kk, int db, int lane) {
  typedef QTile<float, D> Q;
  return t[Q::at(8 * (kk / 4) + 4 * (lane >> 5) + (kk % 4), 32 * db + (lane & 31))];
}

template <typename T, int D>
struct KvBwdShape {
  // fp32 at d = 128 has twice the bytes per tile: two waves keep LDS in bounds
  static constexpr int kWaves = (sizeof(T) == 4 && D == 128) ? 2 : 4;
  static constexpr int kThreads = 64 * kWaves;
  static constexpr int kKeys = 32 * kWaves;  // keys per block, 32 per wave
};

// Item of block bid in a dK/dV grid of nblk blocks over pairs x T key blocks
// (items pair-major, pair = (sequence, KV head)).  The work of key block kt
// falls with kt (later keys are seen by fewer query rows).  XCD x (= bid mod
// 8) runs a contiguous item range; its blocks fill its 32 CUs one round at
// a time, so local blocks i, i + 32, ... share a CU while they are resident
// together.  A pair whose first item opens an odd round of its XCD takes its
// key blocks in descending order, which pairs the heavy blocks of one round
// with the light ones of the next on each CU (at 1596 x 471, b = 8: 12%
// less time than ascending order everywhere).  The order is reversed within
// whole pairs, so every item is still run exactly once.
constexpr int kCusPerXcd = 32;
__device__ __forceinline__ void dkdv_item(int bid, int nblk, int T, int& pair, int& kt) {
  const int xcd = bid & 7, per = nblk >> 3, rem = nblk & 7;
  const int item = xcd * per + min(xcd, rem) + (bid >> 3);
  pair = item / T;
  const int kt0 = item - pair * T;
  // the XCD range holding the pair's first item, and that item's place in it
  const int first = pair * T;
  const int x = first < rem * (per + 1) ? first / (per + 1) : rem + (first - rem * (per + 1)) / max(per, 1);
  const int local = first - (x * per + min(x, rem));
  kt = ((local / kCusPerXcd) & 1) ? T - 1 - kt0 : kt0;
}

template <typename T, int D, int G, bool kRuns>
__global__ __launch_bounds__((KvBwdShape<T, D>::kThreads)) void prefill_bwd_dkdv_kernel(PrefillBwdArgs a) {
  typedef Mfma<T> M;
  typedef typename M::Frag Frag;
  typedef QTile<T, D> Q;
  constexpr int kWaves = KvBwdShape<T, D>::kWaves;
  constexpr int kBlockKeys = KvBwdShape<T, D>::kKeys;
  constexpr int kQ = 32;      // query rows per step
  constexpr int kPack = M::kPack;
  constexpr int kStep = 2 * kPack;
  constexpr int kQChunks = D / kStep;
  constexpr int kElems16 = Q::kElems16;

  // the shared Q / dO tile (with LSE and Delta) of kBufs steps, each buffer
  // its own array so that the compiler sees that direct loads in flight never
  // touch the buffer being read
  struct Buf {
    T q[Q::kElems];
    T g[Q::kElems];
    float l[2 * kQ];  // LSE, Delta
  };
  constexpr int kBufs = 4 * (int)sizeof(Buf) <= 160 * 1024 ? 4 : 2;
  typedef std::conditional_t<(kBufs > 2), Buf, char> Buf23;  // (unused with two buffers)
  __shared__ __attribute__((aligned(16))) Buf s_b0;
  __shared__ __attribute__((aligned(16))) Buf s_b1;
  __shared__ __attribute__((aligned(16))) Buf23 s_b2;
  __shared__ __attribute__((aligned(16))) Buf23 s_b3;
  auto buf = [&](auto n) -> auto& {
    constexpr int kN = decltype(n)::value % kBufs;
    if constexpr (kN == 0) return s_b0;
    else if constexpr (kN == 1) return s_b1;
    else if constexpr (kN == 2) return s_b2;
    else return s_b3;
  };

  int pair, kt;
  dkdv_item(blockIdx.x, gridDim.x, a.num_key_tiles, pair, kt);
  const int heads = a.pv.kv_heads;
  const int g = pair % heads;
  const int b = pair / heads;

  const auto sp = span_view<kRuns>(a, b, a.w_eff);
  const int rows = min(sp.rows(), a.q_len);
  const int clen = min(min(sp.clen(), a.pv.max_pages << a.pv.page_shift), a.hat_cap);
  const int kb0 = kt * kBlockKeys;
  if (kb0 >= clen) return;  // block-uniform

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int col = lane & 31, hg = lane >> 5;
  const int hq = a.num_q_heads;
  const int kb = kb0 + 32 * wave;  // this wave's keys
  const int key = kb + col;       // this lane's key (C-layout column)
  const int tau = key < clen ? sp.visible_from(key, a.mask_mode) : INT_MAX;
  // first row that sees a key of this wave (none: INT_MAX)
  const int wave_from = kb < clen ? sp.visible_from(kb, a.mask_mode) : INT_MAX;

  // this lane's K and V rows, the B operands of S = Q K^T and dP = dO V^T,
  // in registers for every step (a key past the compressed length or without
  // a page reads page 0 and is zeroed)
  Frag kf[kQChunks], vf[kQChunks];
  {
    const int shift = a.pv.page_shift;
    const int32_t page = a.table[(int64_t)b * a.pv.max_pages + min(key >> shift, a.pv.max_pages - 1)];
    const bool ok = key < clen && page >= 0 && page < a.pv.num_pages;
    const int64_t off = page_row<D>(ok ? page : 0, g, key & ((1 << shift) - 1), a.pv) + hg * kPack;
#pragma unroll
    for (int kc = 0; kc < kQChunks; ++kc) {
      const Frag k = M::load(static_cast<const T*>(a.k_pages) + off + kc * kStep);
      const Frag v = M::load(static_cast<const T*>(a.v_pages) + off + kc * kStep);
      kf[kc] = ok ? k : M::zero();
      vf[kc] = ok ? v : M::zero();
    }
  }

  // query rows that see some key of the block: from tau(kb0) (tau grows with
  // c); one step per (query head, 32-row tile) pair
  const int q_first = sp.visible_from(kb0, a.mask_mode);
  const int t0 = q_first / kQ, t1 = (rows + kQ - 1) / kQ;
  const int n_steps = max(t1 - t0, 0) * G;

  // step it into a buffer by direct loads, the block's wave-wide loads dealt
  // round the waves: Q and dO rows, then LSE (lanes 0-31) and Delta (32-63).
  // Rows past the end load row 0: finite, never visible.
  const int lrow = lane / Q::kChunks, lpos = lane % Q::kChunks;
  auto load_step = [&](int it, Buf& bf) __attribute__((always_inline)) {
    const int h = g * G + it % G;
    const int q0 = (t0 + it / G) * kQ;
#pragma unroll
    for (int l0 = 0; l0 < Q::kLoads; l0 += kWaves) {
      const int l = l0 + wave;
      if (Q::kLoads % kWaves != 0 && l >= Q::kLoads) break;
      const int r = l * Q::kRowsPerLoad + lrow;
      const int pr = q0 + r < rows ? q0 + r : 0;
      const int64_t off = (((int64_t)b * a.q_len + pr) * hq + h) * D + (lpos ^ Q::swz(r)) * kElems16;
      __builtin_amdgcn_global_load_lds((global_void_ptr)(static_cast<const T*>(a.q) + off),
                                       (lds_void_ptr)(bf.q + l * Q::kRowsPerLoad * D), 16, 0, 0);
      __builtin_amdgcn_global_load_lds((global_void_ptr)(static_cast<const T*>(a.dout) + off),
                                       (lds_void_ptr)(bf.g + l * Q::kRowsPerLoad * D), 16, 0, 0);
    }
    if (wave == kWaves - 1) {
      const int pr = q0 + col < rows ? q0 + col : 0;
      const int64_t stat = ((int64_t)b * hq + h) * a.q_len + pr;
      __builtin_amdgcn_global_load_lds((global_void_ptr)(hg ? a.delta + stat : a.lse + stat),
                                       (lds_void_ptr)bf.l, 4, 0, 0);
    }
  };

  f32x16_t dk[D / 32], dv[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) dk[db][i] = dv[db][i] = 0.f;

  // loads per wave and step: its share of the Q and dO loads (the last wave
  // also loads LSE / Delta)
  constexpr int kMine = 2 * ((Q::kLoads + kWaves - 1) / kWaves);
  // step n from buffer kPar while the next kBufs - 1 steps load into the others
  auto step = [&](int n, auto par) __attribute__((always_inline)) {
    constexpr int kPar = decltype(par)::value;
    const Buf& bf = buf(par);
    const T* sq = bf.q;
    const T* sg = bf.g;
    const float* sl = bf.l;
    // this buffer's loads (issued kBufs - 1 steps ago by every wave) have
    // landed: only the loads of the later steps may remain in flight, kMine
    // per step (the LSE / Delta load is not counted, so that wave waits a
    // little longer than it must); then every wave is done with the buffer
    // the next load refills
    const int later = min(n_steps - 1 - n, kBufs - 2);
    if (later >= 2) __builtin_amdgcn_s_waitcnt(wait_vmcnt(2 * kMine));
    else if (later == 1) __builtin_amdgcn_s_waitcnt(wait_vmcnt(kMine));
    else __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    __syncthreads();
    if (n + kBufs - 1 < n_steps) load_step(n + kBufs - 1, buf(std::integral_constant<int, kPar + kBufs - 1>()));
    const int q0 = (t0 + n / G) * kQ;
    if (q0 + kQ <= wave_from) return;  // no row of the tile sees a key of this wave

    // S - LSE/scale and dP - Delta: row = query (8*(i/4) + 4*hg + i%4), column
    // = this lane's key.  The accumulators start from -LSE/scale and -Delta
    // of their rows (four consecutive rows at a time), so that P = exp(scale
    // S - LSE) and dZ = P (dP - Delta) need nothing more per row.
    f32x16_t s, dp;
    const float neg_inv_scale = -1.f / a.scale;
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
      const float4 lv = *reinterpret_cast<const float4*>(sl + 8 * q4 + 4 * hg);
      const float4 dv4 = *reinterpret_cast<const float4*>(sl + kQ + 8 * q4 + 4 * hg);
      s[4 * q4] = lv.x * neg_inv_scale; s[4 * q4 + 1] = lv.y * neg_inv_scale;
      s[4 * q4 + 2] = lv.z * neg_inv_scale; s[4 * q4 + 3] = lv.w * neg_inv_scale;
      dp[4 * q4] = -dv4.x; dp[4 * q4 + 1] = -dv4.y; dp[4 * q4 + 2] = -dv4.z; dp[4 * q4 + 3] = -dv4.w;
    }
#pragma unroll
    for (int kc = 0; kc < kQChunks; ++kc) {
      const int e = hg * kPack + kc * kStep;
      s = M::mma(tile_a(sq, Q::at(col, e)), kf[kc], s);
      dp = M::mma(tile_a(sg, Q::at(col, e)), vf[kc], dp);
    }
    float pr[16], dz[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int r = 8 * (i / 4) + 4 * hg + (i % 4);
      const bool vis = q0 + r >= tau && q0 + r < rows;
      const float e = fast_exp2(s[i] * a.scale_log2);
      pr[i] = vis ? e : 0.f;
      dz[i] = vis ? e * dp[i] : 0.f;
    }
    // dV^T += dO^T P and dK^T += Q^T dZ over the 32 query rows (the row order
    // of the C layout carried into the transposed reads)
#pragma unroll
    for (int kk = 0; kk < kQ / kStep; ++kk) {
      const Frag pf = M::pack_p(pr + kk * kPack);
      const Frag zf = M::pack_p(dz + kk * kPack);
#pragma unroll
      for (int db = 0; db < D / 32; ++db) {
        dv[db] = M::mma(tile_t<D>(sg, kk, db, lane), pf, dv[db]);
        dk[db] = M::mma(tile_t<D>(sq, kk, db, lane), zf, dk[db]);
      }
    }
  };

  // the first kBufs - 1 steps, then steps in groups of kBufs (compile-time buffers)
  if (n_steps > 0) load_step(0, buf(std::integral_constant<int, 0>()));
  if constexpr (kBufs == 4) {
    if (n_steps > 1) load_step(1, buf(std::integral_constant<int, 1>()));
    if (n_steps > 2) load_step(2, buf(std::integral_constant<int, 2>()));
  }
  for (int n = 0; n < n_steps; n += kBufs) {
    step(n, std::integral_constant<int, 0>());
    if (n + 1 < n_steps) step(n + 1, std::integral_constant<int, 1>());
    if constexpr (kBufs == 4) {
      if (n + 2 < n_steps) step(n + 2, std::integral_constant<int, 2>());
      if (n + 3 < n_steps) step(n + 3, std::integral_constant<int, 3>());
    }
  }

  // this lane's key: d = 32 db + 8 (i/4) + 4 hg + i%4, four consecutive at a time
  if (key >= clen) return;
  float* dkrow = a.dk_hat + (((int64_t)b * a.hat_cap + key) * heads + g) * D + 4 * hg;
  float* dvrow = a.dv_hat + (((int64_t)b * a.hat_cap + key) * heads + g) * D + 4 * hg;
  const float sc = a.scale;
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int ig = 0; ig < 4; ++ig) {
      *reinterpret_cast<float4*>(dkrow + 32 * db + 8 * ig) =
          make_float4(dk[db][4 * ig] * sc, dk[db][4 * ig + 1] * sc, dk[db][4 * ig + 2] * sc, dk[db][4 * ig + 3] * sc);
      *reinterpret_cast<float4*>(dvrow + 32 * db + 8 * ig) =
          make_float4(dv[db][4 * ig], dv[db][4 * ig + 1], dv[db][4 * ig + 2], dv[db][4 * ig + 3]);
    }
}

// ---------------------------------------------------- dQ, bf16, 16 rows a wave
//
// The bf16 dQ kernel on the 16x16x32 MFMA.  A wave owns 16 query rows of one
// query head and keeps their Q and dO operands in registers; a block of
// kWaves waves owns 16 * kWaves / G rows of one (sequence, KV head) for all G
// heads and streams the 32-key tiles they see through LDS (three buffers,
// untracked direct loads two tiles ahead, as in the forward).  Per tile a
// wave computes, keys as rows of the 16x16 blocks (so that P and dZ0 are
// their own B operands, as in the dK/dV kernel):
//   S^T = K Q^T,  dP^T = V dO^T       (two 16-key blocks)
//   P = exp2(scale log2e S - log2e LSE),  dZ0 = P (dP - Delta0)
//   dQ^T += K^T dZ0^T,  Kbar^T += K^T P^T    (16-row blocks of d)
// with Delta0 = dO . O (the stored output) and the exact Delta = sum P dP
// beside it; at the end dQ = scale (dZ0 K + (Delta0 - Delta) Kbar).
template <int G>
struct DqShape16 {
  static constexpr int kRowBlocks = G >= 4 ? 1 : 4 / G;
  static constexpr int kWaves = G * kRowBlocks;
  static constexpr int kThreads = 64 * kWaves;
  static constexpr int kRows = 16 * kRowBlocks;
};

template <int D, int G, bool kRuns>
__global__ __launch_bounds__(DqShape16<G>::kThreads, 3) void prefill_bwd_dq16_kernel(PrefillBwdArgs a) {
  typedef bf16_bits T;
  typedef QTile<T, D> Q;  // the K and V tiles: 32 rows, chunks swizzled per row
  typedef bf16x8_t Frag;
  typedef float f32x4 __attribute__((ext_vector_type(4)));
  constexpr int kWaves = DqShape16<G>::kWaves;
  constexpr int kRows = DqShape16<G>::kRows;
  constexpr int kKeys = 32;
  constexpr int kDC = D / 32;  // K-dim chunks of S^T and dP^T
  constexpr int kDB = D / 16;  // 16-row blocks of dQ^T and Kbar^T
  constexpr int kLoadsPerWave = Q::kLoads >= kWaves ? Q::kLoads / kWaves : 1;
  static_assert(Q::kLoads % kWaves == 0 || kWaves % Q::kLoads == 0, "loads split evenly over waves");
  constexpr int kVm = 2 * kLoadsPerWave;

  __shared__ __attribute__((aligned(256))) T s_k0[Q::kElems];
  __shared__ __attribute__((aligned(256))) T s_k1[Q::kElems];
  __shared__ __attribute__((aligned(256))) T s_k2[Q::kElems];
  __shared__ __attribute__((aligned(256))) T s_v0[Q::kElems];
  __shared__ __attribute__((aligned(256))) T s_v1[Q::kElems];
  __shared__ __attribute__((aligned(256))) T s_v2[Q::kElems];

  // XCD-aware, heaviest-first item order (as in the forward)
  int pair, tile;
  query_tile_item(blockIdx.x, gridDim.x, a.num_q_tiles, pair, tile);
  const int heads = a.pv.kv_heads;
  const int g = pair % heads;
  const int b = pair / heads;
  const int p0 = tile * kRows;

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int gq = lane >> 4, j = lane & 15;
  const int h = g * G + wave % G;
  const int wrow0 = p0 + (wave / G) * 16;  // first row of this wave
  const int q = wrow0 + j;                 // this lane's row (column of the C layout)
  const int hq = a.num_q_heads;

  // this lane's row of Q, dO and O (elements 32c + 8gq .. +7, the B operand
  // layout of S^T = K Q^T) and its LSE: the rows do not depend on the span
  // lengths, so with one run they are requested first and are in flight
  // during the span and block-table round trips (a row past the tensor reads
  // its last row: in range, never stored); a segment table's scan comes
  // first (its tracked loads' waits would take these along)
  Frag qf[kDC], gf[kDC], of[kDC];
  float lse = 0.f;
  auto load_rows = [&]() __attribute__((always_inline)) {
    const int qr = min(q, a.q_len - 1);
    const int64_t row = ((int64_t)b * a.q_len + qr) * hq + h;
    const T* qp = static_cast<const T*>(a.q) + row * D + 8 * gq;
    const T* gp = static_cast<const T*>(a.dout) + row * D + 8 * gq;
    const T* op = static_cast<const T*>(a.out) + row * D + 8 * gq;
    static_for<kDC>([&](auto c) {
      constexpr int kC = decltype(c)::value;
      untracked_load16<kC * 64>(qf[kC], qp);
      untracked_load16<kC * 64>(gf[kC], gp);
      untracked_load16<kC * 64>(of[kC], op);
    });
    const float* lp = a.lse + ((int64_t)b * hq + h) * a.q_len + qr;
    asm volatile("global_load_dword %0, %1, off" : "=v"(lse) : "v"(lp) : "memory");
    __builtin_amdgcn_sched_barrier(0);
  };
  if constexpr (!kRuns) load_rows();

  const auto sp = span_view<kRuns>(a, b, a.w_eff);
  const int rows = min(sp.rows(), a.q_len);
  const int clen = min(sp.clen(), a.pv.max_pages << a.pv.page_shift);
  if (p0 >= rows) {
    // the row loads land before the wave ends (with one run they were
    // issued above; an asm statement ahead of a segment scan would turn its
    // scalar loads into vector loads)
    if constexpr (!kRuns) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    return;
  }
  const int kmax = min(sp.visible(min(p0 + kRows, rows) - 1, a.mask_mode), clen);
  const int kclamp = max(kmax - 1, 0);  // last visible key: the row loaded for keys past kmax

  const bool qvalid = q < rows;
  const int nvis = qvalid ? min(sp.visible(q, a.mask_mode), clen) : 0;
  const int nvis_lo = wrow0 < rows ? min(sp.visible(wrow0, a.mask_mode), clen) : 0;
  const int shift = a.pv.page_shift, slot_mask = (1 << shift) - 1;
  const int32_t* table_row = a.table + (int64_t)b * a.pv.max_pages;
  const int ntiles = (kmax + kKeys - 1) / kKeys;
  const bool loads = Q::kLoads >= kWaves || wave < Q::kLoads;
  auto load_row0 = [&](int i) { return (Q::kLoads >= kWaves ? wave * kLoadsPerWave + i : wave) * Q::kRowsPerLoad; };
  const int lrow = lane / Q::kChunks, lpos = lane % Q::kChunks;
  if constexpr (kRuns) load_rows();  // after every segment scan

  // block-table entries: one per wave and tile (the forward's scheme)
  constexpr int kWaveRows = kLoadsPerWave * Q::kRowsPerLoad;
  static_assert(kWaveRows <= 8, "one page holds a wave's rows of a tile");
  const int wrow_load = loads ? load_row0(0) : 0;
  typedef __attribute__((address_space(4))) const int32_t* const_ptr;
  auto table_load = [&](int kt) __attribute__((always_inline)) {
    const int row0 = min(kt * kKeys + wrow_load, kclamp);
    return ((const_ptr)table_row)[min(row0 >> shift, a.pv.max_pages - 1)];
  };
  const uint64_t head_bytes = (uint64_t)D * sizeof(T) << shift;
  const uint64_t page_bytes = head_bytes * heads;
  const uintptr_t kpool_g = (uintptr_t)a.k_pages + (uint64_t)g * head_bytes;
  const uintptr_t v_minus_k = (uintptr_t)a.v_pages - (uintptr_t)a.k_pages;
  const uint32_t npages = (uint32_t)a.pv.num_pages;
  auto tile_load = [&](int kt, int e, T* sk, T* sv) __attribute__((always_inline)) {
    if (!loads) return;
    const uint32_t page = (uint32_t)e < npages ? (uint32_t)e : 0u;  // a bad entry reads an in-range page
    const uintptr_t kbase = kpool_g + (uint64_t)page * page_bytes;
    const uintptr_t vbase = kbase + v_minus_k;
#pragma unroll
    for (int i = 0; i < kLoadsPerWave; ++i) {
      const int r = load_row0(i) + lrow;
      const int key = min(kt * kKeys + r, kclamp);
      const uint32_t off = (uint32_t)((key & slot_mask) * D * 2) + ((lpos ^ Q::swz(r)) << 4);
      lds_dma16((const void*)kbase, off, lds_addr(sk + load_row0(i) * D));
      lds_dma16((const void*)vbase, off, lds_addr(sv + load_row0(i) * D));
    }
  };

  f32x4 dq[kDB], kbar[kDB];
#pragma unroll
  for (int db = 0; db < kDB; ++db)
#pragma unroll
    for (int i = 0; i < 4; ++i) dq[db][i] = kbar[db][i] = 0.f;
  float dsum = 0.f;  // this lane's share of Delta = sum over keys of P dP

  // prologue: the row operands (issued above), tiles 0 and 1; wait for the
  // operands and tile 0
  int pg[3] = {table_load(0), table_load(1), table_load(2)};
  tile_load(0, pg[0], s_k0, s_v0);
  if (ntiles > 1 && loads) {
    tile_load(1, pg[1], s_k1, s_v1);
    bare_barrier<kVm>();
  } else {
    // (a wave that loads no tile rows has only its row operands in flight:
    // it waits for all of them)
    bare_barrier<0>();
  }
  // Delta0 = dO . O over the row: the lane's 32 products, then the four lane
  // groups that share the row
  float delta0 = 0.f;
#pragma unroll
  for (int c = 0; c < kDC; ++c) delta0 += frag_dot(gf[c], of[c]);
  delta0 += __shfl_xor(delta0, 16, 64);
  delta0 += __shfl_xor(delta0, 32, 64);
  const float lse2 = lse * kLog2eF;

  // fragment addresses (bytes), one register per tile and pattern, as in the
  // dK/dV kernel: row-wise operands of S^T / dP^T at ar ^ 64c (+16 rows for
  // the second key block), transposed K^T operands at at ^ 32db (+16 rows)
  const int rr = 4 * gq + (j >> 2);
  const uint32_t ar_off = (uint32_t)(j * D * 2 + ((gq ^ Q::swz(j)) << 4));
  const uint32_t at_off = (uint32_t)(rr * D * 2 + ((((j & 3) >> 1) ^ Q::swz(rr)) << 4) + ((j & 1) << 3));
  typedef __attribute__((address_space(3))) const u16x8_t* lds_frag_ptr;

  auto attend = [&](int kt, const T* sk, const T* sv) __attribute__((always_inline)) {
    uint32_t ar_k = lds_addr(sk) + ar_off, ar_v = lds_addr(sv) + ar_off, at_k = lds_addr(sk) + at_off;
    asm volatile("" : "+v"(ar_k), "+v"(ar_v), "+v"(at_k));
    auto arow = [&](uint32_t base, int blk, int c) __attribute__((always_inline)) {
      return __builtin_bit_cast(Frag, *(lds_frag_ptr)(uintptr_t)((base ^ (uint32_t)(64 * c)) + (uint32_t)(blk * 16 * D * 2)));
    };
    auto atr = [&](int db) __attribute__((always_inline)) {
      const uint32_t al = at_k ^ (uint32_t)(32 * db);
      const s16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_ptr)(uintptr_t)al);
      const s16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_ptr)(uintptr_t)(al + 16 * D * 2));
      const u16x8_t v = {(unsigned short)lo[0], (unsigned short)lo[1], (unsigned short)lo[2], (unsigned short)lo[3],
                         (unsigned short)hi[0], (unsigned short)hi[1], (unsigned short)hi[2], (unsigned short)hi[3]};
      return __builtin_bit_cast(Frag, v);
    };
    // S^T and dP^T: rows = keys 16 blk + 4 gq + i of the tile, column = row q
    f32x4 s[2], dp[2];
#pragma unroll
    for (int blk = 0; blk < 2; ++blk)
#pragma unroll
      for (int i = 0; i < 4; ++i) s[blk][i] = dp[blk][i] = 0.f;
    constexpr int kNS = 4 * kDC;  // (c, blk, S or dP)
    auto aop = [&](int idx) __attribute__((always_inline)) {
      const int c = idx / 4, blk = (idx / 2) % 2, t = idx % 2;
      return arow(t ? ar_v : ar_k, blk, c);
    };
    constexpr int kAheadS = 3;
    Frag sb[kAheadS];
#pragma unroll
    for (int i = 0; i < kAheadS; ++i) sb[i] = aop(i);
#pragma unroll
    for (int idx = 0; idx < kNS; ++idx) {
      const Frag cur = sb[idx % kAheadS];
      if (idx + kAheadS < kNS) sb[idx % kAheadS] = aop(idx + kAheadS);
      const int c = idx / 4, blk = (idx / 2) % 2;
      if (idx % 2 == 0) s[blk] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(cur, qf[c], s[blk], 0, 0, 0);
      else dp[blk] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(cur, gf[c], dp[blk], 0, 0, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x100, kAheadS, 0);
#pragma unroll
    for (int idx = 0; idx + kAheadS < kNS; ++idx) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, kAheadS, 0);

    constexpr int kAheadT = 2;
    Frag tb[kAheadT];
#pragma unroll
    for (int i = 0; i < kAheadT; ++i) tb[i] = atr(i);
    __builtin_amdgcn_sched_barrier(0);

    // P and dZ0 in the order of the B operand (element t: key 4gq + t, t < 4,
    // or 16 + 4gq + t - 4); keys past the row's bound get weight 0
    float pv[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) pv[t] = fast_exp2(__builtin_fmaf(s[t / 4][t % 4], a.scale_log2, -lse2));
    const int kb = kt * kKeys;
    if (kb + kKeys > nvis_lo) {  // uniform: the tile straddles some row's bound
      const int lim = nvis - kb - 4 * gq;  // element t is visible iff 16 (t/4) + t%4 < lim
#pragma unroll
      for (int t = 0; t < 8; ++t) pv[t] = 16 * (t / 4) + t % 4 < lim ? pv[t] : 0.f;
    }
    Frag pf, zf;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const float d = dp[t / 4][t % 4];
      dsum = __builtin_fmaf(pv[t], d, dsum);
      pf[t] = (__bf16)pv[t];
      zf[t] = (__bf16)(pv[t] * (d - delta0));
    }
    // dQ^T += K^T dZ0^T and Kbar^T += K^T P^T, one transposed K operand each
#pragma unroll
    for (int db = 0; db < kDB; ++db) {
      const Frag cur = tb[db % kAheadT];
      if (db + kAheadT < kDB) tb[db % kAheadT] = atr(db + kAheadT);
      dq[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(cur, zf, dq[db], 0, 0, 0);
      kbar[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(cur, pf, kbar[db], 0, 0, 0);
    }
#pragma unroll
    for (int db = 0; db + kAheadT < kDB; ++db) {
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 1);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 1);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 2 * kAheadT, 1);
  };

  auto tile_step = [&](int kt, auto par) {
    constexpr int kPar = decltype(par)::value;
    constexpr int kNext2 = (kPar + 2) % 3;
    T* const sk = kPar == 0 ? s_k0 : kPar == 1 ? s_k1 : s_k2;
    T* const sv = kPar == 0 ? s_v0 : kPar == 1 ? s_v1 : s_v2;
    const bool more = kt + 2 < ntiles;  // uniform
    if (more) {
      tile_load(kt + 2, pg[kNext2], kNext2 == 0 ? s_k0 : kNext2 == 1 ? s_k1 : s_k2,
                kNext2 == 0 ? s_v0 : kNext2 == 1 ? s_v1 : s_v2);
      if (kt + 3 < ntiles) pg[kPar] = table_load(kt + 3);
    }
    attend(kt, sk, sv);
    if (more) bare_barrier<kVm>();
    else bare_barrier<0>();
  };
  for (int kt = 0; kt < ntiles; kt += 3) {
    tile_step(kt, std::integral_constant<int, 0>());
    if (kt + 1 >= ntiles) break;
    tile_step(kt + 1, std::integral_constant<int, 1>());
    if (kt + 2 >= ntiles) break;
    tile_step(kt + 2, std::integral_constant<int, 2>());
  }

  // Delta over the whole row, then dQ = scale (dZ0 K + (Delta0 - Delta) Kbar)
  float delta = dsum;
  delta += __shfl_xor(delta, 16, 64);
  delta += __shfl_xor(delta, 32, 64);
  const int64_t stat = ((int64_t)b * hq + h) * a.q_len + q;
  if (gq == 0 && qvalid) a.delta[stat] = delta;
  const float sc = a.scale, fix = delta0 - delta;
  // rows leave through LDS (the idle tile buffers, 4 KB per wave: row j,
  // 16-byte chunks swizzled as in the tiles) as 16-byte row stores
  static_assert(kWaves <= 8, "a 16-row half of one tile buffer per wave");
  T* const so = (wave / 2 == 0 ? s_k0 : wave / 2 == 1 ? s_k1 : wave / 2 == 2 ? s_k2 : s_v0) + (wave % 2) * 16 * D;
#pragma unroll
  for (int db = 0; db < kDB; ++db) {
    const int e = 16 * db + 4 * gq;  // first of the lane's four elements
    Mfma<T>::store4(so + j * D + ((((e >> 3) ^ Q::swz(j)) << 3) | (e & 7)),
                    sc * __builtin_fmaf(fix, kbar[db][0], dq[db][0]), sc * __builtin_fmaf(fix, kbar[db][1], dq[db][1]),
                    sc * __builtin_fmaf(fix, kbar[db][2], dq[db][2]), sc * __builtin_fmaf(fix, kbar[db][3], dq[db][3]));
  }
  __syncthreads();
  T* const dqp = static_cast<T*>(a.dq);
#pragma unroll
  for (int r0 = 0; r0 < 16; r0 += Q::kRowsPerLoad) {
    const int r = r0 + lrow, row = wrow0 + r;
    if (row < rows) {
      const uint4 v = *reinterpret_cast<const uint4*>(so + r * D + ((lpos ^ Q::swz(r)) << 3));
      // non-temporal: nothing later in the backward reads dQ (-1%)
      typedef unsigned int nt_u32x4 __attribute__((ext_vector_type(4)));
      __builtin_nontemporal_store(nt_u32x4{v.x, v.y, v.z, v.w},
                                  reinterpret_cast<nt_u32x4*>(dqp + (((int64_t)b * a.q_len + row) * hq + h) * D + lpos * 8));
    }
  }
}

// ----------------------------------------------- dK / dV, bf16, 16 keys a wave
//
// The bf16 dK/dV kernel on the 16x16x32 MFMA: a wave owns 16 keys, so its K
// and V operands (16 VGPRs each at d = 128) and its dK^T and dV^T
// accumulators (32 each) leave room for three waves per SIMD.  A block of four
// waves owns 64 keys of one (sequence, KV head) and walks the (query head,
// 32-row query tile) steps that see them; each step's Q, dO, LSE and Delta are
// staged once in LDS for the four waves by untracked direct loads, two steps
// ahead in three buffers, as in the forward, and each wave reads its MFMA
// operands four ahead of the products.  Per step a wave computes
//   S  = Q K^T  - LSE/scale    (two 16 x 16 blocks: query rows 0-15, 16-31)
//   dP = dO V^T - Delta
//   P = exp2(scale log2e S),  dZ = P dP     (masked)
//   dV^T += dO^T P,  dK^T += Q^T dZ          (d x keys, 16-row blocks of d)
// The C layout of the 16x16 MFMA gives lane (g, j) (g = lane / 16) rows 4g +
// i (i < 4) and column j; the P.V-type products take their K index (query
// rows) in the order k = 8g + t <-> row 4g + t (t < 4), 16 + 4g + t - 4
// (t >= 4), so P and dZ are their own B operands and dO^T / Q^T come from two
// transposed LDS reads (rows 4g.., 16 + 4g..) per head-dim block.
template <int D, int G, bool kRuns>
__global__ __launch_bounds__(256, 3) void prefill_bwd_dkdv16_kernel(PrefillBwdArgs a) {
  typedef bf16_bits T;
  typedef QTile<T, D> Q;
  typedef bf16x8_t Frag;
  constexpr int kWaves = 4;
  constexpr int kBlockKeys = 16 * kWaves;
  constexpr int kQ = 32;           // query rows per step
  constexpr int kDC = D / 32;      // K-dim chunks of the S and dP products
  constexpr int kDB = D / 16;      // 16-row blocks of dK^T and dV^T
  constexpr int kLoadsPerWave = 2 * Q::kLoads / kWaves;  // Q and dO direct loads per step
  static_assert((2 * Q::kLoads) % kWaves == 0, "loads split evenly over waves");
  constexpr int kVm = kLoadsPerWave;                     // (+1 for the wave that loads LSE / Delta)

  struct __attribute__((aligned(256))) Buf {
    T q[Q::kElems];
    T g[Q::kElems];
    float l[2 * kQ];  // LSE, Delta
  };
  __shared__ Buf s_b0, s_b1, s_b2;

  int pair, kt;
  dkdv_item(blockIdx.x, gridDim.x, a.num_key_tiles, pair, kt);
  const int heads = a.pv.kv_heads;
  const int g = pair % heads;
  const int b = pair / heads;

  const auto sp = span_view<kRuns>(a, b, a.w_eff);
  const int rows = min(sp.rows(), a.q_len);
  const int clen = min(min(sp.clen(), a.pv.max_pages << a.pv.page_shift), a.hat_cap);
  const int kb0 = kt * kBlockKeys;
  if (kb0 >= clen || rows == 0) return;  // block-uniform

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int gq = lane >> 4, j = lane & 15;  // lane group, column of the 16x16 C layout
  const int hq = a.num_q_heads;
  const int kw = kb0 + 16 * wave;   // this wave's first key
  const int key = kw + j;           // this lane's key
  const int tau = key < clen ? sp.visible_from(key, a.mask_mode) : INT_MAX;
  // first row that sees a key of this wave, and from which row on every
  // valid key of the wave is visible
  const int wave_from = kw < clen ? sp.visible_from(kw, a.mask_mode) : INT_MAX;
  const int wave_all = kw < clen ? sp.visible_from(min(kw + 15, clen - 1), a.mask_mode) : INT_MAX;

  // K and V operands of this lane's key: elements 32c + 8 gq .. +7 (B operand
  // layout of S = Q K^T and dP = dO V^T); a key past the cache or without a
  // page reads a row of page 0 (its column of every product is never stored)
  Frag kf[kDC], vf[kDC];
  {
    const int shift = a.pv.page_shift;
    const int32_t e = a.table[(int64_t)b * a.pv.max_pages + min(key >> shift, a.pv.max_pages - 1)];
    const bool ok = key < clen && e >= 0 && e < a.pv.num_pages;
    const int64_t off = page_row<D>(ok ? e : 0, g, key & ((1 << shift) - 1), a.pv) + 8 * gq;
    const T* kp = static_cast<const T*>(a.k_pages) + off;
    const T* vp = static_cast<const T*>(a.v_pages) + off;
    static_for<kDC>([&](auto c) {
      constexpr int kC = decltype(c)::value;
      untracked_load16<kC * 64>(kf[kC], kp);
      untracked_load16<kC * 64>(vf[kC], vp);
    });
  }

  // steps: (query head, 32-row tile) pairs from the first tile a key of the
  // block is visible in
  const int q_first = sp.visible_from(kb0, a.mask_mode);
  const int t0 = q_first / kQ, t1 = (rows + kQ - 1) / kQ;
  const int n_steps = max(t1 - t0, 0) * G;

  // Step n's Q and dO rows (rows past the end read the last row: finite, and
  // masked), 16-byte chunks swizzled per row (QTile), plus LSE (lanes 0-31)
  // and Delta (32-63) of its rows by the last wave.  The row base is uniform.
  const int lrow = lane / Q::kChunks, lpos = lane % Q::kChunks;
  const int rlast = rows - 1;
  auto load_step = [&](int n, Buf& bf) __attribute__((always_inline)) {
    const int h = g * G + n % G;
    const int q0 = (t0 + n / G) * kQ;
    const int rbase = min(q0, rlast);
    const uint64_t row_bytes = (uint64_t)hq * D * sizeof(T);
    const uint64_t base_off = (((uint64_t)b * a.q_len + rbase) * hq + h) * D * sizeof(T);
    const char* qb = static_cast<const char*>(a.q) + base_off;
    const char* gb = static_cast<const char*>(a.dout) + base_off;
#pragma unroll
    for (int i = 0; i < kLoadsPerWave; ++i) {
      const int l = wave * kLoadsPerWave + i;           // 0 .. 2 kLoads - 1: Q loads, then dO loads
      const bool is_g = l >= Q::kLoads;                 // uniform
      const int lq = is_g ? l - Q::kLoads : l;
      const int r = lq * Q::kRowsPerLoad + lrow;        // row within the tile
      const uint32_t off = (uint32_t)((uint64_t)(min(q0 + r, rlast) - rbase) * row_bytes) +
                           ((lpos ^ Q::swz(r)) << 4);
      lds_dma16(is_g ? gb : qb, off, lds_addr((is_g ? bf.g : bf.q) + lq * Q::kRowsPerLoad * D));
    }
    if (wave == kWaves - 1) {
      const float* src = lane < 32 ? a.lse : a.delta;
      const int64_t stat = ((int64_t)b * hq + h) * a.q_len + min(q0 + (lane & 31), rlast);
      lds_dma4(src + stat, lds_addr(bf.l));
    }
  };

  typedef float f32x4 __attribute__((ext_vector_type(4)));
  f32x4 dk[kDB], dv[kDB];
#pragma unroll
  for (int db = 0; db < kDB; ++db)
#pragma unroll
    for (int i = 0; i < 4; ++i) dk[db][i] = dv[db][i] = 0.f;

  // Fragment addresses (bytes), one register per tile and pattern:
  //  - row-wise A operand of S / dP: lane (gq, j) reads row 16blk + j, chunk
  //    (4c + gq) ^ swz(row) = 4c ^ x with x = gq ^ swz(j) (swz(16blk + j) =
  //    swz(j)): address ar ^ 64c, plus 16 rows for blk = 1;
  //  - transposed A operand of dV^T / dK^T (ds_read_b64_tr_b16): lane j of
  //    group gq points at row 4gq + j/4 (and 16 + 4gq + j/4), elements 16db +
  //    4(j%4) .. +3, i.e. chunk 2db + e (e = (j%4)/2) at position 2db ^ (e ^
  //    swz(row)), swz(row) the same for both rows: address at ^ 32db.
  const int rr = 4 * gq + (j >> 2);
  const uint32_t ar_off = (uint32_t)(j * D * 2 + ((gq ^ Q::swz(j)) << 4));
  const uint32_t at_off = (uint32_t)(rr * D * 2 + ((((j & 3) >> 1) ^ Q::swz(rr)) << 4) + ((j & 1) << 3));
  const float neg_inv_scale = -1.f / a.scale;
  typedef __attribute__((address_space(3))) const u16x8_t* lds_frag_ptr;

  // step n from buffer bf; the loads of steps n+1 and n+2 may be in flight
  auto compute = [&](int n, const Buf& bf) __attribute__((always_inline)) {
    const int q0 = (t0 + n / G) * kQ;
    if (q0 + kQ <= wave_from) return;  // no row of the tile sees a key of this wave
    uint32_t ar_q = lds_addr(bf.q) + ar_off, ar_g = lds_addr(bf.g) + ar_off;
    uint32_t at_q = lds_addr(bf.q) + at_off, at_g = lds_addr(bf.g) + at_off;
    asm volatile("" : "+v"(ar_q), "+v"(ar_g), "+v"(at_q), "+v"(at_g));
    auto arow = [&](uint32_t base, int blk, int c) __attribute__((always_inline)) {
      return __builtin_bit_cast(Frag, *(lds_frag_ptr)(uintptr_t)((base ^ (uint32_t)(64 * c)) + (uint32_t)(blk * 16 * D * 2)));
    };
    auto atr = [&](uint32_t base, int db) __attribute__((always_inline)) {
      const uint32_t al = base ^ (uint32_t)(32 * db);
      const s16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_ptr)(uintptr_t)al);
      const s16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_ptr)(uintptr_t)(al + 16 * D * 2));
      const u16x8_t v = {(unsigned short)lo[0], (unsigned short)lo[1], (unsigned short)lo[2], (unsigned short)lo[3],
                         (unsigned short)hi[0], (unsigned short)hi[1], (unsigned short)hi[2], (unsigned short)hi[3]};
      return __builtin_bit_cast(Frag, v);
    };
    // S and dP accumulators start from -LSE/scale and -Delta of their rows
    f32x4 s[2], dp[2];
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
      const float4 lv = *reinterpret_cast<const float4*>(bf.l + 16 * blk + 4 * gq);
      const float4 dl = *reinterpret_cast<const float4*>(bf.l + kQ + 16 * blk + 4 * gq);
      s[blk][0] = lv.x * neg_inv_scale; s[blk][1] = lv.y * neg_inv_scale;
      s[blk][2] = lv.z * neg_inv_scale; s[blk][3] = lv.w * neg_inv_scale;
      dp[blk][0] = -dl.x; dp[blk][1] = -dl.y; dp[blk][2] = -dl.z; dp[blk][3] = -dl.w;
    }
    __builtin_amdgcn_sched_barrier(0);  // (these reads first)
    // S / dP: 4 kDC MFMAs over 2 kDC row-wise operands of each tile, read
    // kAheadS ahead of the chain
    constexpr int kNS = 4 * kDC;  // (c, blk, S or dP)
    auto aop = [&](int idx) __attribute__((always_inline)) {
      const int c = idx / 4, blk = (idx / 2) % 2, t = idx % 2;
      return arow(t ? ar_g : ar_q, blk, c);
    };
    constexpr int kAheadS = 4;
    Frag sb[kAheadS];
#pragma unroll
    for (int i = 0; i < kAheadS; ++i) sb[i] = aop(i);
#pragma unroll
    for (int idx = 0; idx < kNS; ++idx) {
      const Frag cur = sb[idx % kAheadS];
      if (idx + kAheadS < kNS) sb[idx % kAheadS] = aop(idx + kAheadS);
      const int c = idx / 4, blk = (idx / 2) % 2;
      if (idx % 2 == 0) s[blk] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(cur, kf[c], s[blk], 0, 0, 0);
      else dp[blk] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(cur, vf[c], dp[blk], 0, 0, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x100, kAheadS, 0);  // DS reads
#pragma unroll
    for (int idx = 0; idx + kAheadS < kNS; ++idx) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);      // MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, kAheadS, 0);

    // the first transposed operands of dV / dK, read during the softmax
    constexpr int kNT = 2 * kDB;  // (db, dV or dK)
    auto top = [&](int idx) __attribute__((always_inline)) { return atr(idx % 2 ? at_q : at_g, idx / 2); };
    constexpr int kAheadT = 4;
    Frag tb[kAheadT];
#pragma unroll
    for (int i = 0; i < kAheadT; ++i) tb[i] = top(i);
    __builtin_amdgcn_sched_barrier(0);

    // P and dZ in the B-operand order of the dV / dK products: element t of
    // a lane is row 4gq + t (t < 4) or 16 + 4gq + t - 4
    Frag pf, zf;
    float pv[8];
#pragma unroll
    for (int blk = 0; blk < 2; ++blk)
#pragma unroll
      for (int i = 0; i < 4; ++i) pv[4 * blk + i] = fast_exp2(s[blk][i] * a.scale_log2);
    if (q0 < wave_all || q0 + kQ > rows) {  // uniform: some row or key masked
      // row 16 blk + 4 gq + i of the tile is visible to this lane's key iff
      // it lies in [tau, rows): 16 blk + i in [lo, hi)
      const int lo = tau - q0 - 4 * gq, hi = rows - q0 - 4 * gq;
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const int r = 16 * (t / 4) + t % 4;
        pv[t] = r >= lo && r < hi ? pv[t] : 0.f;
      }
    }
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      pf[t] = (__bf16)pv[t];
      zf[t] = (__bf16)(pv[t] * dp[t / 4][t % 4]);
    }
#pragma unroll
    for (int idx = 0; idx < kNT; ++idx) {
      const Frag cur = tb[idx % kAheadT];
      if (idx + kAheadT < kNT) tb[idx % kAheadT] = top(idx + kAheadT);
      const int db = idx / 2;
      if (idx % 2 == 0) dv[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(cur, pf, dv[db], 0, 0, 0);
      else dk[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(cur, zf, dk[db], 0, 0, 0);
    }
#pragma unroll
    for (int idx = 0; idx + kAheadT < kNT; ++idx) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 1);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 1);  // (two transposed reads)
    }
    __builtin_amdgcn_sched_group_barrier(0x008, kAheadT, 1);
  };

  // prologue: this wave's K/V operands, steps 0 and 1; wait for the operands
  // and step 0 (step 1 may stay in flight)
  const int my_vm = kVm + (wave == kWaves - 1 ? 1 : 0);
  if (n_steps > 0) load_step(0, s_b0);
  if (n_steps > 1) load_step(1, s_b1);
  auto barrier_after = [&](int n) __attribute__((always_inline)) {
    // step n+1's loads landed once only step n+2's are in flight
    if (n + 2 < n_steps) {
      if (my_vm == kVm) bare_barrier<kVm>();
      else bare_barrier<kVm + 1>();
    } else {
      bare_barrier<0>();
    }
  };
  barrier_after(-1);
  auto step = [&](int n, auto par) __attribute__((always_inline)) {
    constexpr int kPar = decltype(par)::value;
    Buf& cur = kPar == 0 ? s_b0 : kPar == 1 ? s_b1 : s_b2;
    Buf& nxt2 = kPar == 0 ? s_b2 : kPar == 1 ? s_b0 : s_b1;  // the buffer step n-1 used
    if (n + 2 < n_steps) load_step(n + 2, nxt2);
    compute(n, cur);
    barrier_after(n);
  };
  for (int n = 0; n < n_steps; n += 3) {
    step(n, std::integral_constant<int, 0>());
    if (n + 1 >= n_steps) break;
    step(n + 1, std::integral_constant<int, 1>());
    if (n + 2 >= n_steps) break;
    step(n + 2, std::integral_constant<int, 2>());
  }

  // lane (gq, j) holds d = 16db + 4gq + i (i < 4) of its key
  if (key >= clen) return;
  float* dkrow = a.dk_hat + (((int64_t)b * a.hat_cap + key) * heads + g) * D + 4 * gq;
  float* dvrow = a.dv_hat + (((int64_t)b * a.hat_cap + key) * heads + g) * D + 4 * gq;
  const float sc = a.scale;
#pragma unroll
  for (int db = 0; db < kDB; ++db) {
    *reinterpret_cast<float4*>(dkrow + 16 * db) = make_float4(dk[db][0] * sc, dk[db][1] * sc, dk[db][2] * sc, dk[db][3] * sc);
    *reinterpret_cast<float4*>(dvrow + 16 * db) = make_float4(dv[db][0], dv[db][1], dv[db][2], dv[db][3]);
  }
}

template <typename T, int D, int G, bool kRuns>
hipError_t launch_bwd_r(const PrefillBwdArgs& a, int batch, hipStream_t s) {
  const unsigned qitems = (unsigned)(batch * a.pv.kv_heads * a.num_q_tiles);
  hipError_t e;
  if constexpr (sizeof(T) == 2)
    e = launch_struct(prefill_bwd_dq16_kernel<D, G, kRuns>, dim3(qitems), dim3(DqShape16<G>::kThreads), s, a);
  else
    e = launch_struct(prefill_bwd_dq_kernel<T, D, G, kRuns>, dim3(qitems), dim3(PrefillShape<G>::kThreads), s, a);
  if (e != hipSuccess) return e;
  const unsigned kitems = (unsigned)(batch * a.pv.kv_heads * a.num_key_tiles);
  if constexpr (sizeof(T) == 2)
    return launch_struct(prefill_bwd_dkdv16_kernel<D, G, kRuns>, dim3(kitems), dim3(256), s, a);
  else
    return launch_struct(prefill_bwd_dkdv_kernel<T, D, G, kRuns>, dim3(kitems),
                         dim3(KvBwdShape<T, D>::kThreads), s, a);
}

template <typename T, int D, int G>
hipError_t launch_bwd_g(const PrefillBwdArgs& a, int batch, hipStream_t s) {
  return a.segs.seg_start ? launch_bwd_r<T, D, G, true>(a, batch, s)
                          : launch_bwd_r<T, D, G, false>(a, batch, s);
}

template <typename T, int D>
hipError_t launch_bwd_d(const PrefillBwdArgs& a, int group, int batch, hipStream_t s) {
  switch (group) {
    case 1: return launch_bwd_g<T, D, 1>(a, batch, s);
    case 2: return launch_bwd_g<T, D, 2>(a, batch, s);
    case 4: return launch_bwd_g<T, D, 4>(a, batch, s);
    default: return launch_bwd_g<T, D, 8>(a, batch, s);
  }
}

}  // namespace

int prefill_bwd_rows_per_tile(int dtype, int group) {
  if (dtype == 1) {  // prefill_bwd_dq16_kernel
    switch (group) {
      case 1: return DqShape16<1>::kRows;
      case 2: return DqShape16<2>::kRows;
      case 4: return DqShape16<4>::kRows;
      default: return DqShape16<8>::kRows;
    }
  }
  switch (group) {
    case 1: return PrefillShape<1>::kRows;
    case 2: return PrefillShape<2>::kRows;
    case 4: return PrefillShape<4>::kRows;
    default: return PrefillShape<8>::kRows;
  }
}

int prefill_bwd_keys_per_block(int dtype, int head_dim) {
  if (dtype == 1) return 64;  // prefill_bwd_dkdv16_kernel: 16 keys per wave, four waves
  return head_dim == 128 ? KvBwdShape<float, 128>::kKeys : KvBwdShape<float, 64>::kKeys;
}

hipError_t launch_prefill_bwd(const PrefillBwdArgs& a, int dtype, int head_dim, int group,
                              int batch, hipStream_t s) {
  if (dtype == 1) {
    if (head_dim == 128) return launch_bwd_d<bf16_bits, 128>(a, group, batch, s);
    return launch_bwd_d<bf16_bits, 64>(a, group, batch, s);
  }
  if (head_dim == 128) return launch_bwd_d<float, 128>(a, group, batch, s);
  return launch_bwd_d<float, 64>(a, group, batch, s);
}

}  // namespace skv
